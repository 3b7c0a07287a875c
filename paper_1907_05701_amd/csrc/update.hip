// HBM-streaming kernels on the flat parameter vector:
//   - the super-learner reduction g = scale * sum_r g_r (eq. 6's bracket),
//   - the ADPSGD local update fused with it (one column of eq. 7: SGD plus
//     0.5/0.5 averaging with a ring neighbour), optionally refreshing the
//     bf16 operand copy and the neighbour's column,
//   - the float32 -> bf16 operand copy on its own.
// Each element goes through one fixed float32 operation order with no fused
// multiply-add (contraction is switched off in these functions), so results
// are reproducible bit for bit.
#include "common.hpp"

struct GradPtrs {
  const float* p[MAX_REPLICAS];
};

__device__ __forceinline__ float reduce_one(const GradPtrs& g, int R, float scale, int64_t i) {
#pragma clang fp contract(off)
  float s = g.p[0][i];
  for (int r = 1; r < R; ++r) s = s + g.p[r][i];
  return s * scale;
}

__device__ __forceinline__ f32x4 ld4(const float* p, int64_t i4) {
  return __builtin_nontemporal_load((const f32x4*)p + i4);
}

__device__ __forceinline__ f32x4 reduce_four(const GradPtrs& g, int R, float scale, int64_t i4) {
#pragma clang fp contract(off)
  f32x4 s = ld4(g.p[0], i4);
  for (int r = 1; r < R; ++r) s = s + ld4(g.p[r], i4);
  return s * scale;
}

__device__ __forceinline__ float update_one(float th, float pe, float g, float lr, bool eq7) {
#pragma clang fp contract(off)
  const float t = lr * g;
  if (eq7) {
    const float v = th + pe;
    const float a = v * 0.5f;
    return a - t;
  }
  const float u = th - t;
  const float v = u + pe;
  return v * 0.5f;
}

__global__ __launch_bounds__(256) void replica_reduce_kernel(GradPtrs g, int R, float scale,
                                                             int64_t n, float* out, int vec) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t done = 0;
  if (vec) {
    const int64_t n4 = n / 4;
    for (int64_t i4 = tid; i4 < n4; i4 += stride) ((f32x4*)out)[i4] = reduce_four(g, R, scale, i4);
    done = n4 * 4;
  }
  for (int64_t i = done + tid; i < n; i += stride) out[i] = reduce_one(g, R, scale, i);
}

__global__ __launch_bounds__(256) void adpsgd_kernel(float* __restrict__ theta,
                                                     float* __restrict__ peer, GradPtrs g, int R,
                                                     float scale, int64_t n, float lr,
                                                     uint32_t flags, bf16* __restrict__ lp, int vec) {
  const bool eq7 = flags & ADPSGD_ORDER_EQ7;
  const bool wpeer = flags & ADPSGD_WRITE_PEER;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t done = 0;
  if (vec) {
    const int64_t n4 = n / 4;
    for (int64_t i4 = tid; i4 < n4; i4 += stride) {
      const f32x4 gg = reduce_four(g, R, scale, i4);
      const f32x4 th = ld4(theta, i4);
      const f32x4 pe = ld4(peer, i4);
      f32x4 nw;
#pragma unroll
      for (int k = 0; k < 4; ++k) nw[k] = update_one(th[k], pe[k], gg[k], lr, eq7);
      __builtin_nontemporal_store(nw, (f32x4*)theta + i4);
      if (wpeer) __builtin_nontemporal_store(nw, (f32x4*)peer + i4);
      if (lp) {
        typedef bf16 bf16x4 __attribute__((ext_vector_type(4)));
        bf16x4 b;
#pragma unroll
        for (int k = 0; k < 4; ++k) b[k] = (bf16)nw[k];
        __builtin_nontemporal_store(b, (bf16x4*)lp + i4);
      }
    }
    done = n4 * 4;
  }
  for (int64_t i = done + tid; i < n; i += stride) {
    const float nw = update_one(theta[i], peer[i], reduce_one(g, R, scale, i), lr, eq7);
    theta[i] = nw;
    if (wpeer) peer[i] = nw;
    if (lp) lp[i] = (bf16)nw;
  }
}

__global__ __launch_bounds__(256) void pack_bf16_kernel(const float* __restrict__ theta, int64_t n,
                                                        bf16* __restrict__ lp, int vec) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t done = 0;
  if (vec) {
    typedef bf16 bf16x4 __attribute__((ext_vector_type(4)));
    const int64_t n4 = n / 4;
    for (int64_t i4 = tid; i4 < n4; i4 += stride) {
      const f32x4 v = ld4(theta, i4);
      bf16x4 b;
#pragma unroll
      for (int k = 0; k < 4; ++k) b[k] = (bf16)v[k];
      ((bf16x4*)lp)[i4] = b;
    }
    done = n4 * 4;
  }
  for (int64_t i = done + tid; i < n; i += stride) lp[i] = (bf16)theta[i];
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }
static bool aligned8(const void* p) { return ((uintptr_t)p & 7) == 0; }

static unsigned stream_grid(int64_t n) {
  // one 4-element vector per thread up to 64 Ki workgroups (measured on
  // MI355X at n = 43 M: 5.98 TB/s with a 4 Ki cap, 6.14 TB/s without it)
  const int64_t blocks = cdiv(cdiv(n, 4), 256);
  return (unsigned)std::max<int64_t>(1, std::min<int64_t>(blocks, 65536));
}

static int fill_grads(const float* const* grads, int32_t R, GradPtrs* g, bool* all16) {
  if (!grads) return blstm_fail(BLSTM_EINVAL, "grads is NULL");
  if (R < 1 || R > MAX_REPLICAS) return blstm_fail(BLSTM_EUNSUPPORTED, "R must be in [1, %d]", MAX_REPLICAS);
  for (int r = 0; r < MAX_REPLICAS; ++r) g->p[r] = nullptr;
  for (int r = 0; r < R; ++r) {
    if (!grads[r]) return blstm_fail(BLSTM_EINVAL, "grads[%d] is NULL", r);
    g->p[r] = grads[r];
    *all16 = *all16 && aligned16(grads[r]);
  }
  return BLSTM_OK;
}

extern "C" int replica_grad_reduce(const float* const* grads, int32_t R, int64_t n, float scale,
                                   float* out, hipStream_t stream) {
  if (!out) return blstm_fail(BLSTM_EINVAL, "out is NULL");
  if (n < 0) return blstm_fail(BLSTM_EINVAL, "n < 0");
  GradPtrs g;
  bool a16 = aligned16(out);
  int rc = fill_grads(grads, R, &g, &a16);
  if (rc) return rc;
  if (n == 0) return BLSTM_OK;
  BLSTM_LAUNCH("replica_reduce", replica_reduce_kernel, dim3(stream_grid(n)), dim3(256), 0, stream,
               g, R, scale, n, out, a16 ? 1 : 0);
  return blstm_check_launch("replica_grad_reduce");
}

extern "C" int adpsgd_step(float* theta, float* theta_peer, const float* const* grads, int32_t R,
                           float scale, int64_t n, float lr, uint32_t flags, void* theta_lp,
                           hipStream_t stream) {
  if (!theta || !theta_peer) return blstm_fail(BLSTM_EINVAL, "theta/theta_peer is NULL");
  if (n < 0) return blstm_fail(BLSTM_EINVAL, "n < 0");
  if (flags & ~(uint32_t)(ADPSGD_ORDER_EQ7 | ADPSGD_WRITE_PEER))
    return blstm_fail(BLSTM_EINVAL, "unknown flags 0x%x", flags);
  if (theta == theta_peer) return blstm_fail(BLSTM_EINVAL, "theta and theta_peer alias");
  GradPtrs g;
  bool a16 = aligned16(theta) && aligned16(theta_peer) && (!theta_lp || aligned8(theta_lp));
  int rc = fill_grads(grads, R, &g, &a16);
  if (rc) return rc;
  if (n == 0) return BLSTM_OK;
  BLSTM_LAUNCH("adpsgd_update", adpsgd_kernel, dim3(stream_grid(n)), dim3(256), 0, stream, theta,
               theta_peer, g, R, scale, n, lr, flags, (bf16*)theta_lp, a16 ? 1 : 0);
  return blstm_check_launch("adpsgd_step");
}

extern "C" int blstm_pack_params(const blstm_dims* dims, const float* theta, void* theta_lp,
                                 hipStream_t stream) {
  Layout lo;
  int rc = make_layout(dims, &lo);
  if (rc) return rc;
  if (lo.prec != BLSTM_BF16) return BLSTM_OK;
  if (!theta || !theta_lp) return blstm_fail(BLSTM_EINVAL, "theta/theta_lp is NULL");
  const int vec = aligned16(theta) && aligned8(theta_lp);
  BLSTM_LAUNCH("pack_bf16", pack_bf16_kernel, dim3(stream_grid(lo.n)), dim3(256), 0, stream, theta,
               lo.n, (bf16*)theta_lp, vec);
  return blstm_check_launch("blstm_pack_params");
}
