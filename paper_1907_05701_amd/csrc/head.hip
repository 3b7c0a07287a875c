// Output head of the acoustic model (Section 5.2): a linear bottleneck
// z = W_l y + b_l (no nonlinearity), a softmax layer s = W_s z + b_s over the
// context-dependent HMM states, and the frame cross-entropy averaged over the
// mini-batch (eqs. 1-2, 4), together with its backward pass.
//
// bf16 path: the logits are float32 values that stay in the product's
// accumulators (see the fused products below); ds = scale * (softmax -
// onehot) leaves in bf16 and feeds the three backward GEMMs (dW_s, dz, and
// via dz dW_l and dy).  float32 path: one product writes the logits, then
// one workgroup per frame reduces the row and overwrites it with ds.
#include <math.h>

#include <mutex>
#include <type_traits>

#include "common.hpp"
#include "gemm_kc.hpp"
#include "reduce.hpp"

__device__ __forceinline__ void lse_combine(float& m, float& s, float m2, float s2) {
  const float mx = fmaxf(m, m2);
  const float a = s > 0.f ? s * __expf(m - mx) : 0.f;
  const float b = s2 > 0.f ? s2 * __expf(m2 - mx) : 0.f;
  m = mx;
  s = a + b;
}

// float32 path, any K: logits S (row pitch Kp) -> ds of type TO written in
// place at the start of each row (for TO = float, ds replaces the logits).  Three passes over the row: (max, sum) with a
// running maximum, the frame loss, then ds in 256-wide chunks with a barrier
// between a chunk's reads and its writes (a bf16 write at column k overlaps
// float column k/2, which an earlier or the same chunk has read).
template <typename TO>
__global__ __launch_bounds__(256) void softmax_ce_rows_kernel(float* __restrict__ S, int K, int Kp,
                                                              const int32_t* __restrict__ labels,
                                                              float scale, float* __restrict__ rowloss) {
  const int64_t m = blockIdx.x;
  const float* s = S + m * Kp;
  TO* o = (TO*)(S + m * Kp);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  float mx = -INFINITY, sm = 0.f;
  for (int k = tid; k < K; k += 256) {
    const float v = s[k];
    if (v > mx) {
      sm = sm * __expf(mx - v) + 1.f;
      mx = v;
    } else {
      sm += __expf(v - mx);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const float m2 = __shfl_xor(mx, off);
    const float s2 = __shfl_xor(sm, off);
    lse_combine(mx, sm, m2, s2);
  }
  __shared__ float wm[4], ws[4], sh_lse;
  if (lane == 0) { wm[wid] = mx; ws[wid] = sm; }
  __syncthreads();
  if (tid == 0) {
    float M0 = wm[0], S0 = ws[0];
    for (int w = 1; w < 4; ++w) lse_combine(M0, S0, wm[w], ws[w]);
    const float lse = M0 + __logf(S0);
    const int lab = labels[m];
    // an out-of-range label is not read (the loss becomes NaN instead)
    const float sl = (lab >= 0 && lab < K) ? s[lab] : __int_as_float(0x7fc00000);
    sh_lse = lse;
    rowloss[m] = lse - sl;
  }
  __syncthreads();
  const float lse = sh_lse;
  const int lab = labels[m];
  for (int k0 = 0; k0 < Kp; k0 += 256) {
    const int k = k0 + tid;
    float g = 0.f;
    if (k < K) g = scale * (__expf(s[k] - lse) - (k == lab ? 1.f : 0.f));
    __syncthreads();
    if (k < Kp) o[k] = from_f32<TO>(g);
  }
}

// ---------------------------------------------------------------------------
// bf16 path: the logits never leave the product's accumulators.
//
// Two products with the same tiling compute the logits transposed, s^T =
// W_s z^T (rows: classes, columns: frames), so that each lane holds four
// consecutive classes of one frame.  The first product's epilogue reduces
// each wave's tile to (max, sum of exp(s - max)) per frame and class strip
// (the wave's rows); a small kernel combines the strips into each frame's
// log-sum-exp; the second product's epilogue recomputes the same float32
// logits and writes ds = scale * (softmax - onehot) as bf16 (8 bytes per
// lane) and the frame loss lse - s[label].  The logits are thus exact
// float32 values (bf16 storage of a logit of 20 would carry an error of up
// to 0.06 into the loss and softmax) and 344 MB of float32 logits are neither
// written nor read back.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void lse_pair(float& m, float& s, float m2, float s2) {
  const float mx = fmaxf(m, m2);
  s = (m == -INFINITY ? 0.f : s * __expf(m - mx)) + (m2 == -INFINITY ? 0.f : s2 * __expf(m2 - mx));
  m = mx;
}

template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
// sum over the 16 lanes of a DPP row, in every lane of the row
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_mov<0xB1>(v);    // quad_perm [1,0,3,2]
  v += dpp_mov<0x4E>(v);    // quad_perm [2,3,0,1]
  v += dpp_mov<0x141>(v);   // row_half_mirror
  v += dpp_mov<0x140>(v);   // row_mirror
  return v;
}

// First product: per (frame, strip of `srows` classes) maximum and sum.
struct EpiLogitStats {
  const float* bias;   // b_s [K]
  float2* stats;       // [M][nstrip] (maximum, sum of exp(s - maximum))
  int64_t K, M;        // classes (product rows), frames (product columns)
  int nstrip, srows;
  template <int FM, int FN>
  __device__ __forceinline__ void apply(int, int, int64_t mw, int64_t nw, f32x4 (&acc)[FM][FN], int lane) const {
    if (mw >= K) return;
    const int strip = (int)(mw / srows);
    float bv[FM][4];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t k = mw + i * 16 + (lane >> 4) * 4 + r;
        bv[i][r] = k < K ? bias[k] : -INFINITY;
      }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) mx = fmaxf(mx, acc[i][j][r] + bv[i][r]);
      float sm = 0.f;
      if (mx != -INFINITY) {
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r) sm += __expf(acc[i][j][r] + bv[i][r] - mx);
      }
      // the four lane groups hold the other classes of the same frame
      lse_pair(mx, sm, __shfl_xor(mx, 16), __shfl_xor(sm, 16));
      lse_pair(mx, sm, __shfl_xor(mx, 32), __shfl_xor(sm, 32));
      const int64_t f = nw + j * 16 + (lane & 15);
      if ((lane >> 4) == 0 && f < M) stats[f * nstrip + strip] = make_float2(mx, sm);
    }
  }
};

// Per frame: log-sum-exp of its strips (one wave per frame); a frame whose
// label is outside [0, K) gets a NaN loss (its label is never read).
__global__ __launch_bounds__(256) void logit_lse_kernel(const float2* __restrict__ stats, int nstrip, int64_t M,
                                                        const int32_t* __restrict__ labels, int K,
                                                        float* __restrict__ lse, float* __restrict__ rowloss) {
  const int64_t m = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (m >= M) return;
  float mx = -INFINITY, sm = 0.f;
  for (int i = lane; i < nstrip; i += 64) {
    const float2 p = stats[m * nstrip + i];
    lse_pair(mx, sm, p.x, p.y);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) lse_pair(mx, sm, __shfl_xor(mx, off), __shfl_xor(sm, off));
  if (lane == 0) {
    lse[m] = mx + __logf(sm);
    const int lab = labels[m];
    if (!(lab >= 0 && lab < K)) rowloss[m] = __int_as_float(0x7fc00000);
  }
}

// Second product: ds (bf16, [M][Kp], zero in the padding classes), the
// frame loss at the label's class, and the column sums of ds over the wave's
// frames (db_s partials, one row per block of `fcols` frames, summed in a
// fixed order).  Lane group g = lane / 16 holds classes 4g .. 4g+3 of each
// 16-class fragment; for a fragment pair (i, i+1) the groups g and g ^ 1
// swap halves so that each lane stores 8 consecutive classes (16 bytes):
// even groups classes 8(g/2) .. +7 of fragment i, odd groups those of i+1.
struct EpiSoftmaxDs {
  const float* bias;
  const float* lse;
  const int32_t* labels;
  bf16* ds;
  float* rowloss;
  float* dbp;          // [cdiv(M, fcols)][K] column-sum partials
  float scale;
  int64_t K, Kp, M;
  int fcols;
  template <int FM, int FN>
  __device__ __forceinline__ void apply(int, int, int64_t mw, int64_t nw, f32x4 (&acc)[FM][FN], int lane) const {
    static_assert(FM % 2 == 0, "fragment pairs");
    const int g = lane >> 4;
    float bv[FM][4];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t k = mw + i * 16 + g * 4 + r;
        bv[i][r] = k < K ? bias[k] : 0.f;
      }
    float csum[FM][4];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) csum[i][r] = 0.f;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int64_t f = nw + j * 16 + (lane & 15);
      const bool fok = f < M;
      const float L = fok ? lse[f] : 0.f;
      const int lab = fok ? labels[f] : -1;
      uint2 pk[FM];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        bf16 e[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t k = mw + i * 16 + g * 4 + r;
          const float sv = acc[i][j][r] + bv[i][r];
          const float v = (fok && k < K) ? __expf(sv - L) * scale - (k == lab ? scale : 0.f) : 0.f;
          csum[i][r] += v;
          e[r] = (bf16)v;
          if (fok && k == lab) rowloss[f] = L - sv;
        }
        pk[i] = *(const uint2*)e;
      }
#pragma unroll
      for (int i = 0; i < FM; i += 2) {
        const uint2 send = (g & 1) ? pk[i] : pk[i + 1];
        const uint2 got = make_uint2((uint32_t)__shfl_xor((int)send.x, 16), (uint32_t)__shfl_xor((int)send.y, 16));
        const uint4 v = (g & 1) ? make_uint4(got.x, got.y, pk[i + 1].x, pk[i + 1].y)
                                : make_uint4(pk[i].x, pk[i].y, got.x, got.y);
        const int64_t k0 = mw + (i + (g & 1)) * 16 + (g >> 1) * 8;
        if (fok && k0 < Kp) *(uint4*)(ds + f * Kp + k0) = v;
      }
    }
    // column sums over the wave's frames: across the 16 lanes of a group
    // with DPP adds (lane ^ 1, lane ^ 2 within quads, then the half-row and
    // row mirrors), a fixed order that leaves the sum in every lane
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) csum[i][r] = row16_sum(csum[i][r]);
    if ((lane & 15) == 0 && nw < M) {
      float* row = dbp + (nw / fcols) * K;
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t k = mw + i * 16 + g * 4 + r;
          if (k < K) row[k] = csum[i][r];
        }
    }
  }
};

// loss = scale * sum of per-frame losses, in a fixed order.
__global__ __launch_bounds__(256) void loss_sum_kernel(const float* __restrict__ rowloss, int64_t M,
                                                       float scale, float* __restrict__ loss) {
  __shared__ float buf[256];
  float s = 0.f;
  for (int64_t i = threadIdx.x; i < M; i += 256) s += rowloss[i];
  buf[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) buf[threadIdx.x] += buf[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) *loss = scale * buf[0];
}

template <typename T> struct VecH { static constexpr int v = 8; };
template <> struct VecH<float> { static constexpr int v = 4; };

template <typename T>
static int head_impl(const Layout& lo, const float* theta, const T* W, const T* ytop,
                     const int32_t* labels, float scale, float* loss, float* dytop, float* grad,
                     char* hws, hipStream_t s) {
  constexpr int V = VecH<T>::v;
  const int64_t M = lo.M;
  const int P = lo.P, K = lo.K, Kp = lo.Kp, H2 = 2 * lo.H;
  T* Z = (T*)(hws + lo.Z);
  float* RL = (float*)(hws + lo.RL);
  float* DZ = (float*)(hws + lo.DZ);
  T* DZT = (T*)(hws + lo.DZT);
  float* csp = (float*)(hws + lo.HCSP);
  float* part = (float*)(hws + lo.HSKP);

  // z = y W_l^T + b_l.  bf16: split over k (only P/128 column blocks), the
  // fixed-order reduction adds b_l and writes the bf16 z
  if (std::is_same<T, bf16>::value && lo.sp_z > 1) {
    gemm_launch<T, true, true, V, V>("gemm_z", s, opnd(ytop, H2, H2, M), opnd(W + lo.Wl, H2, H2, P), M, P, H2, 1,
                                     lo.sp_z, epi_store<float>(part, P, M, P, (int64_t)lo.sp_z * M * P, M * P));
    BLSTM_LAUNCH("splitk_reduce", splitk_reduce4_kernel<T>, dim3((unsigned)M, (unsigned)cdiv(P, 256), 1), dim3(64), 0,
                 s, (const float*)part, lo.sp_z, M, (int64_t)P, (float*)nullptr, (int64_t)P, (int64_t)0, Z, (int64_t)P,
                 theta + lo.bl);
  } else {
    gemm_launch<T, true, true, V, V>("gemm_z", s, opnd(ytop, H2, H2, M), opnd(W + lo.Wl, H2, H2, P), M,
                                     P, H2, 1, 1, epi_store<T>(Z, P, M, P, 0, 0, theta + lo.bl));
  }
  constexpr bool lp = std::is_same<T, bf16>::value;
  T* DS = (T*)(hws + lo.S);
  if constexpr (lp) {
    // logits transposed (classes x frames) twice: strip statistics, then ds,
    // the frame losses and the db_s partials
    const Opnd Aw = opnd(W + lo.Ws, P, P, K), Bz = opnd(Z, P, P, M);
    const bool kc = kc_eligible(Aw, Bz, P, true, true);
    const int srows = (kc && kc_tall(K, M, 1, 1)) ? KcTileTall::BM / KcTileTall::WM : KcTile::BM / KcTile::WM;
    const int fcols = kc ? KcTile::BN / KcTile::WN : GemmCfgK32::BN / GemmCfgK32::WN;
    static_assert(KcTile::BM / KcTile::WM == GemmCfgK32::BM / GemmCfgK32::WM, "strip rows of the fallback tiles");
    static_assert(KcTile::BN / KcTile::WN == KcTileTall::BN / KcTileTall::WN, "frame columns of the kc tiles");
    const int nstrip = (int)cdiv(K, srows);
    float2* stats = (float2*)(hws + lo.LST);
    float* lse = (float*)(hws + lo.LSE);
    float* dbp = (float*)(hws + lo.LDB);
    EpiLogitStats e1{theta + lo.bs, stats, K, M, nstrip, srows};
    gemm_launch<T, true, true, V, V>("gemm_logits", s, Aw, Bz, K, M, P, 1, 1, e1);
    BLSTM_LAUNCH("logit_lse", logit_lse_kernel, dim3((unsigned)cdiv(M, 4)), dim3(256), 0, s, stats, nstrip, M, labels,
                 K, lse, RL);
    EpiSoftmaxDs e2{theta + lo.bs, lse, labels, (bf16*)DS, RL, dbp, scale, K, Kp, M, fcols};
    gemm_launch<T, true, true, V, V>("gemm_logits_ds", s, Aw, Bz, K, M, P, 1, 1, e2);
    BLSTM_LAUNCH("loss_sum", loss_sum_kernel, dim3(1), dim3(256), 0, s, RL, M, scale, loss);
    // db_s = sum of the per-frame-block partials, in order
    colsum_parts("colsum_dbs", s, dbp, (int)cdiv(M, fcols), K, K, 0, grad + lo.bs, nullptr);
  } else {
    // s = z W_s^T + b_s, then loss and ds in place
    float* S = (float*)(hws + lo.S);
    gemm_launch<T, true, true, V, V>("gemm_logits", s, opnd(Z, P, P, M), opnd(W + lo.Ws, P, P, K), M,
                                     K, P, 1, 1, epi_store<float>(S, Kp, M, K, 0, 0, theta + lo.bs));
    BLSTM_LAUNCH("softmax_ce_rows", softmax_ce_rows_kernel<T>, dim3((unsigned)M), dim3(256), 0, s, S, K, Kp, labels,
                 scale, RL);
    BLSTM_LAUNCH("loss_sum", loss_sum_kernel, dim3(1), dim3(256), 0, s, RL, M, scale, loss);
    // db_s = sum over frames of ds
    colsum<T>("colsum_dbs", s, DS, M, K, Kp, csp, K, 0, grad + lo.bs, nullptr);
  }
  // dW_s = ds^T z
  gemm_f32<T, false, false, V, V>("gemm_dws", s, opnd(DS, Kp, Kp, M), opnd(Z, P, P, M), K, P, M, 1,
                                  lo.sp_dWs, grad + lo.Ws, P, 0, part);
  // bf16: W_s^T and W_l^T copies make dz and dy K-contiguous products
  // dz = ds W_s (float32 and a low-precision copy for the next products);
  // W_s [K][P] is the MN-contiguous operand as it lies (the direct-to-LDS
  // kernel reads it with transposing LDS reads; measured faster than
  // transposing W_s each step first)
  gemm_f32<T, true, false, V, V>("gemm_dz", s, opnd(DS, Kp, Kp, M), opnd(W + lo.Ws, P, P, K), M, P,
                                 K, 1, lo.sp_dz, DZ, P, 0, part, DZT, P);
  // db_l = sum over frames of dz
  colsum<float>("colsum_dbl", s, DZ, M, P, P, csp, P, 0, grad + lo.bl, nullptr);
  // dW_l = dz^T y
  gemm_f32<T, false, false, V, V>("gemm_dwl", s, opnd(DZT, P, P, M), opnd(ytop, H2, H2, M), P, H2, M,
                                  1, lo.sp_dWl, grad + lo.Wl, H2, 0, part);
  // dy = dz W_l (W_l [P][2H] MN-contiguous as it lies)
  gemm_f32<T, true, false, V, V>("gemm_dy", s, opnd(DZT, P, P, M), opnd(W + lo.Wl, H2, H2, P), M,
                                 H2, P, 1, lo.sp_dy, dytop, H2, 0, part);
  return blstm_check_launch("softmax_ce_fwd_bwd");
}

extern "C" int softmax_ce_fwd_bwd(const blstm_dims* dims, const float* theta, const void* theta_lp,
                                  const void* y_top, const int32_t* labels, float loss_scale,
                                  float* loss, float* dy_top, float* grad, void* head_ws,
                                  hipStream_t stream) {
  Layout lo;
  int rc = make_layout(dims, &lo);
  if (rc) return rc;
  if (!theta || !y_top || !labels || !loss || !dy_top || !grad || !head_ws)
    return blstm_fail(BLSTM_EINVAL, "softmax_ce_fwd_bwd: NULL pointer");
  if (lo.M > 0x7fffffff) return blstm_fail(BLSTM_EUNSUPPORTED, "too many frames");
  if (lo.prec == BLSTM_BF16) {
    if (!theta_lp) return blstm_fail(BLSTM_EINVAL, "softmax_ce_fwd_bwd: theta_lp is NULL (bf16)");
    return head_impl<bf16>(lo, theta, (const bf16*)theta_lp, (const bf16*)y_top, labels, loss_scale,
                           loss, dy_top, grad, (char*)head_ws, stream);
  }
  return head_impl<float>(lo, theta, theta, (const float*)y_top, labels, loss_scale, loss, dy_top,
                          grad, (char*)head_ws, stream);
}

// ---------------------------------------------------------------------------
// Allocation-free variant: the head workspace is a file-scope device array
// instead of a caller buffer.  Each device that runs it holds its own copy
// (HEAD_STATIC_SCRATCH_BYTES) until the process ends; host code reaches it
// only through the address hipGetSymbolAddress returns for the current device
// (the array's name is a host-side stand-in), looked up once per device on
// the first call there.  Nothing in the head's kernels needs the workspace
// to start at zero (every partial is written before it is read).  Calls
// that overlap on one device share the array and race.
// ---------------------------------------------------------------------------
static __device__ __attribute__((aligned(256))) unsigned char scratch[HEAD_STATIC_SCRATCH_BYTES];

static int scratch_address(void** out) {
  static std::mutex mu;
  static void* per_dev[64] = {};
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess)
    return blstm_fail(BLSTM_EHIP, "softmax_ce_fwd_bwd_static: hipGetDevice: %s", hipGetErrorString(hipGetLastError()));
  if (dev < 0 || dev >= 64) return blstm_fail(BLSTM_EUNSUPPORTED, "softmax_ce_fwd_bwd_static: device %d", dev);
  std::lock_guard<std::mutex> lock(mu);
  if (!per_dev[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return blstm_fail(BLSTM_EHIP, "softmax_ce_fwd_bwd_static: hipGetSymbolAddress: %s", hipGetErrorString(e));
    per_dev[dev] = p;
  }
  *out = per_dev[dev];
  return BLSTM_OK;
}

extern "C" int softmax_ce_fwd_bwd_static(const blstm_dims* dims, const float* theta, const void* theta_lp,
                                         const void* y_top, const int32_t* labels, float loss_scale, float* loss,
                                         float* dy_top, float* grad, hipStream_t stream) {
  Layout lo;
  int rc = make_layout(dims, &lo);
  if (rc) return rc;
  if (!theta || !y_top || !labels || !loss || !dy_top || !grad)
    return blstm_fail(BLSTM_EINVAL, "softmax_ce_fwd_bwd_static: NULL pointer");
  if (lo.head_bytes > HEAD_STATIC_SCRATCH_BYTES)
    return blstm_fail(BLSTM_EUNSUPPORTED,
                      "softmax_ce_fwd_bwd_static: these dims need %zu bytes of head workspace, above the static "
                      "%zu (use softmax_ce_fwd_bwd with a caller buffer)",
                      lo.head_bytes, (size_t)HEAD_STATIC_SCRATCH_BYTES);
  if (lo.M > 0x7fffffff) return blstm_fail(BLSTM_EUNSUPPORTED, "too many frames");
  void* ws = nullptr;
  rc = scratch_address(&ws);
  if (rc) return rc;
  if (lo.prec == BLSTM_BF16) {
    if (!theta_lp) return blstm_fail(BLSTM_EINVAL, "softmax_ce_fwd_bwd_static: theta_lp is NULL (bf16)");
    return head_impl<bf16>(lo, theta, (const bf16*)theta_lp, (const bf16*)y_top, labels, loss_scale, loss, dy_top,
                           grad, (char*)ws, stream);
  }
  return head_impl<float>(lo, theta, theta, (const float*)y_top, labels, loss_scale, loss, dy_top, grad, (char*)ws,
                          stream);
}
