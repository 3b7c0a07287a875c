// Output head of the acoustic model (Section 5.2): a linear bottleneck
// z = W_l y + b_l (no nonlinearity), a softmax layer s = W_s z + b_s over the
// context-dependent HMM states, and the frame cross-entropy averaged over the
// mini-batch (eqs. 1-2, 4), together with its backward pass.
//
// The logits are produced once by an MFMA GEMM with the bias fused in; one
// workgroup per frame then computes max and sum-of-exponentials with an
// online (running-max) reduction across 64-lane wavefronts, the frame loss,
// and overwrites the logits in place with ds = scale * (softmax - onehot),
// which feeds the three backward GEMMs (dW_s, dz, and via dz dW_l and dy).
#include <math.h>

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

template <typename T>
__global__ __launch_bounds__(256) void softmax_ce_rows_kernel(T* __restrict__ S, int K, int Kp,
                                                              const int32_t* __restrict__ labels,
                                                              float scale, float* __restrict__ rowloss) {
  const int64_t m = blockIdx.x;
  T* s = S + m * Kp;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  float mx = -INFINITY, sm = 0.f;
  for (int k = tid; k < K; k += 256) {
    const float v = to_f32(s[k]);
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
  __shared__ float wm[4], ws[4], sh_lse, sh_sl;
  if (lane == 0) { wm[wid] = mx; ws[wid] = sm; }
  __syncthreads();
  if (tid == 0) {
    float M0 = wm[0], S0 = ws[0];
    for (int w = 1; w < 4; ++w) lse_combine(M0, S0, wm[w], ws[w]);
    const float lse = M0 + __logf(S0);
    const int lab = labels[m];
    // an out-of-range label is not read (the loss becomes NaN instead)
    const float sl = (lab >= 0 && lab < K) ? to_f32(s[lab]) : __int_as_float(0x7fc00000);
    sh_lse = lse;
    sh_sl = sl;
    rowloss[m] = lse - sl;
  }
  __syncthreads();
  const float lse = sh_lse;
  const int lab = labels[m];
  for (int k = tid; k < Kp; k += 256) {
    float g = 0.f;
    if (k < K) g = scale * (__expf(to_f32(s[k]) - lse) - (k == lab ? 1.f : 0.f));
    s[k] = from_f32<T>(g);
  }
}

// Single-pass variant for rows of up to SM_TPB*8*NV classes: each thread
// keeps its NV 8-element vectors of the row in registers, so the logits are
// read once and ds written once.  512 threads per row (eight waves, 64
// values each at 32000 classes) measured 25% faster on MI355X than 256
// threads with twice the registers, and than 1024.  The row is held as
// loaded (bf16) and the exponentials are evaluated twice, which halves the
// registers: at eight waves per SIMD (64 VGPRs, a few spilled) four rows
// per CU are in flight, 96 -> 79 us for 2688 rows of 32000 classes (the
// float32 exponentials held instead: 118 VGPRs, two rows per CU).
#define SM_TPB 512
template <typename T, int NV>
__global__ __launch_bounds__(SM_TPB) __attribute__((amdgpu_waves_per_eu(8, 8))) void softmax_ce_rows_reg_kernel(T* __restrict__ S, int K, int Kp,
                                                                     const int32_t* __restrict__ labels,
                                                                     float scale, float* __restrict__ rowloss) {
  // One pass over the row: each thread keeps its logits' exponentials
  // e = exp(s - m_t) against its own maximum m_t and their sum; the
  // (maximum, sum) pairs are combined across the workgroup (one barrier), and
  // ds = scale * (e * exp(m_t - m) / sum - [k == label]).  The thread holding
  // the label's logit writes the frame loss logsumexp - s[label].
  const int64_t m = blockIdx.x;
  T* s = S + m * Kp;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int nvec = Kp / 8;
  const int lab = labels[m];
  // the row stays in registers as loaded (eight bf16 per vector, half the
  // registers of float32 exponentials, so twice the rows per CU); the
  // exponentials are evaluated again for the output
  uint4 raw[NV];
  auto logit = [&](int i, int j) {   // -inf past the K classes
    const int k = (tid + SM_TPB * i) * 8 + j;
    return k < K ? to_f32(((const T*)&raw[i])[j]) : -INFINITY;
  };
  float mt = -INFINITY, slab = 0.f;
  bool have_lab = false;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = tid + SM_TPB * i;
    raw[i] = c < nvec ? *(const uint4*)(s + (int64_t)c * 8) : make_uint4(0u, 0u, 0u, 0u);
  }
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    if (tid + SM_TPB * i >= nvec) continue;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float x = logit(i, j);
      mt = fmaxf(mt, x);
      if ((tid + SM_TPB * i) * 8 + j == lab) { slab = x; have_lab = true; }
    }
  }
  float st = 0.f;
  const float mref = mt == -INFINITY ? 0.f : mt;   // a thread with padding only
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    if (tid + SM_TPB * i >= nvec) continue;
#pragma unroll
    for (int j = 0; j < 8; ++j) st += __expf(logit(i, j) - mref);   // exp(-inf) = 0 for padding
  }
  // combine (max, sum) pairs: within the wave by shuffles, then the waves
  float mw = mt, sw = st;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const float mo = __shfl_xor(mw, off), so = __shfl_xor(sw, off);
    const float mn = fmaxf(mw, mo);
    sw = (mw == -INFINITY ? 0.f : sw * __expf(mw - mn)) + (mo == -INFINITY ? 0.f : so * __expf(mo - mn));
    mw = mn;
  }
  constexpr int NW = SM_TPB / 64;
  __shared__ float rm[NW], rs[NW];
  if (lane == 0) { rm[wid] = mw; rs[wid] = sw; }
  __syncthreads();
  float mx = -INFINITY;
#pragma unroll
  for (int q = 0; q < NW; ++q) mx = fmaxf(mx, rm[q]);
  float sum = 0.f;
#pragma unroll
  for (int q = 0; q < NW; ++q) sum += rm[q] == -INFINITY ? 0.f : rs[q] * __expf(rm[q] - mx);
  const float lse = mx + __logf(sum);
  if (have_lab) rowloss[m] = lse - slab;
  // an out-of-range label is not read (the loss becomes NaN instead)
  if (tid == 0 && !(lab >= 0 && lab < K)) rowloss[m] = __int_as_float(0x7fc00000);
  const float f = scale * __expf(mref - mx) / sum;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int c = tid + SM_TPB * i;
    if (c >= nvec) continue;
    uint4 out;
    T* e = (T*)&out;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int k = c * 8 + j;
      e[j] = from_f32<T>(k < K ? __expf(logit(i, j) - mref) * f - (k == lab ? scale : 0.f) : 0.f);
    }
    *(uint4*)(s + (int64_t)c * 8) = out;
  }
}

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
  T* S = (T*)(hws + lo.S);
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
  // s = z W_s^T + b_s
  gemm_launch<T, true, true, V, V>("gemm_logits", s, opnd(Z, P, P, M), opnd(W + lo.Ws, P, P, K), M,
                                   K, P, 1, 1, epi_store<T>(S, Kp, M, K, 0, 0, theta + lo.bs));
  // per-frame loss and ds (in place)
  {
    // ds in place; rows of up to 32768 classes stay in registers (bf16, 16 B vectors)
    const int nv = (int)cdiv(Kp / 8, SM_TPB);
    const dim3 g((unsigned)M), b(SM_TPB), b256(256);
    if (std::is_same<T, bf16>::value && nv <= 8) {
      if (nv <= 1)
        BLSTM_LAUNCH("softmax_ce_rows", (softmax_ce_rows_reg_kernel<bf16, 1>), g, b, 0, s, (bf16*)S, K, Kp, labels, scale, RL);
      else if (nv <= 2)
        BLSTM_LAUNCH("softmax_ce_rows", (softmax_ce_rows_reg_kernel<bf16, 2>), g, b, 0, s, (bf16*)S, K, Kp, labels, scale, RL);
      else if (nv <= 4)
        BLSTM_LAUNCH("softmax_ce_rows", (softmax_ce_rows_reg_kernel<bf16, 4>), g, b, 0, s, (bf16*)S, K, Kp, labels, scale, RL);
      else
        BLSTM_LAUNCH("softmax_ce_rows", (softmax_ce_rows_reg_kernel<bf16, 8>), g, b, 0, s, (bf16*)S, K, Kp, labels, scale, RL);
    } else {
      BLSTM_LAUNCH("softmax_ce_rows", softmax_ce_rows_kernel<T>, g, b256, 0, s, S, K, Kp, labels, scale, RL);
    }
  }
  BLSTM_LAUNCH("loss_sum", loss_sum_kernel, dim3(1), dim3(256), 0, s, RL, M, scale, loss);
  // db_s = sum over frames of ds
  colsum<T>("colsum_dbs", s, S, M, K, Kp, csp, K, 0, grad + lo.bs, nullptr);
  // dW_s = ds^T z
  gemm_f32<T, false, false, V, V>("gemm_dws", s, opnd(S, Kp, Kp, M), opnd(Z, P, P, M), K, P, M, 1,
                                  lo.sp_dWs, grad + lo.Ws, P, 0, part);
  // bf16: W_s^T and W_l^T copies make dz and dy K-contiguous products
  // dz = ds W_s (float32 and a low-precision copy for the next products);
  // W_s [K][P] is the MN-contiguous operand as it lies (the direct-to-LDS
  // kernel reads it with transposing LDS reads; measured faster than
  // transposing W_s each step first)
  gemm_f32<T, true, false, V, V>("gemm_dz", s, opnd(S, Kp, Kp, M), opnd(W + lo.Ws, P, P, K), M, P,
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
