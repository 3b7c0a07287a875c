// Bidirectional LSTM stack: forward pass and back-propagation through time
// (Section 5.2 of the paper: 6 bidirectional layers, 512 cells per direction,
// 21-frame non-overlapping chunks; the cell is PyTorch's nn.LSTM: gates
// i, f, g, o, no peepholes, two biases; each chunk starts at h = c = 0).
//
// Per layer the forward is
//   1. one all-frames MFMA GEMM for the input projection of both directions,
//      G_x = X W_ih^T + b_ih + b_hh  ([T*B] x [2 * 4H]);
//   2. T recurrent steps, each one launch that advances BOTH directions:
//      a = G_x[t] + h_prev W_hh^T, then the fused gates and cell update.
// The backward runs T reverse-time steps (dh_rec = da_next W_hh, fused gate
// derivatives), then all-frames MFMA GEMMs for dW_ih, dW_hh, dx and a
// column sum for the biases.
//
// Recurrent-step kernels: one workgroup owns 16 batch rows x 16 hidden units
// of one direction; its four waves split the reduction dimension, feed MFMA
// fragments straight from global memory (the step's operands are small and
// L2-resident) and combine their partial sums through LDS in a fixed order,
// so the step is latency-bound rather than bandwidth-bound.
#include <stdlib.h>
#include <string.h>

#include <type_traits>

#include <mutex>

#include "common.hpp"
#include "gemm_kc.hpp"
#include "lstm_persist.hpp"
#include "xpose.hpp"
#include "reduce.hpp"

template <typename T>
__device__ __forceinline__ typename Mfma<T>::frag load_frag(const T* p);
template <>
__device__ __forceinline__ bf16x8 load_frag<bf16>(const bf16* p) {
  return *(const bf16x8*)p;
}
template <>
__device__ __forceinline__ float load_frag<float>(const float* p) {
  return *p;
}

// --------------------------------------------------------------------------
// Forward recurrent step.
//
// Workgroup (unit block q of 16 units, row block of 16*MBK rows, direction).
// Wave w takes m-block w % MBK and the k-part w / MBK of the reduction; all
// of its global loads (W_hh and h_prev fragments, and for the epilogue waves
// the input projection and c_prev) are issued before any arithmetic, so a
// step costs one memory round trip.  Partial sums of the k-parts meet in LDS
// in a fixed order.
// --------------------------------------------------------------------------
template <typename T>
struct RecFwdArgs {
  T* Y;              // layer output [M][2H]; h_prev is read from row tp, h written at row t
  const T* Whh0;     // W_hh of the forward direction [4H][H]
  const T* Whh1;     // W_hh of the reverse direction
  const T* Gx;       // input projection incl. both biases [M][8H]
  float* C;          // cell states [M][2H]
  T* G;              // saved gate pre-activations [M][2][H][4] (direction, unit, gate i/f/g/o)
  int Tn, B, H, tau;
};

template <typename T, int MBK>
__global__ __launch_bounds__(256) void lstm_rec_fwd_step(const RecFwdArgs<T> a) {
  typedef Mfma<T> MT;
  constexpr int KP = 4 / MBK;
  const int q = blockIdx.x, rb = blockIdx.y, d = blockIdx.z;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int mb = w % MBK, kp = w / MBK;
  const int H = a.H, B = a.B;
  const int t = d ? a.Tn - 1 - a.tau : a.tau;
  const int tp = d ? t + 1 : t - 1;
  const int u = q * 16 + (lane & 15);
  const bool epi = kp == 0;

  // epilogue operands first: they do not depend on the reduction
  float gx[4][4], cp[4];
  if (epi) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      int b = rb * 16 * MBK + mb * 16 + (lane >> 4) * 4 + r;
      b = b < B ? b : 0;
      const T* p = a.Gx + ((int64_t)t * B + b) * 8 * H + (int64_t)d * 4 * H + u;
#pragma unroll
      for (int g = 0; g < 4; ++g) gx[r][g] = to_f32(p[g * H]);
      cp[r] = a.tau > 0 ? a.C[((int64_t)tp * B + b) * 2 * H + (int64_t)d * H + u] : 0.f;
    }
  }

  f32x4 acc[4];
#pragma unroll
  for (int g = 0; g < 4; ++g) acc[g] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (a.tau > 0) {
    const T* Wd = d ? a.Whh1 : a.Whh0;
    const int bl = rb * 16 * MBK + mb * 16 + (lane & 15);
    const bool rowok = bl < B;
    const T* arow = a.Y + ((int64_t)tp * B + (rowok ? bl : 0)) * 2 * H + (int64_t)d * H;
    const T* brow[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) brow[g] = Wd + ((int64_t)g * H + u) * H;
    const int koff = (lane >> 4) * MT::KPL;
    const int nks = H / MT::KSTEP;
    // NB k-steps of loads in flight before the first product (a loop of
    // load-then-multiply would wait one memory round trip per k-step)
    constexpr int NB = 4;
    for (int ks0 = kp; ks0 < nks; ks0 += NB * KP) {
      typename MT::frag af[NB], bf[NB][4];
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const int k = (ks0 + j * KP) * MT::KSTEP + koff;
        if (ks0 + j * KP < nks) {
          af[j] = load_frag<T>(arow + k);
#pragma unroll
          for (int g = 0; g < 4; ++g) bf[j][g] = load_frag<T>(brow[g] + k);
        }
      }
#pragma unroll
      for (int j = 0; j < NB; ++j)
        if (ks0 + j * KP < nks) {
          const typename MT::frag a0 = rowok ? af[j] : MT::zero();
#pragma unroll
          for (int g = 0; g < 4; ++g) acc[g] = MT::mma(a0, bf[j][g], acc[g]);
        }
    }
  }

  __shared__ f32x4 red[KP - 1][MBK][4][64];
  if (!epi) {
#pragma unroll
    for (int g = 0; g < 4; ++g) red[kp - 1][mb][g][lane] = acc[g];
  }
  __syncthreads();
  if (!epi) return;
#pragma unroll
  for (int j = 0; j < KP - 1; ++j)
#pragma unroll
    for (int g = 0; g < 4; ++g) acc[g] += red[j][mb][g][lane];

#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int b = rb * 16 * MBK + mb * 16 + (lane >> 4) * 4 + r;
    if (b >= B) continue;
    const int64_t row = (int64_t)t * B + b;
    const float pre[4] = {acc[0][r] + gx[r][0], acc[1][r] + gx[r][1], acc[2][r] + gx[r][2], acc[3][r] + gx[r][3]};
    const float ig = sigmoidf_(pre[0]), fg = sigmoidf_(pre[1]);
    const float gg = tanhf_(pre[2]), og = sigmoidf_(pre[3]);
    const float c = fg * cp[r] + ig * gg;
    const float h = og * tanhf_(c);
    a.C[row * 2 * H + (int64_t)d * H + u] = c;
    a.Y[row * 2 * H + (int64_t)d * H + u] = from_f32<T>(h);
    // the unit's four gate pre-activations together (the backward evaluates
    // the activations from them: stored activations near 1 in bf16 would
    // lose sigma' = sigma (1 - sigma))
    T* gs = a.G + row * 8 * H + (int64_t)d * 4 * H + (int64_t)u * 4;
#pragma unroll
    for (int g = 0; g < 4; ++g) gs[g] = from_f32<T>(pre[g]);
  }
}

// --------------------------------------------------------------------------
// Backward recurrent step (BPTT), same workgroup shape and load schedule:
// dh_rec = da_next W_hh for 16 units, then the gate derivatives.
// --------------------------------------------------------------------------
template <typename T>
struct RecBwdArgs {
  T* DA;             // gate pre-activation gradients [M][8H]; read at t_next, written at t
  const T* WT0;      // W_hh^T of the forward direction [H][4H]
  const T* WT1;      // W_hh^T of the reverse direction
  const float* DY;   // gradient reaching the layer output [M][2H]
  const T* G;        // saved gate pre-activations [M][2][H][4]
  const float* C;    // saved cell states [M][2H]
  float* DC;         // carried cell gradient [2][B][H]
  T* DAT;            // optional: da also written frame-contiguous, [8H][M]
  float* DBP;        // optional: per-(step, 16-row block) sums of da, [Tn][B/16][8H]
  int64_t M;
  int Tn, B, H, tau;
};

template <typename T, int MBK>
__global__ __launch_bounds__(256) void lstm_rec_bwd_step(const RecBwdArgs<T> a) {
  typedef Mfma<T> MT;
  constexpr int KP = 4 / MBK;
  const int q = blockIdx.x, rb = blockIdx.y, d = blockIdx.z;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int mb = w % MBK, kp = w / MBK;
  const int H = a.H, B = a.B, Tn = a.Tn;
  const int t = d ? a.tau : Tn - 1 - a.tau;
  const int tn = d ? t - 1 : t + 1;   // processed just before t in this pass
  const int tp = d ? t + 1 : t - 1;   // forward-pass predecessor of t
  const int u = q * 16 + (lane & 15);
  const bool epi = kp == 0;

  // dh_rec of this 16x16 block over this wave's share of the 4H gate rows.
  // A batch of NB k-steps of operand loads goes out before the first product
  // (load-then-multiply would wait one memory round trip per k-step), and the
  // cell-derivative inputs are loaded behind the first batch.
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
  const bool prod = a.tau > 0;
  const int bl = rb * 16 * MBK + mb * 16 + (lane & 15);
  const bool rowok = bl < B;
  const T* arow = a.DA + ((int64_t)tn * B + (rowok ? bl : 0)) * 8 * H + (int64_t)d * 4 * H;
  const T* brow = (d ? a.WT1 : a.WT0) + (int64_t)u * 4 * H;
  const int koff = (lane >> 4) * MT::KPL;
  const int nks = 4 * H / MT::KSTEP;
  constexpr int NB = 16;
  typename MT::frag af[NB], bf[NB];
  auto issue = [&](int ks0) {
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int k = (ks0 + j * KP) * MT::KSTEP + koff;
      if (ks0 + j * KP < nks) {
        af[j] = load_frag<T>(arow + k);
        bf[j] = load_frag<T>(brow + k);
      }
    }
  };
  auto multiply = [&](int ks0) {
#pragma unroll
    for (int j = 0; j < NB; ++j)
      if (ks0 + j * KP < nks) acc = MT::mma(rowok ? af[j] : MT::zero(), bf[j], acc);
  };
  if (prod) issue(kp);

  // everything the cell derivative needs besides dh_rec (gates stay bf16
  // until used)
  float dy[4], cc[4], cpv[4], dcn[4];
  T graw[4][4];
  if (epi) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      int b = rb * 16 * MBK + mb * 16 + (lane >> 4) * 4 + r;
      b = b < B ? b : 0;
      const int64_t row = (int64_t)t * B + b;
      dy[r] = a.DY[row * 2 * H + (int64_t)d * H + u];
      const T* gs = a.G + row * 8 * H + (int64_t)d * 4 * H + (int64_t)u * 4;
#pragma unroll
      for (int g = 0; g < 4; ++g) graw[r][g] = gs[g];
      cc[r] = a.C[row * 2 * H + (int64_t)d * H + u];
      cpv[r] = (tp >= 0 && tp < Tn) ? a.C[((int64_t)tp * B + b) * 2 * H + (int64_t)d * H + u] : 0.f;
      dcn[r] = a.tau > 0 ? a.DC[((int64_t)d * B + b) * H + u] : 0.f;
    }
  }

  if (prod) {
    multiply(kp);
    for (int ks0 = kp + NB * KP; ks0 < nks; ks0 += NB * KP) {
      issue(ks0);
      multiply(ks0);
    }
  }

  __shared__ f32x4 red[KP - 1][MBK][64];
  if (!epi) red[kp - 1][mb][lane] = acc;
  __syncthreads();
  if (!epi) return;
#pragma unroll
  for (int j = 0; j < KP - 1; ++j) acc += red[j][mb][lane];

  float dav[4][4];   // [row r][gate]
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int b = rb * 16 * MBK + mb * 16 + (lane >> 4) * 4 + r;
    const float ig = sigmoidf_(to_f32(graw[r][0])), fg = sigmoidf_(to_f32(graw[r][1]));
    const float gg = tanhf_(to_f32(graw[r][2])), og = sigmoidf_(to_f32(graw[r][3]));
    const float dh = acc[r] + dy[r];
    const float tc = tanhf_(cc[r]);
    const float dc = dh * og * (1.f - tc * tc) + dcn[r];
    const bool ok = b < B;
    dav[r][0] = ok ? dc * gg * ig * (1.f - ig) : 0.f;
    dav[r][1] = ok ? dc * cpv[r] * fg * (1.f - fg) : 0.f;
    dav[r][2] = ok ? dc * ig * (1.f - gg * gg) : 0.f;
    dav[r][3] = ok ? dh * tc * og * (1.f - og) : 0.f;
    if (!ok) continue;
    const int64_t row = (int64_t)t * B + b;
    a.DC[((int64_t)d * B + b) * H + u] = dc * fg;
    T* da = a.DA + row * 8 * H + (int64_t)d * 4 * H + u;
#pragma unroll
    for (int g = 0; g < 4; ++g) da[g * H] = from_f32<T>(dav[r][g]);
  }
  const int b0 = rb * 16 * MBK + mb * 16 + (lane >> 4) * 4;
  if (a.DAT && b0 < B) {
    // 4 consecutive frames of one gate row: one 8-byte store (B % 4 == 0)
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      T* p = a.DAT + ((int64_t)d * 4 * H + g * H + u) * a.M + (int64_t)t * B + b0;
      if constexpr (sizeof(T) == 2) {
        const bf16 v[4] = {(bf16)dav[0][g], (bf16)dav[1][g], (bf16)dav[2][g], (bf16)dav[3][g]};
        *(uint2*)p = *(const uint2*)v;
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) p[r] = from_f32<T>(dav[r][g]);
      }
    }
  }
  if (a.DBP) {
    // bias gradient partial: the 16 rows of this block, in a fixed order
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      float sg = (dav[0][g] + dav[1][g]) + (dav[2][g] + dav[3][g]);
      sg += __shfl_xor(sg, 16);
      sg += __shfl_xor(sg, 32);
      if (lane < 16)
        a.DBP[((int64_t)a.tau * gridDim.y * MBK + rb * MBK + mb) * 8 * H + (int64_t)d * 4 * H + g * H + u] = sg;
    }
  }
}

// --------------------------------------------------------------------------
// Small helpers: feature conversion, W_hh transposition, column sums.
// --------------------------------------------------------------------------
// The input in the operand precision, rows padded from D to Dp columns
// (zeros).  bf16 with D not a multiple of 8 also gets a copy of the layer-0
// W_ih of both directions padded the same way (wp non-null), so that the
// gate projection's k range (Dp) takes the direct-to-LDS product.  Dp is a
// multiple of 8: each thread writes 8 consecutive columns of one row (one
// 16-byte store for bf16), from vector loads where its 8 columns lie inside
// D and the source is aligned for them.
template <typename T>
__global__ __launch_bounds__(256) void convert_input_kernel(const float* __restrict__ x, int64_t M,
                                                            int D, int Dp, T* __restrict__ X,
                                                            const bf16* __restrict__ w0, int64_t wz, int wrows,
                                                            bf16* __restrict__ wp) {
  const int cpr = Dp / 8;
  const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t row = g / cpr;
  const int k0 = (int)(g % cpr) * 8;
  if (row >= M + (wp ? 2 * (int64_t)wrows : 0)) return;
  if (row < M) {
    const float* src = x + row * D + k0;
    float v[8];
    if (k0 + 8 <= D && (D & 3) == 0 && ((uintptr_t)x & 15) == 0) {
      const float4 p = *(const float4*)src, q = *(const float4*)(src + 4);
      v[0] = p.x; v[1] = p.y; v[2] = p.z; v[3] = p.w; v[4] = q.x; v[5] = q.y; v[6] = q.z; v[7] = q.w;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = x[row * D + min(k0 + e, D - 1)];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = k0 + e < D ? v[e] : 0.f;
    }
    T o[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = from_f32<T>(v[e]);
    T* dst = X + row * Dp + k0;
    if constexpr (sizeof(T) == 2) {
      *(uint4*)dst = *(const uint4*)o;
    } else {
      *(uint4*)dst = *(const uint4*)o;
      *(uint4*)(dst + 4) = *(const uint4*)(o + 4);
    }
  } else {
    const int zr = (int)(row - M), z = zr / wrows, r = zr % wrows;
    const bf16* src = w0 + z * wz + (int64_t)r * D;
    bf16 o[8];
    if (k0 + 8 <= D && ((D | (int)(wz & 3)) & 3) == 0 && ((uintptr_t)w0 & 7) == 0) {
      const uint2 p = *(const uint2*)(src + k0), q = *(const uint2*)(src + k0 + 4);
      *(uint2*)o = p;
      *(uint2*)(o + 4) = q;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = src[min(k0 + e, D - 1)];
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = k0 + e < D ? o[e] : (bf16)0.f;
    }
    *(uint4*)(wp + (int64_t)zr * Dp + k0) = *(const uint4*)o;
  }
}

// out[z][c][r] = in_z[r][c] for 2L matrices of R = 4H rows and C = H columns.
struct TransposeSrc {
  const void* p[2 * MAX_LAYERS];
};

template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(TransposeSrc src, int R, int C, T* out) {
  __shared__ T tile[32][33];
  const T* in = (const T*)src.p[blockIdx.z];
  T* o = out + (int64_t)blockIdx.z * R * C;
  const int r0 = blockIdx.y * 32, c0 = blockIdx.x * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int i = ty; i < 32; i += 8) {
    const int r = r0 + i, c = c0 + tx;
    if (r < R && c < C) tile[i][tx] = in[(int64_t)r * C + c];
  }
  __syncthreads();
  for (int i = ty; i < 32; i += 8) {
    const int c = c0 + i, r = r0 + tx;
    if (r < R && c < C) o[(int64_t)c * R + r] = tile[tx][i];
  }
}


// --------------------------------------------------------------------------
// Host entry points.
// --------------------------------------------------------------------------
template <typename T> struct VecW { static constexpr int v = 8; };   // 16-byte chunks
template <> struct VecW<float> { static constexpr int v = 4; };

// Per-step kernels take 32 rows per workgroup when that still gives at least
// one workgroup per compute unit (W_hh is then read half as often); this
// pays off in the forward step only (measured on MI355X).
static bool step_rows_32(int H, int B) { return (int64_t)(H / 16) * cdiv(B, 32) * 2 >= 256; }

// Which recurrent kernels run.  Default (measured fastest on MI355X at the
// paper's shapes): the persistent kernels for both passes;
// ADPSGD_BLSTM_RECURRENCE=per-step (or ADPSGD_BLSTM_NO_PERSIST=1) the
// per-step kernels.  The persistent kernels need bf16 and a W_hh slice that fits in LDS;
// inside stream capture they are recorded as cooperative kernel nodes.
template <typename T>
static bool use_persistent(int H, int steps, bool backward, hipStream_t s) {
  if (!std::is_same<T, bf16>::value) return false;
  const char* off = getenv("ADPSGD_BLSTM_NO_PERSIST");
  if (off && atoi(off)) return false;
  const char* pol = getenv("ADPSGD_BLSTM_RECURRENCE");
  if (pol && strcmp(pol, "per-step") == 0) return false;
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(s, &cap) != hipSuccess) return false;
  if (cap != hipStreamCaptureStatusNone) {
    // captured launches carry the cooperative attribute; ADPSGD_BLSTM_GRAPH_PERSIST=0
    // keeps graphs on the per-step kernels
    const char* g = getenv("ADPSGD_BLSTM_GRAPH_PERSIST");
    if (g && !atoi(g)) return false;
  }
  return persist_supported(H, steps);
}

static PersistArgs persist_args(const Layout& lo, const bf16* W, char* ws, int l) {
  PersistArgs pa;
  memset(&pa, 0, sizeof(pa));
  pa.W = W;
  pa.whh0 = lo.Whh[l][0];
  pa.whh1 = lo.Whh[l][1];
  pa.X = (uint64_t*)(ws + lo.XCH);
  pa.status = (int*)(ws + lo.SYNC);
  pa.Tn = lo.T;
  pa.B = lo.B;
  pa.H = lo.H;
  pa.tag = (uint32_t)l;
  return pa;
}

// Whether the persistent BPTT adds the split-K partial sums of dX itself
// (ADPSGD_BLSTM_FUSE_DY=0: a separate reduction launch, for comparisons).
static bool fuse_dy() {
  const char* e = getenv("ADPSGD_BLSTM_FUSE_DY");
  return !(e && e[0] == '0');
}

// Whether the persistent forward computes the input projection itself
// (ADPSGD_BLSTM_FUSE_GX=0: a separate product launch, for comparisons).
static bool fuse_gx() {
  const char* e = getenv("ADPSGD_BLSTM_FUSE_GX");
  return !(e && e[0] == '0');
}

template <typename T>
static int fwd_impl(const Layout& lo, const float* theta, const T* W, const float* x, char* ws,
                    T* ytop, hipStream_t s) {
  constexpr int V = VecW<T>::v;
  const int64_t M = lo.M;
  const int H = lo.H, B = lo.B;
  bool xch_cleared = false;   // exchange words cleared once per call (persist_clear)
  // the recurrence status block is initialised on first use (by the
  // persistent path's exchange clear, else here); its flag is sticky until
  // blstm_recurrence_ok reads it
  const bool persist = use_persistent<T>(H, lo.T, false, s);
  bool status_cleared = false;
  if (!persist) {
    if (persist_status_init((int*)(ws + lo.SYNC), s) != hipSuccess) return blstm_check_launch("blstm_fwd");
    status_cleared = true;
  }
  T* X0 = (T*)(ws + lo.X0);
  T* GX = (T*)(ws + lo.GX);
  bf16* WP0 = lo.WP0_bytes ? (bf16*)(ws + lo.WP0) : nullptr;
  {
    const int64_t rows = M + (WP0 ? 2 * 4 * H : 0);
    const unsigned grid = (unsigned)cdiv(rows * (lo.Dp0 / 8), 256);
    BLSTM_LAUNCH("convert_input", convert_input_kernel<T>, dim3(grid), dim3(256), 0, s, x, M, lo.D,
                 lo.Dp0, X0, (const bf16*)W + lo.Wih[0][0], lo.Wih[0][1] - lo.Wih[0][0], 4 * H, WP0);
  }
  for (int l = 0; l < lo.L; ++l) {
    const T* Xl = l == 0 ? X0 : (const T*)(ws + lo.Y[l - 1]);
    const int Dl = lo.layer_in(l), Dpl = lo.layer_in_pitch(l);
    T* Yl = l == lo.L - 1 ? ytop : (T*)(ws + lo.Y[l]);
    T* Gl = (T*)(ws + lo.G[l]);
    float* Cl = (float*)(ws + lo.C[l]);
    // G_x = X W_ih^T + b_ih + b_hh for both directions (batch z = direction)
    const Opnd A = opnd(Xl, Dpl, Dpl, M);
    Opnd Bw = opnd(W + lo.Wih[l][0], Dl, Dl, 4 * H, lo.Wih[l][1] - lo.Wih[l][0]);
    const auto epi = epi_store<T>(GX, 8 * H, M, 4 * H, 4 * H, 0, theta + lo.bih[l][0],
                                  theta + lo.bhh[l][0], lo.bih[l][1] - lo.bih[l][0]);
    // bf16 persistent path: the forward launch computes G_x itself (each
    // workgroup its own rows and gate columns), with the same operands
    const bf16* wih = (l == 0 && WP0) ? WP0 : (const bf16*)(W + lo.Wih[l][0]);
    const int64_t ldw = (l == 0 && WP0) ? Dpl : Dl;
    const int64_t wih_d = (l == 0 && WP0) ? (int64_t)4 * H * Dpl : lo.Wih[l][1] - lo.Wih[l][0];
    const int kin = (l == 0 && WP0) ? Dpl : Dl;
    const bool fuse = persist && std::is_same<T, bf16>::value && fuse_gx() && kin % 8 == 0 && Dpl % 8 == 0 &&
                      ldw % 8 == 0 && wih_d % 8 == 0 && ((uintptr_t)Xl & 15) == 0 && ((uintptr_t)wih & 15) == 0;
    auto launch_gx = [&]() {
      if (l == 0 && WP0) {
        // bf16 with D not a multiple of 8: W_ih padded to the input's pitch
        Bw = opnd(WP0, Dpl, Dpl, 4 * H, (int64_t)4 * H * Dpl);
        gemm_launch<T, true, true, V, V>("gemm_gx", s, A, Bw, M, 4 * H, Dpl, 2, 1, epi);
      } else if (Dl % V == 0)
        gemm_launch<T, true, true, V, V>("gemm_gx", s, A, Bw, M, 4 * H, Dl, 2, 1, epi);
      else
        gemm_launch<T, true, true, V, 4>("gemm_gx", s, A, Bw, M, 4 * H, Dl, 2, 1, epi);
    };
    if (!fuse) launch_gx();
    if (persist) {
      PersistArgs pa = persist_args(lo, (const bf16*)W, ws, l);
      pa.Y = (bf16*)Yl; pa.Gx = (bf16*)GX; pa.C = Cl; pa.G = (bf16*)Gl;
      if (fuse) {
        pa.Xin = (const bf16*)Xl; pa.ldx = Dpl; pa.Kin = kin;
        pa.Wih = wih; pa.ldw = ldw; pa.wih_d = wih_d;
        pa.bih = theta + lo.bih[l][0]; pa.bhh = theta + lo.bhh[l][0]; pa.b_d = lo.bih[l][1] - lo.bih[l][0];
      }
      if (!xch_cleared) {
        xch_cleared = persist_clear(false, pa, s) == hipSuccess;
        status_cleared = status_cleared || xch_cleared;
      }
      if (!status_cleared) {
        (void)hipGetLastError();
        if (persist_status_init((int*)(ws + lo.SYNC), s) != hipSuccess) return blstm_check_launch("blstm_fwd");
        status_cleared = true;
      }
      if (xch_cleared && persist_layer(false, pa, s) == hipSuccess) continue;
      (void)hipGetLastError();   // cooperative launch refused: take the per-step path
      if (fuse) launch_gx();
    }
    RecFwdArgs<T> ra;
    ra.Y = Yl; ra.Whh0 = W + lo.Whh[l][0]; ra.Whh1 = W + lo.Whh[l][1]; ra.Gx = GX; ra.C = Cl;
    ra.G = Gl; ra.Tn = lo.T; ra.B = B; ra.H = H;
    const bool two = step_rows_32(H, B);
    const dim3 grid(H / 16, (unsigned)cdiv(B, two ? 32 : 16), 2);
    TimedRun timed("lstm_rec_fwd", s, lo.T);
    for (int tau = 0; tau < lo.T; ++tau) {
      ra.tau = tau;
      if (two)
        BLSTM_LAUNCH("lstm_rec_fwd", (lstm_rec_fwd_step<T, 2>), grid, dim3(256), 0, s, ra);
      else
        BLSTM_LAUNCH("lstm_rec_fwd", (lstm_rec_fwd_step<T, 1>), grid, dim3(256), 0, s, ra);
    }
  }
  return blstm_check_launch("blstm_fwd");
}

// Side stream for the weight-gradient work of a layer, which then runs
// concurrently with the BPTT of the layer below (it depends only on that
// layer's da, which the per-step kernels write in their own buffer).  One
// non-blocking stream at default priority and 2 events per layer, per device,
// created on first use; used for eager calls only.  ADPSGD_BLSTM_OVERLAP=0
// keeps everything on the caller's stream.
struct SideStream {
  hipStream_t st = nullptr;
  hipEvent_t bptt_done[MAX_LAYERS] = {}, dw_done[MAX_LAYERS] = {};
  bool ok = false, tried = false;
};
static SideStream* side_stream() {
  static SideStream per_dev[64];
  static std::mutex mu;
  const char* env = getenv("ADPSGD_BLSTM_OVERLAP");
  if (env && atoi(env) == 0) return nullptr;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  SideStream& ss = per_dev[dev];
  if (!ss.tried) {
    ss.tried = true;
    bool ok = hipStreamCreateWithFlags(&ss.st, hipStreamNonBlocking) == hipSuccess;
    for (int i = 0; ok && i < MAX_LAYERS; ++i)
      ok = hipEventCreateWithFlags(&ss.bptt_done[i], hipEventDisableTiming) == hipSuccess &&
           hipEventCreateWithFlags(&ss.dw_done[i], hipEventDisableTiming) == hipSuccess;
    ss.ok = ok;
    if (!ok) (void)hipGetLastError();
  }
  return ss.ok ? &ss : nullptr;
}

template <typename T>
static int bwd_impl(const Layout& lo, const T* W, char* ws, const T* ytop, const float* dytop,
                    float* grad, hipStream_t s) {
  bool xch_cleared = false;   // exchange words cleared once per call (persist_clear)
  constexpr int V = VecW<T>::v;
  const int64_t M = lo.M;
  const int H = lo.H, B = lo.B, Tn = lo.T;
  T* WT = (T*)(ws + lo.WT);
  T* DA = (T*)(ws + lo.GX);
  float* DC = (float*)(ws + lo.DC);
  float* part = (float*)(ws + lo.SKP);
  float* csp = (float*)(ws + lo.CSP);
  constexpr bool lp = std::is_same<T, bf16>::value;
  // W_hh^T (bf16 and float32 paths): the per-step BPTT kernels' operand and
  // the persistent kernel's LDS staging source when a workgroup takes more
  // than one 16-row block.  One launch makes all layers'.
  bool have_wt = false;
  auto make_copies = [&]() {
    if constexpr (lp) {
      XposeJobs jobs;
      int n = 0;
      for (int l = 0; l < lo.L; ++l)
        for (int d = 0; d < 2; ++d)
          jobs.j[n++] = XposeJob{(const bf16*)(W + lo.Whh[l][d]), (bf16*)(WT + (int64_t)(2 * l + d) * 4 * H * H),
                                 H, 4 * H, 4 * H, H};
      transpose_bf16("transpose_w", s, jobs, n);
    } else {
      TransposeSrc src;
      for (int i = 0; i < 2 * MAX_LAYERS; ++i) src.p[i] = nullptr;
      for (int l = 0; l < lo.L; ++l)
        for (int d = 0; d < 2; ++d) src.p[2 * l + d] = W + lo.Whh[l][d];
      BLSTM_LAUNCH("transpose_whh", transpose_kernel<T>,
                   dim3((unsigned)cdiv(H, 32), (unsigned)cdiv(4 * H, 32), 2 * lo.L), dim3(256), 0, s,
                   src, 4 * H, H, WT);
    }
    have_wt = true;
  };
  if (!use_persistent<T>(H, lo.T, true, s) || persist_bwd_needs_wt(H, B)) make_copies();
  // weight gradients on the side stream (bf16 per-step BPTT writing da^T):
  // layer l's buffers (da^T, bias partials, split-K partials) alternate by
  // layer parity, so BPTT of layer l waits only for the side work of l+2
  SideStream* side = nullptr;
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(s, &cap) != hipSuccess) { (void)hipGetLastError(); cap = hipStreamCaptureStatusActive; }
  // not under stream capture: replaying graphs with these parallel branches
  // measured far slower on MI355X than the serial graph
  if (lp && lo.write_dat && cap == hipStreamCaptureStatusNone && !use_persistent<T>(H, lo.T, true, s))
    side = side_stream();
  hipStream_t ss = side ? side->st : s;
  float* part_side = side ? (float*)(ws + lo.SKP2) : part;
  // bf16 with da^T and no side stream: each layer's weight-gradient products
  // wait for one grouped launch after the last BPTT (their da^T kept per
  // layer), so a layer's own launch after its BPTT holds only dX, the
  // product the next BPTT needs; the deferred products all have about the
  // same k length and fill whole rounds of the chip together
  const bool defer = lp && lo.write_dat && !side;
  F32Job deferred[2 * MAX_LAYERS];
  int nd = 0;
  // with the persistent BPTT, a layer's dX stays as its split-K partial
  // sums, which the next BPTT adds itself (in the reduction's order) before
  // its steps; the bias sums of every layer then wait for one reduction
  // launch after the last BPTT (on per-layer bias partials)
  const bool dy_parts = defer && fuse_dy() && use_persistent<T>(H, lo.T, true, s) &&
                        persist_bwd_dy_partials_ok(H, B, lo.T);
  ReduceGroup pending_dy;   // the held dX reduction the next BPTT takes over
  pending_dy.n = 0;
  ColSumJob bias_jobs[MAX_LAYERS];
  int nbias = 0;
  const float* dY = dytop;
  for (int l = lo.L - 1; l >= 0; --l) {
    const int par = side ? (l & 1) : 0;
    T* DATl = (T*)(ws + lo.DAT + (defer ? l : par) * lo.dat_bytes);
    float* DBPl = (float*)(ws + lo.DBP + (dy_parts ? l : par) * lo.dbp_bytes);
    if (side && l + 2 < lo.L) (void)hipStreamWaitEvent(s, side->dw_done[l + 2], 0);
    const T* Xl = l == 0 ? (const T*)(ws + lo.X0) : (const T*)(ws + lo.Y[l - 1]);
    const int Dl = lo.layer_in(l), Dpl = lo.layer_in_pitch(l);
    const T* Yl = l == lo.L - 1 ? ytop : (const T*)(ws + lo.Y[l]);
    const T* Gl = (const T*)(ws + lo.G[l]);
    const float* Cl = (const float*)(ws + lo.C[l]);
    // BPTT over the chunk, both directions at once
    bool done = false, step_fused = false;
    if (use_persistent<T>(H, lo.T, true, s)) {
      PersistArgs pa = persist_args(lo, (const bf16*)W, ws, l);
      pa.tag = (uint32_t)(lo.L - 1 - l);   // the backward runs the layers top-down
      pa.DA = (bf16*)DA; pa.DY = dY; pa.C = (float*)Cl; pa.G = (bf16*)Gl;
      pa.WT = have_wt ? (const bf16*)(WT + (int64_t)(2 * l) * 4 * H * H) : nullptr;
      pa.DAT = lo.write_dat ? (bf16*)DATl : nullptr;
      pa.DBP = DBPl;
      pa.M = M;
      if (pending_dy.n == 1) {
        pa.DYP = pending_dy.j[0].part;
        pa.ndy = pending_dy.j[0].splits;
        pa.dy_kstride = pending_dy.j[0].kstride;
      }
      if (!xch_cleared) xch_cleared = persist_clear(true, pa, s) == hipSuccess;
      done = xch_cleared && persist_layer(true, pa, s) == hipSuccess;
      if (!done) (void)hipGetLastError();
      else pending_dy.n = 0;   // the BPTT summed the partials
      step_fused = done;
    }
    // partials nobody summed (the persistent launch did not run): reduce them now
    reduce_group_launch(s, pending_dy);
    pending_dy.n = 0;
    if (!done) {
      if (!have_wt) make_copies();
      RecBwdArgs<T> rb;
      rb.DA = DA; rb.WT0 = WT + (int64_t)(2 * l) * 4 * H * H; rb.WT1 = WT + (int64_t)(2 * l + 1) * 4 * H * H;
      rb.DY = dY; rb.G = Gl; rb.C = Cl; rb.DC = DC; rb.Tn = Tn; rb.B = B; rb.H = H;
      rb.DAT = lo.write_dat ? DATl : nullptr;
      rb.DBP = DBPl;
      rb.M = M;
      const dim3 grid(H / 16, (unsigned)cdiv(B, 16), 2);
      TimedRun timed("lstm_rec_bwd", s, Tn);
      for (int tau = 0; tau < Tn; ++tau) {
        rb.tau = tau;
        BLSTM_LAUNCH("lstm_rec_bwd", (lstm_rec_bwd_step<T, 1>), grid, dim3(256), 0, s, rb);
      }
      step_fused = true;
    }
    if (side) {
      (void)hipEventRecord(side->bptt_done[l], s);
      (void)hipStreamWaitEvent(ss, side->bptt_done[l], 0);
    }
    const int64_t Kr = (int64_t)(Tn - 1) * B;
    float* part_ih = part_side;
    float* part_hh = (float*)((char*)part_side + lo.skp_hh[l]);
    float* part_dx = (float*)((char*)part + lo.skp_dx[l]);
    float* dst_dx = (dY == (const float*)(ws + lo.DYa)) ? (float*)(ws + lo.DYb) : (float*)(ws + lo.DYa);
    bool dw_done = false, dx_done = l == 0, db_done = false;
    // W_ih of both directions as the dX product's B operand, read as it lies
    // (k = gate row of direction d in segment d, n = input unit)
    Opnd Bw = opnd(W + lo.Wih[l][0], Dl, Dl, 8 * H);
    Bw.seg = 4 * H;
    Bw.segstride = lo.Wih[l][1] - lo.Wih[l][0];
    if constexpr (lp) {
      if (lo.write_dat) {
        // A: da^T (frame-contiguous, written by the BPTT kernel); B: the layer
        // input X_l and output h_l as they lie (frame rows).
        // dW_ih[d] = da_d^T X_l  (4H x D_l, reduction over all frames);
        // dW_hh[d] = sum_t da_d[t]^T h_d[t_prev] (the forward direction pairs
        // frame t with t-1, the reverse one t with t+1);
        // without the side stream also dX_l (below), all in one launch
        T* DAT = DATl;
        F32Job g[3];
        g[0] = F32Job{opnd(DAT, M, (int)M, 4 * H, 4 * H * M), opnd(Xl, Dpl, Dpl, M), 4 * H, Dl, M, 2,
                      lo.sp_dWih[l], grad + lo.Wih[l][0], Dl, lo.Wih[l][1] - lo.Wih[l][0], part_ih};
        g[1] = F32Job{opnd(DAT + B, M, (int)Kr, 4 * H, 4 * H * M - B), opnd(Yl, 2 * H, H, Kr, (int64_t)B * 2 * H + H),
                      4 * H, H, Kr, 2, lo.sp_dWhh[l], grad + lo.Whh[l][0], H, lo.Whh[l][1] - lo.Whh[l][0], part_hh};
        // the whole k range per tile (the deferred launch has tiles enough;
        // the side-stream path does the same, so that both sum alike)
        g[0].splits = g[1].splits = 1;
        int ng = 2;
        if (defer) {
          deferred[nd++] = g[0];
          deferred[nd++] = g[1];
          ng = 0;
        }
        const bool dx_here = !side && l > 0;
        if (dx_here)
          g[ng++] = F32Job{opnd(DA, 8 * H, 8 * H, M), Bw, M, Dl, 8 * H, 1, lo.sp_dX[l], dst_dx, Dl, 0, part_dx};
        // db_ih = db_hh = sum over frames of da, from the BPTT kernel's
        // per-row-block partials, in the same reduction launch
        const int dbp_rows = done ? (int)cdiv(B, persist_rows_per_workgroup(H, B)) : Tn * (int)cdiv(B, 16);
        const ColSumJob cs{DBPl, dbp_rows, 2, 4 * H, 8 * H, 4 * H,
                           grad + lo.bih[l][0], grad + lo.bhh[l][0], lo.bih[l][1] - lo.bih[l][0]};
        const bool with_db = step_fused && colsum_job_ok(cs);
        if (dy_parts && with_db) {
          // the bias sums wait for the last BPTT; dX (if any) keeps its
          // partials for the next BPTT when it is split
          bias_jobs[nbias++] = cs;
          db_done = true;
          ReduceGroup held;
          if (ng == 0 || gemm_f32_group<true, false>("gemm_bwd_group", ss, ng, g, nullptr, &held)) {
            if (ng > 0 && held.n == 1) pending_dy = held;
            else if (ng > 0) reduce_group_launch(ss, held);
          } else {
            for (int i = 0; i < ng; ++i)
              gemm_f32<T, true, false, V, V>(i == ng - 1 && dx_here ? "gemm_dx" : (i == 0 ? "gemm_dwih" : "gemm_dwhh"),
                                             ss, g[i].A, g[i].B, g[i].M, g[i].N, g[i].K, g[i].batches, g[i].splits,
                                             g[i].dst, g[i].ld, g[i].dst_zstride, g[i].part);
          }
        } else if (ng == 0) {
          // (layer 0, weight gradients deferred: the bias sums alone, by the
          // same reduction)
          db_done = with_db && colsum_job_launch("splitk_reduce_group", ss, cs);
        } else if (gemm_f32_group<true, false>("gemm_bwd_group", ss, ng, g, with_db ? &cs : nullptr)) {
          db_done = with_db;
        } else {
          for (int i = 0; i < ng; ++i)
            gemm_f32<T, true, false, V, V>(i == ng - 1 && dx_here ? "gemm_dx" : (i == 0 ? "gemm_dwih" : "gemm_dwhh"),
                                           ss, g[i].A, g[i].B, g[i].M, g[i].N, g[i].K, g[i].batches, g[i].splits,
                                           g[i].dst, g[i].ld, g[i].dst_zstride, g[i].part);
        }
        dx_done = dx_done || dx_here;
        dw_done = true;
      }
    }
    if (!dw_done) {
      // dW_ih[d] = da_d^T X_l  (4H x D_l, reduction over all frames)
      const Opnd A = opnd(DA, 8 * H, 4 * H, M, 4 * H);
      const Opnd Bx = opnd(Xl, Dpl, Dpl, M);
      gemm_f32<T, false, false, V, V>("gemm_dwih", s, A, Bx, 4 * H, Dl, M, 2, lo.sp_dWih[l],
                                      grad + lo.Wih[l][0], Dl, lo.Wih[l][1] - lo.Wih[l][0], part_ih);
      // dW_hh[d] = sum_t da_d[t]^T h_d[t_prev]: frames shifted by one step, the
      // forward direction pairing t with t-1 and the reverse direction t with t+1
      const Opnd Ad = opnd(DA + (int64_t)B * 8 * H, 8 * H, 4 * H, Kr, 4 * H - (int64_t)B * 8 * H);
      const Opnd Bh = opnd(Yl, 2 * H, H, Kr, (int64_t)B * 2 * H + H);
      gemm_f32<T, false, false, V, V>("gemm_dwhh", s, Ad, Bh, 4 * H, H, Kr, 2, lo.sp_dWhh[l],
                                      grad + lo.Whh[l][0], H, lo.Whh[l][1] - lo.Whh[l][0], part_hh);
    }
    // db_ih = db_hh = sum over frames of da (unless the reduction above did it)
    if (!db_done) {
      if (step_fused)
        colsum_parts("colsum_db", ss, DBPl,
                     done ? (int)cdiv(B, persist_rows_per_workgroup(H, B)) : Tn * (int)cdiv(B, 16), 8 * H, 4 * H,
                     lo.bih[l][1] - lo.bih[l][0], grad + lo.bih[l][0], grad + lo.bhh[l][0]);
      else
        colsum<T>("colsum_db", s, DA, M, 8 * H, 8 * H, csp, 4 * H, lo.bih[l][1] - lo.bih[l][0],
                  grad + lo.bih[l][0], grad + lo.bhh[l][0]);
    }
    if (side) (void)hipEventRecord(side->dw_done[l], ss);
    // dX_l = sum_d da_d W_ih[d]  (the gradient reaching the layer below)
    if (!dx_done) {
      const Opnd A = opnd(DA, 8 * H, 8 * H, M);
      gemm_f32<T, true, false, V, V>("gemm_dx", s, A, Bw, M, Dl, 8 * H, 1, lo.sp_dX[l], dst_dx, Dl, 0, part_dx);
    }
    if (l > 0) dY = dst_dx;
  }
  // the held bias sums of every layer, one reduction launch
  if (nbias > 0) {
    ReduceGroup rg;
    std::memset((void*)&rg, 0, sizeof rg);
    int blocks = 0;
    for (int i = 0; i < nbias; ++i) {
      if (rg.n == KC_MAX_GROUP) {
        reduce_group_launch(s, rg);
        std::memset((void*)&rg, 0, sizeof rg);
        blocks = 0;
      }
      rg.j[rg.n] = colsum_reduce_job(bias_jobs[i], blocks);
      blocks += (int)cdiv((int64_t)rg.j[rg.n++].count, 256);
    }
    reduce_group_launch(s, rg);
  }
  // the deferred weight gradients, KC_MAX_GROUP products per launch (all of
  // them for up to six layers: one launch, so that only its last round of
  // the chip is a partial one)
  for (int i0 = 0; i0 < nd; i0 += KC_MAX_GROUP) {
    const int n = std::min(KC_MAX_GROUP, nd - i0);
    if (!gemm_f32_group<true, false>("gemm_dw_group", s, n, deferred + i0)) {
      for (int i = i0; i < i0 + n; ++i) {
        const F32Job& j = deferred[i];
        gemm_f32<T, true, false, V, V>((i & 1) ? "gemm_dwhh" : "gemm_dwih", s, j.A, j.B, j.M, j.N, j.K, j.batches,
                                       1, j.dst, j.ld, j.dst_zstride, part);
      }
    }
  }
  if (side) (void)hipStreamWaitEvent(s, side->dw_done[0], 0);   // join before returning
  return blstm_check_launch("blstm_bwd");
}

extern "C" int blstm_recurrence_ok(const blstm_dims* dims, const void* act_ws, hipStream_t stream) {
  Layout lo;
  int rc = make_layout(dims, &lo);
  if (rc) return rc;
  if (!act_ws) return blstm_fail(BLSTM_EINVAL, "blstm_recurrence_ok: NULL act_ws");
  int gave_up = 0;
  int* status = (int*)((char*)act_ws + lo.SYNC);
  if (hipMemcpyAsync(&gave_up, status, sizeof(int), hipMemcpyDeviceToHost, stream) != hipSuccess ||
      hipStreamSynchronize(stream) != hipSuccess)
    return blstm_fail(BLSTM_EHIP, "blstm_recurrence_ok: %s", hipGetErrorString(hipGetLastError()));
  if (persist_status_reset(status, stream) != hipSuccess)
    return blstm_fail(BLSTM_EHIP, "blstm_recurrence_ok: %s", hipGetErrorString(hipGetLastError()));
  if (gave_up)
    return blstm_fail(BLSTM_EHIP,
                      "blstm_recurrence_ok: a recurrent exchange wait gave up since the last query (the workgroups "
                      "of a persistent launch were not all resident; set ADPSGD_BLSTM_COOPERATIVE=1 on a shared "
                      "device)");
  return BLSTM_OK;
}

extern "C" int blstm_fwd(const blstm_dims* dims, const float* theta, const void* theta_lp,
                         const float* x, void* act_ws, void* y_top, hipStream_t stream) {
  Layout lo;
  int rc = make_layout(dims, &lo);
  if (rc) return rc;
  if (!theta || !x || !act_ws || !y_top) return blstm_fail(BLSTM_EINVAL, "blstm_fwd: NULL pointer");
  if (lo.prec == BLSTM_BF16) {
    if (!theta_lp) return blstm_fail(BLSTM_EINVAL, "blstm_fwd: theta_lp is NULL (bf16)");
    return fwd_impl<bf16>(lo, theta, (const bf16*)theta_lp, x, (char*)act_ws, (bf16*)y_top, stream);
  }
  return fwd_impl<float>(lo, theta, theta, x, (char*)act_ws, (float*)y_top, stream);
}

extern "C" int blstm_bwd(const blstm_dims* dims, const float* theta, const void* theta_lp,
                         void* act_ws, const void* y_top, const float* dy_top, float* grad,
                         hipStream_t stream) {
  Layout lo;
  int rc = make_layout(dims, &lo);
  if (rc) return rc;
  if (!theta || !act_ws || !y_top || !dy_top || !grad)
    return blstm_fail(BLSTM_EINVAL, "blstm_bwd: NULL pointer");
  if (lo.prec == BLSTM_BF16) {
    if (!theta_lp) return blstm_fail(BLSTM_EINVAL, "blstm_bwd: theta_lp is NULL (bf16)");
    return bwd_impl<bf16>(lo, (const bf16*)theta_lp, (char*)act_ws, (const bf16*)y_top, dy_top, grad,
                          stream);
  }
  return bwd_impl<float>(lo, theta, (char*)act_ws, (const float*)y_top, dy_top, grad, stream);
}
