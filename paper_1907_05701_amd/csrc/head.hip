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

#include <cmath>

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
// written nor read back.  The bias gradients come from the second
// product's column-sum partials: db_s directly, and db_l = W_s^T db_s (the
// sum over frames of dz = ds W_s), so no pass reads ds or dz back for them.
//
// Exponentials on the hardware base-2 exponential: exp(x) = 2^(x log2 e),
// with the subtraction of the maximum (or log-sum-exp) and, for a positive
// loss scale, log2(scale) folded into one fused multiply-add per element.
// ---------------------------------------------------------------------------
#define LOG2E_F 1.4426950408889634f
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }
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
  int K, M;            // classes (product rows), frames (product columns)
  int nstrip, srows;
  template <int FM, int FN>
  __device__ __forceinline__ void apply(int, int, int64_t mw64, int64_t nw64, f32x4 (&acc)[FM][FN], int lane) const {
    if (mw64 >= K) return;
    const int mw = (int)mw64, nw = (int)nw64;
    const int strip = mw / srows;
    float bv[FM][4];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int k = mw + i * 16 + (lane >> 4) * 4 + r;
        bv[i][r] = k < K ? bias[k] : -INFINITY;
      }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          acc[i][j][r] += bv[i][r];   // the logit (the accumulators are not used after this)
          mx = fmaxf(mx, acc[i][j][r]);
        }
      float sm = 0.f;
      if (mx != -INFINITY) {
        const float nm = -mx * LOG2E_F;
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r) sm += exp2_hw(fmaf(acc[i][j][r], LOG2E_F, nm));
      }
      // the four lane groups hold the other classes of the same frame
      lse_pair(mx, sm, __shfl_xor(mx, 16), __shfl_xor(sm, 16));
      lse_pair(mx, sm, __shfl_xor(mx, 32), __shfl_xor(sm, 32));
      const int f = nw + j * 16 + (lane & 15);
      if ((lane >> 4) == 0 && f < M) stats[(int64_t)f * nstrip + strip] = make_float2(mx, sm);
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
  // the lane's strips lane, lane + 64, ... combined in that order; eight
  // loads in flight at a time
  constexpr int U = 8;
  for (int i0 = lane; i0 < nstrip; i0 += 64 * U) {
    float2 p[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (i0 + 64 * u < nstrip) p[u] = stats[m * nstrip + i0 + 64 * u];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (i0 + 64 * u < nstrip) lse_pair(mx, sm, p[u].x, p[u].y);
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
// frame loss at the label's class, and the column sums of ds over the
// workgroup's frames (db_s partials, one row per frame tile, summed in a
// fixed order).  Lane group g = lane / 16 holds classes 4g .. 4g+3 of each
// 16-class fragment; for a fragment pair (i, i+1) the groups g and g ^ 1
// swap halves so that each lane stores 8 consecutive classes (16 bytes):
// even groups classes 8(g/2) .. +7 of fragment i, odd groups those of i+1.
// Per element: one subtraction, one fused multiply-add, the exponential, a
// multiplication by the loss scale (by one when it is folded into the
// exponent) and the column-sum add; classes past K carry a bias of -inf and frames past M
// a log-sum-exp of +inf, so both give exact zeros without a test.  The label
// (at most one class of a frame) is handled in a branch that a lane takes
// only for the fragment holding it.
struct EpiSoftmaxDs {
  static constexpr bool workgroup = true;
  const float* bias;      // b_s [K]
  const float* lse;       // [M]
  const int32_t* labels;  // [M]
  bf16* ds;               // [M][Kp]
  float* rowloss;         // [M]: lse - s[label] (frames with an out-of-range label hold NaN already)
  float* dbp;             // [frame tiles][K] column-sum partials (one row per workgroup's frames)
  float scale;
  float l2s;              // log2(scale) folded into the exponent (scale > 0 and normal), else NaN
  int K, Kp, M;
  template <int BM, int WM, int WN, int FM, int FN>
  __device__ __forceinline__ void apply_wg(int64_t mw64, int64_t nw64, f32x4 (&acc)[FM][FN], int lane, char* lds,
                                           int tn) const {
    static_assert(FM % 2 == 0, "fragment pairs");
    const int mw = (int)mw64, nw = (int)nw64;
    const int g = lane >> 4;
    const bool fold = l2s == l2s;
    const float mul = fold ? 1.0f : scale;   // v * 1 is v
    // bias * log2(e), -inf past K; every load is issued before the first
    // use (a load under the k < K test would be waited for one at a time)
    float bl[FM][4];
    const float* bp = bias + mw + g * 4;
    if (mw + FM * 16 <= K) {
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) bl[i][r] = bp[i * 16 + r];
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) bl[i][r] *= LOG2E_F;
    } else {
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) bl[i][r] = bias[min(mw + i * 16 + g * 4 + r, K - 1)];
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) bl[i][r] = mw + i * 16 + g * 4 + r < K ? bl[i][r] * LOG2E_F : -INFINITY;
    }
    float csum[FM][4];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) csum[i][r] = 0.f;
    float Lj[FN];
    int labj[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int f = nw + j * 16 + (lane & 15);
      Lj[j] = f < M ? lse[f] : INFINITY;
      labj[j] = f < M ? labels[f] : -1;
    }
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int f = nw + j * 16 + (lane & 15);
      const bool fok = f < M;
      const float L = Lj[j];
      const int lab = labj[j] < K ? labj[j] : -1;
      const float Lc = fold ? fmaf(L, LOG2E_F, -l2s) : L * LOG2E_F;
      uint2 pk[FM];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          v[r] = exp2_hw(fmaf(acc[i][j][r], LOG2E_F, bl[i][r] - Lc));
          v[r] *= mul;
        }
        const int kb = mw + i * 16 + g * 4;
        if ((unsigned)(lab - kb) < 4u) {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (lab - kb == r) {
              rowloss[f] = L - (acc[i][j][r] + bias[lab]);
              v[r] -= scale;
            }
        }
        bf16 e[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          csum[i][r] += v[r];
          e[r] = (bf16)v[r];
        }
        pk[i] = *(const uint2*)e;
      }
      bf16* drow = ds + (int64_t)f * Kp;
#pragma unroll
      for (int i = 0; i < FM; i += 2) {
        const uint2 send = (g & 1) ? pk[i] : pk[i + 1];
        const uint2 got = make_uint2((uint32_t)__shfl_xor((int)send.x, 16), (uint32_t)__shfl_xor((int)send.y, 16));
        const uint4 v = (g & 1) ? make_uint4(got.x, got.y, pk[i + 1].x, pk[i + 1].y)
                                : make_uint4(pk[i].x, pk[i].y, got.x, got.y);
        const int k0 = mw + (i + (g & 1)) * 16 + (g >> 1) * 8;
        if (fok && k0 < Kp) *(uint4*)(drow + k0) = v;
      }
    }
    // column sums over the wave's frames: across the 16 lanes of a group
    // with DPP adds (lane ^ 1, lane ^ 2 within quads, then the half-row and
    // row mirrors), a fixed order that leaves the sum in every lane; then
    // over the workgroup's frame waves in order through LDS (free once
    // every wave has left the product loop), one partial row per workgroup
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) csum[i][r] = row16_sum(csum[i][r]);
    const int wid = threadIdx.x >> 6, wm = wid % WM, wn = wid / WM;
    float* red = (float*)lds;   // [WN][BM]
    __syncthreads();
    if ((lane & 15) == 0) {
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[wn * BM + wm * (BM / WM) + i * 16 + g * 4 + r] = csum[i][r];
    }
    __syncthreads();
    const int m0 = mw - wm * (BM / WM);
    for (int c = threadIdx.x; c < BM; c += WM * WN * 64) {
      float sum = 0.f;
#pragma unroll
      for (int q = 0; q < WN; ++q) sum += red[q * BM + c];
      if (m0 + c < K) dbp[(int64_t)tn * K + m0 + c] = sum;
    }
  }

};

// ---------------------------------------------------------------------------
// The two logits products with the class block held on chip (bf16, P <= 256).
// One workgroup of 8 waves per block of LB = 128 classes: each wave keeps
// the W_s rows of its 32 classes in registers for the whole launch, and all
// M frames of z pass through an LDS ring in chunks of LF = 64 frames, so W_s
// is read once per workgroup and z once per workgroup from L2 (instead of
// both operands once per output tile), and the 250 workgroups of the full
// model each take one CU for the whole launch.  Wave w = (wm, wn) =
// (w % 4, w / 4) computes classes 32 wm .. +31 of the block for frames
// 32 wn .. +31 of each chunk; a lane holds four consecutive classes of one
// frame, as in the blocked products above.  The bias is the accumulator
// input of the first k-step, so the products give the logits themselves.
//   PASS 1: per (frame, block) maximum and sum of exp over the block's
//     classes (the block is the strip of the statistics, combined per frame
//     by logit_lse): the maximum over the wave's 32 classes, then the sum of
//     exp(s - maximum) (lanes exchange by permlane swaps; max and + are
//     commutative, so all four lane groups hold the same result), then over
//     the four class waves in order through LDS (one chunk later).
//   PASS 2: ds = scale (softmax - onehot) in bf16, the frame loss at the
//     label, and db_s of the block's classes over all frames (per lane over
//     its frames in chunk order, then over the 16 frame lanes (DPP, fixed
//     order) and the two frame waves in order), written as the gradient of
//     b_s; then the block's share of db_l = W_s^T db_s from the W_s rows in
//     registers (the shares are summed over blocks by head_bias_final).
// Software pipeline: iteration j multiplies chunk j + 1 while it runs the
// epilogue of chunk j, so the MFMA and the vector ALU work overlap within
// a wave.  The ring (LSL slots, direct-to-LDS loads; with pass 2 also the
// chunk's log-sum-exp values and labels, read into registers with the
// chunk's fragments) runs three chunks ahead: chunk j + 4 is requested right
// after the barrier that ends every wave's use of chunk j, into its slot.
// The buffer resources advance by the chunk (scalar arithmetic; their range
// ends at frame M, so rows past M read as zeros and their stores are
// dropped) and the per-lane offsets stay fixed.  Every wave issues the same
// number of memory instructions per chunk (a dummy load into a scratch area
// where a wave has no row; stores whose unused lanes carry an out-of-range
// offset), so the wait for a chunk is an exact vmcnt bound: what the wave
// issued after that chunk's loads.
// LDS ring rows: frames in pairs of 1 KB blocks at a pitch of 1056 bytes,
// the second row of a pair with its 16-byte chunks swapped in pairs
// (chunk c in slot c ^ 1): the 8 (16) lanes of one 16-byte read phase hit
// distinct banks, and a fragment's address moves by a constant per k-step.
// ---------------------------------------------------------------------------
#define LB 128
#define LF 64
#define LSL 4
#define LKS 8                        // 32-deep k-steps (P <= 256)
#define LBLK 1056                    // LDS bytes per pair of z rows
#define LSLOT (LF / 2 * LBLK)        // LDS bytes per ring slot
struct LogitsArgs {
  const bf16* Ws;      // [K][P]
  const bf16* Z;       // [M][P]
  const float* bias;   // b_s [K]
  int K, M, P;
  float2* stats;       // PASS 1: [M][nstrip] (nstrip = blocks)
  int nstrip;
  const float* lse;    // PASS 2: [M]
  const int32_t* labels;
  bf16* ds;            // [M][Kp]
  int Kp;
  float* rowloss;      // [M]
  float* dbs;          // [K]: db_s (the gradient of b_s)
  float* share;        // [blocks][P]: W_s^T db_s over each block's classes
  float scale, l2s;    // as in EpiSoftmaxDs
};
static constexpr size_t LG_RING = (size_t)LSL * LSLOT;
static constexpr size_t LG_LSE = LG_RING, LG_LAB = LG_LSE + LSL * LF * 4, LG_EX = LG_LAB + LSL * LF * 4;
static constexpr size_t LG_SCRATCH = LG_EX + 2 * 4 * LF * 8;
static constexpr size_t LG_SIMD = LG_SCRATCH + 256;   // 4 counters
static constexpr size_t LG_LDS = LG_SIMD + 16;
static_assert(LG_LDS <= 160 * 1024, "LDS of one CU");

typedef uint32_t v2u32 __attribute__((ext_vector_type(2)));
typedef uint32_t v4u32 __attribute__((ext_vector_type(4)));

// LDS write and reads of the statistics exchange as inline asm: the
// compiler's own forms are made to wait for every direct-to-LDS load in
// flight (it cannot tell which LDS bytes they write), which would drain the
// ring; the exchange area is disjoint from every load's destination.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}
__device__ __forceinline__ void lds_write_f2(float2* p, float x, float y) {
  const v2u32 v{__float_as_uint(x), __float_as_uint(y)};
  asm volatile("ds_write_b64 %0, %1" ::"v"(lds_addr(p)), "v"(v) : "memory");
}
// the four values p[0], p[LF], p[2 LF], p[3 LF] (512 bytes apart)
__device__ __forceinline__ void lds_read_f2x4(const float2* p, v2u32 (&v)[4]) {
  asm volatile(
      "ds_read_b64 %0, %4\n\tds_read_b64 %1, %4 offset:512\n\tds_read_b64 %2, %4 offset:1024\n\t"
      "ds_read_b64 %3, %4 offset:1536\n\ts_waitcnt lgkmcnt(0)"
      : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3])
      : "v"(lds_addr(p))
      : "memory");
}

__device__ __forceinline__ void dma4(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, void* lds_wave_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)lds_wave_base, 4, byte_off, 0, 0, 0);
}
// buffer resource over rows [0, rows) of rowbytes bytes from base (none
// when rows <= 0; the caller keeps rows * rowbytes below 2^31 - 16)
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_rows(const void* base, int rows, int rowbytes) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, max(rows, 0) * rowbytes, 0x00020000);
}
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
// two floats to a bf16 pair (round to nearest even), x in the low half
__device__ __forceinline__ uint32_t pack_bf16x2(float x, float y) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{x, y}, bf16x2));
}
// x and the same register of lane ^ 16 (^ 32), in an order that depends on
// the lane: for commutative combinations only
__device__ __forceinline__ v2u32 pair16(float x) {
  return __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
}
__device__ __forceinline__ v2u32 pair32(float x) {
  return __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
}
// maxima as plain v_max instructions: the compiler's fmaxf first quiets
// signalling NaNs of operands it cannot prove canonical (every MFMA result
// and permlane output here), one more instruction per operand; a NaN logit
// still reaches the sums (and the loss) through the exponentials
__device__ __forceinline__ float vmax(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ __forceinline__ float vmax3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}
__device__ __forceinline__ float max16x32(float x) {
  v2u32 p = pair16(x);
  x = vmax(__uint_as_float(p[0]), __uint_as_float(p[1]));
  p = pair32(x);
  return vmax(__uint_as_float(p[0]), __uint_as_float(p[1]));
}
__device__ __forceinline__ float sum16x32(float x) {
  v2u32 p = pair16(x);
  x = __uint_as_float(p[0]) + __uint_as_float(p[1]);
  p = pair32(x);
  return __uint_as_float(p[0]) + __uint_as_float(p[1]);
}

// s_getreg operand: HW_ID (register 4), bits 4-5 (the SIMD)
#define HWREG_HW_ID_SIMD ((1 << 11) | (4 << 6) | 4)

template <int PASS, bool FOLD>
__global__ __launch_bounds__(512) void logits_block_kernel(const LogitsArgs a) {
  extern __shared__ __attribute__((aligned(1024))) char lds[];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = w & 3, wn = w >> 2;
  const int fr = lane & 15, fc = lane >> 4;
  const int K = a.K, M = a.M, P = a.P;
  const int c0 = blockIdx.x * LB;
  const int cl = c0 + 32 * wm + 4 * fc;   // the lane's first class (+16 i + r)
  const int nch = (M + LF - 1) / LF;
  constexpr int NLD = PASS == 2 ? 5 : 4;  // loads per wave and chunk
  constexpr int NST = PASS == 2 ? 4 : 1;  // stores per wave and chunk
  // the waves that share a SIMD take the product and the epilogue of a
  // step in alternating orders, so that one's MFMAs run beside the other's
  // vector ALU work: rank among the workgroup's waves on this SIMD (SIMD
  // from the wave's hardware id), by an LDS counter per SIMD.  Only the
  // timing depends on it.
  bool product_first;
  {
    int* cnt = (int*)(lds + LG_SIMD);
    if (tid < 4) cnt[tid] = 0;
    __syncthreads();
    const int simd = (__builtin_amdgcn_s_getreg(HWREG_HW_ID_SIMD) & 3);
    const int rank = __builtin_amdgcn_readfirstlane(lane == 0 ? atomicAdd(&cnt[simd], 1) : 0);
    product_first = (rank & 1) == 0;
  }
  bf16x8 af[2][LKS];   // W_s rows of the wave's classes (loaded after the ring's first chunks)
  f32x4 bv[2];         // their biases: the first k-step's accumulator input
  // ring loads: instruction q of wave w fills rows 2 b, 2 b + 1 of the
  // chunk (b = 8 q + w); lane (parity p = lane / 32, slot s = lane % 32)
  // reads chunk s ^ p of its row
  uint32_t zoff[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int p = lane >> 5, row = 2 * (q * 8 + w) + p, c = (lane & 31) ^ p;
    zoff[q] = c * 8 < P ? (uint32_t)((row * P + c * 8) * 2) : DMA_OFF_NONE;
  }
  auto issue = [&](int j) {
    const int f0 = j * LF, left = M - f0;
    char* st = lds + (j % LSL) * LSLOT;
    const __amdgpu_buffer_rsrc_t rz = rsrc_rows(a.Z + (int64_t)f0 * P, left, P * 2);
#pragma unroll
    for (int q = 0; q < 4; ++q) dma16(rz, zoff[q], st + (q * 8 + w) * LBLK);
    if constexpr (PASS == 2) {
      if (w == 0) dma4(rsrc_rows(a.lse + f0, left, 4), lane * 4, lds + LG_LSE + (j % LSL) * LF * 4);
      else if (w == 1) dma4(rsrc_rows(a.labels + f0, left, 4), lane * 4, lds + LG_LAB + (j % LSL) * LF * 4);
      else dma4(rz, DMA_OFF_NONE, lds + LG_SCRATCH);
    }
  };
  // fragment reads: row 32 wn + 16 jn + fr of the chunk, 16-byte chunk
  // 4 ks + fc; jn = 1 is 8 blocks further, ks 64 bytes
  const int rrow = 32 * wn + fr;
  const uint32_t rbase = (rrow >> 1) * LBLK + (rrow & 1) * 512 + ((fc ^ (rrow & 1)) * 16);
  auto product = [&](int j, f32x4 (&o)[2][2]) {
    const char* st = lds + (j % LSL) * LSLOT + rbase;
#pragma unroll
    for (int ks = 0; ks < LKS; ++ks) {
      bf16x8 b[2];
#pragma unroll
      for (int jn = 0; jn < 2; ++jn) b[jn] = *(const bf16x8*)(st + jn * 8 * LBLK + ks * 64);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jn = 0; jn < 2; ++jn) o[i][jn] = Mfma<bf16>::mma(af[i][ks], b[jn], ks == 0 ? bv[i] : o[i][jn]);
    }
  };
  // the frames' log-sum-exp and labels (+inf and -1 past M)
  auto frame_data = [&](int j, float (&L)[2], int (&lab)[2]) {
    const float* sl = (const float*)(lds + LG_LSE + (j % LSL) * LF * 4);
    const int32_t* sb = (const int32_t*)(lds + LG_LAB + (j % LSL) * LF * 4);
#pragma unroll
    for (int jn = 0; jn < 2; ++jn) {
      const int fl = 32 * wn + 16 * jn + fr;
      const bool fok = j * LF + fl < M;
      L[jn] = fok ? sl[fl] : INFINITY;
      const int lb = sb[fl];
      lab[jn] = fok && lb < K ? lb : -1;
    }
  };

  float2* ex = (float2*)(lds + LG_EX);   // [2 chunks][4 class waves][LF frames]
  // PASS 1: combine chunk j's four class-wave statistics (wave 0) and store
  // them; one store instruction in every wave (none valid for j < 0)
  auto combine = [&](int j) {
    float2 v = make_float2(0.f, 0.f);
    if (w == 0) {
      // maximum of the four, then the sums scaled to it in wave order (a
      // wave whose classes are all past K holds (-inf, 0) and adds zero)
      v2u32 e4[4];
      lds_read_f2x4(ex + (j & 1) * 4 * LF + lane, e4);
      const float m = vmax(vmax3(__uint_as_float(e4[0].x), __uint_as_float(e4[1].x), __uint_as_float(e4[2].x)),
                           __uint_as_float(e4[3].x));
      const float nm = m == -INFINITY ? 0.f : -m * LOG2E_F;
      float sm = 0.f;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        sm = fmaf(__uint_as_float(e4[q].y), exp2_hw(fmaf(__uint_as_float(e4[q].x), LOG2E_F, nm)), sm);
      v = make_float2(m, sm);
    }
    const int f0 = j * LF;
    const __amdgpu_buffer_rsrc_t rs = rsrc_rows(a.stats + (int64_t)f0 * a.nstrip, M - f0, a.nstrip * 8);
    const uint32_t off = w == 0 && j >= 0 ? (uint32_t)((lane * a.nstrip + (int)blockIdx.x) * 8) : DMA_OFF_NONE;
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(v2u32, v), rs, (int)off, 0, 0);
  };
  // PASS 2 store offsets within a chunk: 8 consecutive classes per lane
  // (lane groups g and g ^ 1 swap halves: even groups classes 8 (g / 2) ..
  // of row tile 0, odd groups those of row tile 1)
  const int k0 = c0 + 32 * wm + (fc & 1) * 16 + (fc >> 1) * 8;
  uint32_t dsoff[2];
#pragma unroll
  for (int jn = 0; jn < 2; ++jn)
    dsoff[jn] = k0 < a.Kp ? (uint32_t)(((32 * wn + 16 * jn + fr) * a.Kp + k0) * 2) : DMA_OFF_NONE;
  float csum[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) csum[i][r] = 0.f;

  auto epilogue = [&](int j, const f32x4 (&acc)[2][2], const float (&L)[2], const int (&lab)[2]) {
    if constexpr (PASS == 1) {
#pragma unroll
      for (int jn = 0; jn < 2; ++jn) {
        float mx = vmax3(vmax3(acc[0][jn][0], acc[0][jn][1], acc[0][jn][2]),
                         vmax3(acc[0][jn][3], acc[1][jn][0], acc[1][jn][1]), vmax(acc[1][jn][2], acc[1][jn][3]));
        mx = max16x32(mx);
        const float nm = mx == -INFINITY ? 0.f : -mx * LOG2E_F;
        float sm = exp2_hw(fmaf(acc[0][jn][0], LOG2E_F, nm));
#pragma unroll
        for (int e = 1; e < 8; ++e) sm += exp2_hw(fmaf(acc[e >> 2][jn][e & 3], LOG2E_F, nm));
        sm = sum16x32(sm);
        if (fc == 0) lds_write_f2(ex + ((j & 1) * 4 + wm) * LF + 32 * wn + 16 * jn + fr, mx, sm);
      }
    } else {
      const int f0 = j * LF;
      const __amdgpu_buffer_rsrc_t rd = rsrc_rows(a.ds + (int64_t)f0 * a.Kp, M - f0, a.Kp * 2);
      const __amdgpu_buffer_rsrc_t rr = rsrc_rows(a.rowloss + f0, M - f0, 4);
#pragma unroll
      for (int jn = 0; jn < 2; ++jn) {
        const float Lc = FOLD ? fmaf(L[jn], LOG2E_F, -a.l2s) : L[jn] * LOG2E_F;
        float lv = 0.f;
        bool has = false;
        uint32_t pk[2][2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          float v[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            v[r] = exp2_hw(fmaf(acc[i][jn][r], LOG2E_F, -Lc));
            if constexpr (!FOLD) v[r] *= a.scale;
          }
          const int kb = cl + 16 * i;
          if ((unsigned)(lab[jn] - kb) < 4u) {
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (lab[jn] - kb == r) {
                lv = L[jn] - acc[i][jn][r];
                has = true;
                v[r] -= a.scale;
              }
          }
#pragma unroll
          for (int r = 0; r < 4; ++r) csum[i][r] += v[r];
          pk[i][0] = pack_bf16x2(v[0], v[1]);
          pk[i][1] = pack_bf16x2(v[2], v[3]);
        }
        // odd lane groups take the even partner's row tile 1 classes, even
        // groups the odd partner's row tile 0 classes
        const v2u32 sx = __builtin_amdgcn_permlane16_swap(pk[0][0], pk[1][0], false, false);
        const v2u32 sy = __builtin_amdgcn_permlane16_swap(pk[0][1], pk[1][1], false, false);
        const v4u32 v4{sx[0], sy[0], sx[1], sy[1]};
        __builtin_amdgcn_raw_buffer_store_b128(v4, rd, (int)dsoff[jn], 0, 0);
        const uint32_t loff = has ? (uint32_t)((32 * wn + 16 * jn + fr) * 4) : DMA_OFF_NONE;
        __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(lv), rr, (int)loff, 0, 0);
      }
    }
  };

  // one iteration: wait for chunk j + 1, request chunk j + 4, pass 1's
  // combine of chunk j - 1, the product of chunk j + 1 and the epilogue of
  // chunk j
  // NST store instructions that write nothing (every offset out of range)
  auto no_stores = [&]() {
    const __amdgpu_buffer_rsrc_t rr = rsrc_rows(a.rowloss, 0, 4);
#pragma unroll
    for (int q = 0; q < NST; ++q) __builtin_amdgcn_raw_buffer_store_b32(0u, rr, (int)DMA_OFF_NONE, 0, 0);
  };
  auto step = [&](int j, const f32x4 (&cur)[2][2], f32x4 (&nxt)[2][2], const float (&Lc)[2], const int (&lc)[2],
                  float (&Ln)[2], int (&ln)[2]) {
    // issued after chunk j + 1's loads: chunks j + 2, j + 3 and three
    // chunks' stores (the prologue's empty ones standing in for chunks
    // before the first)
    kc_wait_vm<2 * NLD + 3 * NST>();
    if constexpr (PASS == 1) asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // exchange writes
    // chunk j + 1 in the ring; every wave is done with chunk j's slot (a
    // bare barrier: the fence of __syncthreads would wait for every load)
    kc_barrier();
    issue(j + 4);
    if constexpr (PASS == 1) combine(j - 1);
    if (product_first) {
      product(j + 1, nxt);
      if constexpr (PASS == 2) frame_data(j + 1, Ln, ln);
      epilogue(j, cur, Lc, lc);
    } else {
      epilogue(j, cur, Lc, lc);
      product(j + 1, nxt);
      if constexpr (PASS == 2) frame_data(j + 1, Ln, ln);
    }
  };

  f32x4 accA[2][2], accB[2][2];
  float LA[2], LB_[2];
  int labA[2], labB[2];
  // the ring's first chunks, then the fragments and biases (their latencies
  // overlap; the fragments' wait covers the chunks)
#pragma unroll
  for (int j = 0; j < LSL - 1; ++j) {
    no_stores();
    issue(j);
  }
  no_stores();
  // the wave's W_s rows (A operand): class c0 + 32 wm + 16 i + fr, k = 32 ks + 8 fc
  {
    const __amdgpu_buffer_rsrc_t rw = dma_rsrc(a.Ws);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int ks = 0; ks < LKS; ++ks) {
        const int row = c0 + 32 * wm + 16 * i + fr, k = 32 * ks + 8 * fc;
        const uint32_t off = row < K && k < P ? (uint32_t)(((int64_t)row * P + k) * 2) : DMA_OFF_NONE;
        af[i][ks] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rw, (int)off, 0, 0));
      }
  }
  // the lane's classes cl + 16 i + r: bias, -inf past K (clamped loads)
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) bv[i][r] = a.bias[min(cl + 16 * i + r, K - 1)];
  // fragments, biases and the first chunks in place (a wait the compiler
  // sees, so it adds none of its own for them in the chunk loop)
  __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (cl + 16 * i + r >= K) bv[i][r] = -INFINITY;

  kc_barrier();
  issue(LSL - 1);
  no_stores();
  product(0, accA);
  if constexpr (PASS == 2) frame_data(0, LA, labA);
  for (int j = 0; j < nch; j += 2) {
    step(j, accA, accB, LA, labA, LB_, labB);
    if (j + 1 < nch) step(j + 1, accB, accA, LB_, labB, LA, labA);
  }
  if constexpr (PASS == 1) {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    kc_barrier();
    combine(nch - 1);
  } else {
    // db_s: over the 16 frame lanes of each lane group, then the two frame
    // waves in order
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) csum[i][r] = row16_sum(csum[i][r]);
    float* red = (float*)(lds + LG_EX);   // [2 frame waves][LB]
    __syncthreads();
    if (fr == 0) {
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[wn * LB + 32 * wm + 16 * i + 4 * fc + r] = csum[i][r];
    }
    __syncthreads();
    float* dbl = red + 2 * LB;   // [LB]: the block's db_s, zero past K
    if (tid < LB) {
      const float v = red[tid] + red[LB + tid];
      if (c0 + tid < K) a.dbs[c0 + tid] = v;
      dbl[tid] = c0 + tid < K ? v : 0.f;
    }
    dma_wait_all();   // the ring's last (zero) loads have landed: slot 0 holds the share partials
    __syncthreads();
    // the block's share of db_l = W_s^T db_s, from the W_s fragments in
    // registers (the frame-half waves wn = 1 hold the same rows): per lane
    // its two classes, then the 16 class lanes of its lane group (DPP, fixed
    // order), then the four class waves in order
    float* sp = (float*)lds;   // [4 class waves][256 columns]
    if (wn == 0) {
      const float d0 = dbl[32 * wm + fr], d1 = dbl[32 * wm + 16 + fr];
#pragma unroll
      for (int ks = 0; ks < LKS; ++ks) {
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = row16_sum(fmaf(d1, (float)af[1][ks][e], d0 * (float)af[0][ks][e]));
        if (fr == 0) {
          *(float4*)&sp[wm * 256 + 32 * ks + 8 * fc] = make_float4(v[0], v[1], v[2], v[3]);
          *(float4*)&sp[wm * 256 + 32 * ks + 8 * fc + 4] = make_float4(v[4], v[5], v[6], v[7]);
        }
      }
    }
    __syncthreads();
    if (tid < P) a.share[(int64_t)blockIdx.x * P + tid] = ((sp[tid] + sp[256 + tid]) + sp[512 + tid]) + sp[768 + tid];
  }
  dma_wait_all();   // the ring's last (zero) loads land before the workgroup leaves its LDS
}

// Bias gradients and loss from the second product's outputs, one workgroup
// of 1024 threads per strip of 128 classes plus one for the loss:
//   db_s[k] = sum of the column-sum partial rows of class k (four row
//     quarters, each in row order, then added in quarter order);
//   share[strip][p] = sum over the strip's classes k of db_s[k] W_s[k][p]
//     (with W_s rows 16-byte aligned and P <= 256: 32 groups of 4 classes,
//     each thread 8 adjacent columns of one group by 16-byte loads, groups
//     added in order; otherwise four quarters of 32 classes, each in class
//     order, then in quarter order; the bf16 W_s that the dz product
//     multiplies); db_l = W_s^T db_s is the sum over frames of dz = ds W_s;
//   loss = scale * sum of the frame losses (1024 strided partial sums,
//     then a fixed tree).
// head_bias_final_kernel sums the shares in strip order (64 contiguous
// ranges, then in range order).  Every loop over memory is unrolled so that
// a thread has its loads in flight together.
#define HB_STRIP 128
__global__ __launch_bounds__(1024) void head_bias_kernel(const float* __restrict__ dbp, int nrows, int K, int P,
                                                         const bf16* __restrict__ ws, float* __restrict__ share,
                                                         float* __restrict__ grad_bs, const float* __restrict__ rowloss,
                                                         int M, float scale, float* __restrict__ loss, bool vec) {
  __shared__ float part[4][256];
  __shared__ float sdb[HB_STRIP];
  __shared__ float gsum[HB_STRIP / 4][256];   // vec: class-group sums per column
  const int tid = threadIdx.x;
  const int nstrip = (K + HB_STRIP - 1) / HB_STRIP;
  if ((int)blockIdx.x == nstrip) {
    float* sh = &part[0][0];
    float sum = 0.f;
    for (int f = tid; f < M; f += 1024) sum += rowloss[f];
    sh[tid] = sum;
    __syncthreads();
    for (int w = 512; w > 0; w >>= 1) {
      if (tid < w) sh[tid] += sh[tid + w];
      __syncthreads();
    }
    if (tid == 0) *loss = scale * sh[0];
    return;
  }
  const int k0 = blockIdx.x * HB_STRIP, kn = min(HB_STRIP, K - k0);
  {
    const int c = tid & (HB_STRIP - 1), q = tid / HB_STRIP;   // q < 8: row eighths
    const int per = (nrows + 7) / 8, r0 = q * per, r1 = min(nrows, r0 + per);
    float sum = 0.f;
    if (c < kn) {
#pragma unroll 8
      for (int r = r0; r < r1; ++r) sum += dbp[(int64_t)r * K + k0 + c];
    }
    part[q >> 1][(q & 1) * HB_STRIP + c] = sum;
  }
  __syncthreads();
  if (tid < HB_STRIP) {
    float sum = 0.f;
#pragma unroll
    for (int q = 0; q < 8; ++q) sum += part[q >> 1][(q & 1) * HB_STRIP + tid];
    sdb[tid] = sum;
    if (tid < kn) grad_bs[k0 + tid] = sum;
  }
  __syncthreads();
  if (vec) {
    // thread (class group cg of 4 classes, 8 adjacent columns from p8): four
    // 16-byte loads of W_s in flight together; the 32 group sums then added
    // in group order
    const int cg = tid >> 5, p8 = (tid & 31) * 8;
    float acc[8];
#pragma unroll
    for (int v = 0; v < 8; ++v) acc[v] = 0.f;
    if (p8 < P) {
      uint4 wv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = cg * 4 + i;
        wv[i] = c < kn ? *(const uint4*)(ws + (int64_t)(k0 + c) * P + p8) : make_uint4(0u, 0u, 0u, 0u);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float dv = cg * 4 + i < kn ? sdb[cg * 4 + i] : 0.f;
        const bf16* e = (const bf16*)&wv[i];
#pragma unroll
        for (int v = 0; v < 8; ++v) acc[v] += dv * (float)e[v];
      }
#pragma unroll
      for (int v = 0; v < 8; ++v) gsum[cg][p8 + v] = acc[v];
    }
    __syncthreads();
    if (tid < P) {
      float t = 0.f;
#pragma unroll 8
      for (int g = 0; g < HB_STRIP / 4; ++g) t += gsum[g][tid];
      share[(int64_t)blockIdx.x * P + tid] = t;
    }
    return;
  }
  const int q = tid >> 8, pl = tid & 255;
  const int c0 = q * (HB_STRIP / 4), c1 = min(kn, c0 + HB_STRIP / 4);
  for (int p0 = 0; p0 < P; p0 += 256) {
    const int p = p0 + pl;
    float acc = 0.f;
    if (p < P) {
#pragma unroll 16
      for (int c = c0; c < c1; ++c) acc += sdb[c] * (float)ws[(int64_t)(k0 + c) * P + p];
    }
    part[q][pl] = acc;
    __syncthreads();
    if (q == 0 && p < P) share[(int64_t)blockIdx.x * P + p] = ((part[0][pl] + part[1][pl]) + part[2][pl]) + part[3][pl];
    __syncthreads();
  }
}

// db_l[p] for 16 columns per workgroup: thread (g, column) sums the shares
// of strip range g (64 contiguous ranges) in order; the ranges are added in
// order.
// With rowloss given, one more workgroup (the last) writes
// loss = scale * sum of the frame losses (1024 strided partial sums, then a
// fixed tree), for launches without head_bias_kernel.
__global__ __launch_bounds__(1024) void head_bias_final_kernel(const float* __restrict__ share, int nstrip, int P,
                                                               float* __restrict__ grad_bl,
                                                               const float* __restrict__ rowloss, int M, float scale,
                                                               float* __restrict__ loss) {
  __shared__ float sh[64][16];
  if (rowloss && (int)blockIdx.x == (int)gridDim.x - 1) {
    float* t = &sh[0][0];
    const int tid = threadIdx.x;
    float sum = 0.f;
    for (int f = tid; f < M; f += 1024) sum += rowloss[f];
    t[tid] = sum;
    __syncthreads();
    for (int w = 512; w > 0; w >>= 1) {
      if (tid < w) t[tid] += t[tid + w];
      __syncthreads();
    }
    if (tid == 0) *loss = scale * t[0];
    return;
  }
  const int pl = threadIdx.x & 15, g = threadIdx.x >> 4;
  const int p = blockIdx.x * 16 + pl;
  const int per = (nstrip + 63) / 64, t0 = g * per, t1 = min(nstrip, t0 + per);
  float sum = 0.f;
  if (p < P) {
#pragma unroll 8
    for (int t = t0; t < t1; ++t) sum += share[(int64_t)t * P + p];
  }
  sh[g][pl] = sum;
  __syncthreads();
  if (threadIdx.x < 16 && p < P) {
    float tot = 0.f;
    for (int i = 0; i < 64; ++i) tot += sh[i][pl];
    grad_bl[p] = tot;
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

// Whether the logits products run as the class-block kernels
// (ADPSGD_LOGITS_BLOCK=0: the tiled products with their epilogues, for
// comparisons).
static bool logits_block() {
  const char* e = getenv("ADPSGD_LOGITS_BLOCK");
  return !(e && e[0] == '0');
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
    // frames per workgroup tile of the second product (one db_s partial row each)
    const int ftile = kc ? KcTile::BN : GemmCfgK32::BN;
    static_assert(KcTile::BM / KcTile::WM == GemmCfgK32::BM / GemmCfgK32::WM, "strip rows of the fallback tiles");
    static_assert(KcTile::BN == KcTileTall::BN, "frame columns of the kc tiles");
    float2* stats = (float2*)(hws + lo.LST);
    float* lse = (float*)(hws + lo.LSE);
    float* dbp = (float*)(hws + lo.LDB);
    const float l2s = (scale > 0.f && std::isnormal(scale)) ? std::log2(scale) : NAN;
    // the class-block kernels: every byte offset they form within 31 bits
    // (the buffer resource's range), 16-byte aligned rows
    const int nblk = (int)cdiv(K, LB);
    const bool blk = logits_block() && P % 8 == 0 && P <= 8 * LKS * 4 && M > 0 &&
                     (int64_t)rup(K, LB) * P * 2 < 0x7ffffff0 && M * P * 2 < 0x7ffffff0 &&
                     M * Kp * 2 < 0x7ffffff0 && M * nblk * 8 < 0x7ffffff0 && M * 4 < 0x7ffffff0 &&
                     ((uintptr_t)(W + lo.Ws) & 15) == 0 && ((uintptr_t)Z & 15) == 0 && ((uintptr_t)DS & 15) == 0;
    int nrows_dbp;
    if (blk) {
      static std::atomic<uint64_t> raised1{0}, raised2{0}, raised3{0};
      const bool fold = l2s == l2s;
      const void* k2 = fold ? (const void*)logits_block_kernel<2, true> : (const void*)logits_block_kernel<2, false>;
      kc_raise_lds_limit((const void*)logits_block_kernel<1, true>, LG_LDS, raised1);
      kc_raise_lds_limit(k2, LG_LDS, fold ? raised2 : raised3);
      static_assert(LB == HB_STRIP, "one share row per class block");
      LogitsArgs la{(const bf16*)(W + lo.Ws), (const bf16*)Z, theta + lo.bs, K, (int)M, P, stats, nblk, lse, labels,
                    (bf16*)DS, Kp, RL, grad + lo.bs, (float*)(hws + lo.DBLP), scale, l2s};
      BLSTM_LAUNCH("logits_blk", (logits_block_kernel<1, true>), dim3((unsigned)nblk), dim3(512), LG_LDS, s, la);
      BLSTM_LAUNCH("logit_lse", logit_lse_kernel, dim3((unsigned)cdiv(M, 4)), dim3(256), 0, s, stats, nblk, M, labels,
                   K, lse, RL);
      if (fold)
        BLSTM_LAUNCH("logits_ds_blk", (logits_block_kernel<2, true>), dim3((unsigned)nblk), dim3(512), LG_LDS, s, la);
      else
        BLSTM_LAUNCH("logits_ds_blk", (logits_block_kernel<2, false>), dim3((unsigned)nblk), dim3(512), LG_LDS, s, la);
      nrows_dbp = 1;
    } else {
      const int nstrip = (int)cdiv(K, srows);
      EpiLogitStats e1{theta + lo.bs, stats, K, (int)M, nstrip, srows};
      gemm_launch<T, true, true, V, V>("gemm_logits", s, Aw, Bz, K, M, P, 1, 1, e1);
      BLSTM_LAUNCH("logit_lse", logit_lse_kernel, dim3((unsigned)cdiv(M, 4)), dim3(256), 0, s, stats, nstrip, M,
                   labels, K, lse, RL);
      EpiSoftmaxDs e2{theta + lo.bs, lse, labels, (bf16*)DS, RL, dbp, scale, l2s, K, Kp, (int)M};
      gemm_launch<T, true, true, V, V>("gemm_logits_ds", s, Aw, Bz, K, M, P, 1, 1, e2);
      nrows_dbp = (int)cdiv(M, ftile);
    }
    // db_s, db_l and the loss
    const int nbs = (int)cdiv(K, HB_STRIP);
    float* share = (float*)(hws + lo.DBLP);
    // W_s rows read 8 columns at a time when they are 16-byte aligned
    const bool hb_vec = P % 8 == 0 && P <= 256 && ((uintptr_t)(W + lo.Ws) & 15) == 0;
    if (blk) {
      // the second class-block pass wrote db_s and the shares itself
      BLSTM_LAUNCH("head_bias_final", head_bias_final_kernel, dim3((unsigned)cdiv(P, 16) + 1), dim3(1024), 0, s,
                   share, nbs, P, grad + lo.bl, (const float*)RL, (int)M, scale, loss);
    } else {
      BLSTM_LAUNCH("head_bias", head_bias_kernel, dim3((unsigned)nbs + 1), dim3(1024), 0, s, dbp, nrows_dbp,
                   K, P, (const bf16*)(W + lo.Ws), share, grad + lo.bs, RL, (int)M, scale, loss, hb_vec);
      BLSTM_LAUNCH("head_bias_final", head_bias_final_kernel, dim3((unsigned)cdiv(P, 16)), dim3(1024), 0, s, share,
                   nbs, P, grad + lo.bl, (const float*)nullptr, 0, 0.f, (float*)nullptr);
    }
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
  // dW_s = ds^T z, and dz = ds W_s (float32 and a low-precision copy for
  // the next products); W_s [K][P] is the MN-contiguous operand as it lies
  // (the direct-to-LDS kernel reads it with transposing LDS reads; measured
  // faster than transposing W_s each step first).  bf16: the two products
  // in one launch (dW_s unsplit and stored directly, dz through its split-K
  // partials and reduction), each alone ending on a partial round of the chip
  const Opnd As = opnd(DS, Kp, Kp, M), Bs = opnd(Z, P, P, M);
  const Opnd Az = opnd(DS, Kp, Kp, M), Bz2 = opnd(W + lo.Ws, P, P, K);
  bool paired = false;
  if constexpr (lp) {
    if (lo.sp_dWs == 1 && lo.sp_dz > 1)
      paired = gemm_kc_pair_launch<false, false, true, false>(
          "gemm_dws_dz", s, As, Bs, K, P, M, 1, epi_store<float>(grad + lo.Ws, P, K, P, 0), Az, Bz2, M, P, K,
          lo.sp_dz, epi_store<float>(part, P, M, P, (int64_t)lo.sp_dz * M * P, M * P));
    if (paired) splitk_reduce_launch<T>(s, part, lo.sp_dz, 1, M, P, DZ, P, 0, DZT, P);
  }
  if (!paired) {
    gemm_f32<T, false, false, V, V>("gemm_dws", s, As, Bs, K, P, M, 1, lo.sp_dWs, grad + lo.Ws, P, 0, part);
    gemm_f32<T, true, false, V, V>("gemm_dz", s, Az, Bz2, M, P, K, 1, lo.sp_dz, DZ, P, 0, part, DZT, P);
  }
  // db_l = sum over frames of dz (bf16: already summed with db_s)
  if constexpr (!lp) colsum<float>("colsum_dbl", s, DZ, M, P, P, csp, P, 0, grad + lo.bl, nullptr);
  // dW_l = dz^T y, and dy = dz W_l (W_l [P][2H] MN-contiguous as it lies);
  // bf16: one launch for both (dW_l through its split-K partials, dy stored
  // directly)
  const Opnd Al = opnd(DZT, P, P, M), Bl = opnd(ytop, H2, H2, M);
  const Opnd Ay = opnd(DZT, P, P, M), By = opnd(W + lo.Wl, H2, H2, P);
  bool paired_l = false;
  if constexpr (lp) {
    if (lo.sp_dWl > 1 && lo.sp_dy == 1)
      paired_l = gemm_kc_pair_launch<false, false, true, false>(
          "gemm_dwl_dy", s, Al, Bl, P, H2, M, lo.sp_dWl,
          epi_store<float>(part, H2, P, H2, (int64_t)lo.sp_dWl * P * H2, P * H2), Ay, By, M, H2, P, 1,
          epi_store<float>(dytop, H2, M, H2, 0));
    if (paired_l) splitk_reduce_launch<T>(s, part, lo.sp_dWl, 1, P, H2, grad + lo.Wl, H2, 0, (T*)nullptr, 0);
  }
  if (!paired_l) {
    gemm_f32<T, false, false, V, V>("gemm_dwl", s, Al, Bl, P, H2, M, 1, lo.sp_dWl, grad + lo.Wl, H2, 0, part);
    gemm_f32<T, true, false, V, V>("gemm_dy", s, Ay, By, M, H2, P, 1, lo.sp_dy, dytop, H2, 0, part);
  }
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
