// Persistent recurrent kernels (bf16 operands): one launch runs all T steps
// of one layer, for both directions at once, and each workgroup keeps its
// slice of W_hh in registers for the whole chunk.
//
// Work split.  The batch is cut into slices of R = 16*MB rows; a group of
// NM = H/64 workgroups ("members") owns one (direction, slice) pair, and
// member m owns hidden units [64m, 64m + 64), i.e. 256 gate rows of W_hh
// (256 KB at H = 512: 128 VGPRs in each of the workgroup's 8 waves).  Eight
// members per group instead of sixteen halves the chip-wide exchange volume
// of every step; at the paper's B = 128 a launch takes 128 workgroups.
//   forward : wave (ub, kh) = (w % 4, w / 4) multiplies h_prev (all H units
//             of the slice, gathered from the members' published h) by the
//             four gates of the 16 units of block ub over the k half kh; the
//             two halves meet in LDS; the owning waves add the input
//             projection, apply the cell, publish h and write h, c and the
//             gate pre-activations for the backward.
//   backward: the gate derivatives of the member's 64 units (dc stays in
//             registers), then wave w multiplies the member's own da block
//             [R x 256 own gate rows] by its W_hh rows for the unit blocks
//             w, w+8, w+16, w+24: partial dh_rec for all H units, published;
//             each member sums the NM partials of its own units in member
//             order.
//
// Step-to-step exchange without barriers or cache maintenance.  The values
// one member needs from the others (h, or partial dh) are published in an
// exchange buffer as 8-byte words holding four 15-bit values and a 4-bit
// tag (see h4_tag), written and read with agent-scope relaxed atomic
// stores and loads.  Atomic accesses to one location are coherent across the
// whole GPU, so a reader that sees the expected tag in a word also sees that
// word's payload; readers poll the words they need (bounded; the status flag
// is set if a poll ever gives up).  Two slots alternate by step parity: a
// member overwrites a slot only after it has consumed the next step from
// every member, which those members produce only after they have consumed
// the slot's current contents.  The buffer is cleared once per forward or
// backward call, and the tag tells a word of the expected step from one of
// step n - 2 and from one left by either of the two previous launches of the
// call.  Every member of a group must be resident at once: the launch is
// plain when the occupancy query shows the whole grid fits on the device,
// cooperative otherwise (see launch_one).
#include <stdlib.h>
#include <string.h>

#include "common.hpp"
#include "lstm_persist.hpp"
#include "dma.hpp"

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

#define PU 64                 // hidden units per member
#define NTH 512               // threads per workgroup (8 waves)
#define KH_MAX 8              // forward: 32-deep k-steps per k half at H = 512
#define SPIN_LIMIT (1u << 18)
#define STAGE_BYTES (128 * 1024)   // W_hh staging buffer (half of a member's slice)

__device__ __forceinline__ uint64_t ll_load(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void ll_store64(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// the value of lane l ^ 1 (a DPP quad permutation, no LDS round trip)
__device__ __forceinline__ float lane_xor1(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, false));
}

// the value of lane l ^ 2
__device__ __forceinline__ uint32_t lane_xor2(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);
}

// Forward words: four bf16 h of one row
// (units 4i .. 4i+3, the first in the low half-word).  |h| = |o tanh(c)| <= 1,
// and a bf16 below 2 in magnitude has a zero top exponent bit (bit 14), so
// the four such bits carry a 4-bit tag: bit 0 always set (a cleared word
// never matches), bit 1 = bit 1 of the step number (a slot alternates
// between steps n and n - 2), bits 2-3 = the launch's sequence number in
// its call modulo 4 (a word can be left by one of the two launches before).
// Readers clear the four bits, so the exchanged values are exactly the bf16
// of h; a non-finite h (bit 14 set) reaches the other members clipped, while
// the layer output keeps it.
#define H4_TAG_BITS 0x4000400040004000ull
//
// BPTT words: four partial sums (rows 4i
// .. 4i+3 of one unit) in a 15-bit form that frees the same bits: the bf16
// of x * 2^-64 (so bf16 exponents 65 .. 190, i.e. 2^-62 <= |x| < 2^65, keep
// bit 14 clear and the 8-bit significand of the bf16 of x), magnitudes from
// 2^65 and non-finite values saturated to 2^64; tiny values become bf16
// subnormals.  Decoding multiplies by 2^64 (exact).
__device__ __forceinline__ uint32_t p15_encode(float x) {
  uint32_t b = __builtin_bit_cast(uint16_t, (bf16)(x * 0x1p-64f));
  if (b & 0x4000u) b = (b & 0x8000u) | 0x3F80u;
  return b;
}
__device__ __forceinline__ float p15_decode(uint32_t c) {
  return __builtin_bit_cast(float, (c & 0xBFFFu) << 16) * 0x1p64f;
}
__device__ __forceinline__ uint64_t h4_tag(uint32_t seq, int n) {
  const uint32_t t = 1u | (((uint32_t)n >> 1 & 1u) << 1) | ((seq & 3u) << 2);
  return ((uint64_t)(t & 1u) << 14) | ((uint64_t)(t >> 1 & 1u) << 30) | ((uint64_t)(t >> 2 & 1u) << 46) |
         ((uint64_t)(t >> 3 & 1u) << 62);
}

// two bf16 values in one dword, `lo` in the low half
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (bf16)lo) |
         ((uint32_t)__builtin_bit_cast(uint16_t, (bf16)hi) << 16);
}

// Polls the N words base[j * stride] (want: the expected tag bits; a word
// already holding `want` is never read) until every word carries the tag;
// gives up after SPIN_LIMIT polls, or at once when any wait anywhere has
// given up (the status flag is set), so every wave ends.
template <int N>
__device__ __forceinline__ void poll_words(uint64_t (&wv)[N], const uint64_t* base, int stride, uint64_t want,
                                           int* status) {
  for (unsigned it = 0;; ++it) {
    bool bad = false;
#pragma unroll
    for (int j = 0; j < N; ++j) bad |= (wv[j] & H4_TAG_BITS) != want;
    if (!bad) break;
    if (it > SPIN_LIMIT ||
        ((it & 63) == 63 && __hip_atomic_load(status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))) {
      __hip_atomic_store(status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      break;
    }
    __builtin_amdgcn_s_sleep(1);
#pragma unroll
    for (int j = 0; j < N; ++j)
      if ((wv[j] & H4_TAG_BITS) != want) wv[j] = ll_load(base + (int64_t)j * stride);
  }
}

// ---------------------------------------------------------------------------
// Forward.
// ---------------------------------------------------------------------------
template <int MB>
__global__ __launch_bounds__(NTH) void lstm_fwd_persist(const PersistArgs a) {
  extern __shared__ __attribute__((aligned(16))) char lds_raw[];
  constexpr int R = 16 * MB;
  // MB == 1: the k half 0 waves own the row block; MB > 1: half kh owns the
  // row blocks m with m % 2 == kh
  constexpr int MO = MB == 1 ? 1 : MB / 2;
  const int H = a.H, B = a.B, Tn = a.Tn;
  const int NG = 2 * a.NS;
  const int g = blockIdx.x % NG, mem = blockIdx.x / NG;
  const int d = g & 1, s = g >> 1;
  const int u0 = mem * PU;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int ub = w & 3, kh = w >> 2;
  const int KH = H / 64;   // 32-deep k-steps per k half
  const bool owner = MB > 1 || kh == 0;
  auto mblk = [&](int o) { return MB == 1 ? 0 : 2 * o + kh; };

  // W_hh fragments (B operand): gate q of unit u0 + ub*16 + lane%16, k-step
  // kh*KH + i, k = 8*(lane/16) .. +8 within it.  Staged by direct-to-LDS
  // loads one k half at a time: 256 local rows lr = q*64 + b*16 + u (gate q,
  // unit u0 + 16b + u), 512 bytes each (k past the half read as zeros), the
  // 16-byte chunk c of row lr in slot c ^ (lr & 15) so that the 16 rows of
  // one fragment read fall in distinct bank groups.
  bf16x8 bw[KH_MAX][4];
  {
    char* stg = lds_raw;
    const __amdgpu_buffer_rsrc_t rw = dma_rsrc(a.W + (d ? a.whh1 : a.whh0));
#pragma unroll
    for (int p = 0; p < 2; ++p) {
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int ins = q * 8 + w;                  // one instruction fills rows 2 ins, 2 ins + 1
        const int lr = ins * 2 + (lane >> 5);
        const int c = (lane & 31) ^ (lr & 15);      // chunk held by this lane's slot
        const int64_t grow = (int64_t)(lr >> 6) * H + u0 + ((lr >> 4) & 3) * 16 + (lr & 15);
        const bool ok = c * 8 < H / 2;
        dma16(rw, ok ? (uint32_t)((grow * H + p * (H / 2) + c * 8) * 2) : DMA_OFF_NONE, stg + ins * 1024);
      }
      dma_wait_all();
      __syncthreads();
      if (kh == p) {
#pragma unroll
        for (int i = 0; i < KH_MAX; ++i)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int lr = q * 64 + ub * 16 + (lane & 15);
            const int c = min(i, KH - 1) * 4 + (lane >> 4);
            bw[i][q] = *(const bf16x8*)(stg + lr * 512 + (c ^ (lr & 15)) * 16);
          }
      }
      __syncthreads();   // the next half (then the step buffers) reuse this LDS
    }
  }

  // LDS during the steps: gathered h [H/8][R + 1][8] (MFMA A layout), the
  // k-half partial sums, and (MB == 1) a step's c [16][64] (float), h
  // [16][64] and gate pre-activations [16][64][4] (bf16) for 16-byte stores
  bf16* hl = (bf16*)lds_raw;
  f32x4* red = (f32x4*)(lds_raw + (size_t)(H / 8) * (R + 1) * 16);
  float* sC = (float*)(red + 4 * MB * 4 * 64);
  bf16* sY = (bf16*)(sC + 16 * PU);
  bf16* sG = sY + 16 * PU;

  const int rend = a.b0 + a.rows;
  const int rowbase = a.b0 + s * R;
  const int unit = u0 + ub * 16 + (lane & 15);
  const int wpr = H / 4;   // exchange words per row
  const int64_t slot_stride = (int64_t)2 * a.rows * wpr;

  float creg[MO][4];
#pragma unroll
  for (int o = 0; o < MO; ++o)
#pragma unroll
    for (int r = 0; r < 4; ++r) creg[o][r] = 0.f;

  // input projection of a step (independent of h), loaded one step ahead so
  // that its latency hides behind the previous step's exchange
  bf16 gx[MO][4][4], gxn[MO][4][4];
  auto load_gx = [&](int tt) {
#pragma unroll
    for (int o = 0; o < MO; ++o)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rowbase + mblk(o) * 16 + (lane >> 4) * 4 + r;
        const bf16* p = a.Gx + ((int64_t)tt * B + (row < rend ? row : a.b0)) * 8 * H + (int64_t)d * 4 * H + unit;
#pragma unroll
        for (int q = 0; q < 4; ++q) gxn[o][r][q] = p[q * H];
      }
  };
  if (owner) load_gx(d ? Tn - 1 : 0);

  constexpr int WPT = (R * 128 + NTH - 1) / NTH;   // gathered words per thread (at H = 512)
  for (int tau = 0; tau < Tn; ++tau) {
    const int t = d ? Tn - 1 - tau : tau;
    if (owner) {
#pragma unroll
      for (int o = 0; o < MO; ++o)
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int q = 0; q < 4; ++q) gx[o][r][q] = gxn[o][r][q];
    }

    f32x4 acc[MB][4];
#pragma unroll
    for (int m = 0; m < MB; ++m)
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[m][q] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (tau > 0) {
      // h of the previous step (R rows x H/4 words of this slice, contiguous
      // in the exchange buffer), polled by all threads in whole cache lines
      // and staged in LDS in the MFMA A layout
      const int nwords = R * wpr;
      const uint64_t* src = a.X + ((tau - 1) & 1) * slot_stride + ((int64_t)d * a.rows + (rowbase - a.b0)) * wpr;
      const uint64_t want = h4_tag(a.seq, tau);
      uint64_t wv[WPT];
#pragma unroll
      for (int j = 0; j < WPT; ++j) {
        const int idx = tid + NTH * j;
        const bool ok = idx < nwords && rowbase + idx / wpr < rend;
        wv[j] = ok ? ll_load(src + idx) : want;
      }
      poll_words<WPT>(wv, src + tid, NTH, want, a.status);
#pragma unroll
      for (int j = 0; j < WPT; ++j) {
        const int idx = tid + NTH * j;
        if (idx >= nwords) break;
        const int row = idx / wpr, wc = idx % wpr;   // units 4 wc .. 4 wc + 3
        const bool ok = rowbase + row < rend;
        *(uint64_t*)&hl[((wc >> 1) * (R + 1) + row) * 8 + 4 * (wc & 1)] = ok ? (wv[j] & ~H4_TAG_BITS) : 0ull;
      }
      __syncthreads();
#pragma unroll
      for (int i = 0; i < KH_MAX; ++i) {
        if (i >= KH) break;
        const int kg = (kh * KH + i) * 4 + (lane >> 4);
#pragma unroll
        for (int m = 0; m < MB; ++m) {
          const bf16x8 af = *(const bf16x8*)&hl[(kg * (R + 1) + m * 16 + (lane & 15)) * 8];
#pragma unroll
          for (int q = 0; q < 4; ++q) acc[m][q] = Mfma<bf16>::mma(af, bw[i][q], acc[m][q]);
        }
      }
    }
    // the two k halves of each row block meet at its owner
#pragma unroll
    for (int m = 0; m < MB; ++m) {
      const bool mine = MB == 1 ? kh == 0 : (m & 1) == kh;
      if (!mine) {
#pragma unroll
        for (int q = 0; q < 4; ++q) red[((ub * MB + m) * 4 + q) * 64 + lane] = acc[m][q];
      }
    }
    __syncthreads();
    if (owner) {
      // cell math of all owned rows, then h published (the other members
      // wait for it), then the saved activations (only read after the launch)
      uint64_t* xo = a.X + (tau & 1) * slot_stride;
      float hv[MO][4], gv[MO][4][4];
#pragma unroll
      for (int o = 0; o < MO; ++o) {
        const int m = mblk(o);
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[m][q] += red[((ub * MB + m) * 4 + q) * 64 + lane];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
#pragma unroll
          for (int q = 0; q < 4; ++q) gv[o][r][q] = acc[m][q][r] + (float)gx[o][r][q];
          const float ig = sigmoidf_(gv[o][r][0]), fg = sigmoidf_(gv[o][r][1]);
          const float gg = tanhf_(gv[o][r][2]), og = sigmoidf_(gv[o][r][3]);
          const float c = fg * creg[o][r] + ig * gg;
          creg[o][r] = c;
          hv[o][r] = og * tanhf_(c);
        }
      }
      // every row's h before the first publish (the empty asm pins the
      // values here, so the compiler cannot sink their math past a publish)
#pragma unroll
      for (int o = 0; o < MO; ++o)
#pragma unroll
        for (int r = 0; r < 4; ++r) __asm__ volatile("" : "+v"(hv[o][r]));
#pragma unroll
      for (int o = 0; o < MO; ++o)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = rowbase + mblk(o) * 16 + (lane >> 4) * 4 + r;
          const float h_next_unit = lane_xor1(hv[o][r]);   // lanes of one row, units u and u^1
          // lane 4i stores units 4i .. 4i+3 (the pairs of lanes 4i and 4i+2)
          const uint32_t p2 = pack_bf16x2(hv[o][r], h_next_unit);
          const uint32_t p4 = lane_xor2(p2);
          if (row < rend && (lane & 3) == 0)
            ll_store64(xo + ((int64_t)d * a.rows + (row - a.b0)) * wpr + unit / 4,
                       ((((uint64_t)p4 << 32) | p2) & ~H4_TAG_BITS) | h4_tag(a.seq, tau + 1));
        }
      if constexpr (MB == 1) {
        // into LDS; the whole workgroup writes them out after the barrier
        const int ul = ub * 16 + (lane & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int rl = (lane >> 4) * 4 + r;
          sC[rl * PU + ul] = creg[0][r];
          sY[rl * PU + ul] = (bf16)hv[0][r];
          bf16x4 g4;
#pragma unroll
          for (int q = 0; q < 4; ++q) g4[q] = (bf16)gv[0][r][q];
          *(bf16x4*)&sG[(rl * PU + ul) * 4] = g4;
        }
      } else {
#pragma unroll
        for (int o = 0; o < MO; ++o)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int row = rowbase + mblk(o) * 16 + (lane >> 4) * 4 + r;
            if (row >= rend) continue;
            const int64_t fr = (int64_t)t * B + row;
            a.C[fr * 2 * H + (int64_t)d * H + unit] = creg[o][r];
            a.Y[fr * 2 * H + (int64_t)d * H + unit] = (bf16)hv[o][r];
            bf16x4 g4;
#pragma unroll
            for (int q = 0; q < 4; ++q) g4[q] = (bf16)gv[o][r][q];
            *(bf16x4*)(a.G + fr * 8 * H + (int64_t)d * 4 * H + (int64_t)unit * 4) = g4;
          }
      }
      if (tau + 1 < Tn) load_gx(d ? Tn - 2 - tau : tau + 1);
    }
    __syncthreads();   // h, the partial sums and the staged values are reused by the next step
    if constexpr (MB == 1) {
      // c, h and the gates of the step in 16-byte pieces: a row's 64 units
      // x 4 gates are 512 contiguous bytes (one piece per thread), its c 256
      // bytes (threads 0-255) and its h 128 bytes (threads 256-383).  The
      // next step's gather barrier comes before the LDS is rewritten.
      {
        const int rl = tid >> 5, c = tid & 31;
        const int row = rowbase + rl;
        if (row < rend)
          *(uint4*)(a.G + ((int64_t)t * B + row) * 8 * H + (int64_t)d * 4 * H + (int64_t)u0 * 4 + c * 8) =
              *(const uint4*)&sG[rl * PU * 4 + c * 8];
      }
      if (tid < 256) {
        const int rl = tid >> 4, c = tid & 15;
        const int row = rowbase + rl;
        if (row < rend)
          *(float4*)(a.C + ((int64_t)t * B + row) * 2 * H + (int64_t)d * H + u0 + c * 4) =
              *(const float4*)&sC[rl * PU + c * 4];
      } else if (tid < 384) {
        const int rl = (tid - 256) >> 3, c = (tid - 256) & 7;
        const int row = rowbase + rl;
        if (row < rend)
          *(uint4*)(a.Y + ((int64_t)t * B + row) * 2 * H + (int64_t)d * H + u0 + c * 8) =
              *(const uint4*)&sY[rl * PU + c * 8];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Backward (BPTT).
//
// dh_rec[b][j] = sum over all 4H gate rows g of da[b][g] W_hh[g][j].  Member
// m owns the 256 gate rows of its 64 units, so it computes the partial sums
// P_m = da[:, own rows] W_hh[own rows, :] for ALL H units from data it
// already holds (its own da in LDS, its W_hh rows in registers), publishes
// P_m as exchange words, and gathers for its own 64 units the partials of
// all members, summed in member order.  An exchange word holds one unit's
// partials for four adjacent rows; words are ordered (row quad, member,
// unit), so a member publishes whole cache lines and a reader takes 512
// contiguous bytes of each member.
// ---------------------------------------------------------------------------
template <int MB>
__global__ __launch_bounds__(NTH) void lstm_bwd_persist(const PersistArgs a) {
  extern __shared__ __attribute__((aligned(16))) char lds_raw[];
  constexpr int R = 16 * MB;            // rows of this member's slice
  constexpr int ITEMS = 2 * MB;         // (row, unit) cell items per thread
  constexpr bool SPLIT = MB == 1;       // two threads per gathered (row quad, unit): member halves
  const int H = a.H, B = a.B, Tn = a.Tn;
  const int NM = H / PU, NG = 2 * a.NS;
  const int g = blockIdx.x % NG, mem = blockIdx.x / NG;
  const int d = g & 1, s = g >> 1;
  const int u0 = mem * PU;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int NB = H / 16;                // unit blocks of the partial product

  // W_hh of the 256 own gate rows as the B operand: k = own row kk (gate
  // (kk>>4)&3, unit u0 + (kk>>6)*16 + (kk&15)), n = unit.  Wave w holds the
  // unit blocks nb = w + 8j (j < 4) for all 8 k-steps.  Staged from W_hh as
  // it lies, 128 own rows at a time, by direct-to-LDS loads ([kk][512
  // units], 1 KB rows, the 16-byte chunk c of row kk in slot c ^ wswz(kk);
  // units past H read as zeros), then each lane takes its fragments with
  // transposing LDS reads (ds_read_b64_tr_b16: in a 16-lane group lane r
  // addresses 4 consecutive units of k row r/4 and receives unit column r's
  // values over those 4 rows; two reads give the 8 consecutive k of the
  // MFMA B operand).  The swizzle spreads the 16 rows of one read over
  // distinct chunk pairs.
  bf16x8 bw[8][4];
  {
    auto wswz = [](int k) { return 2 * ((k & 3) | (((k >> 3) & 1) << 2)); };
    char* stg = lds_raw;
    const __amdgpu_buffer_rsrc_t rw = dma_rsrc(a.W + (d ? a.whh1 : a.whh0));
    const int gq = lane >> 4, r = lane & 15;
#pragma unroll
    for (int p = 0; p < 2; ++p) {
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int kl = q * 8 + w;   // one 1 KB row per load instruction
        const int kk = p * 128 + kl;
        const int c = lane ^ wswz(kl);
        const int64_t grow = (int64_t)((kk >> 4) & 3) * H + u0 + (kk >> 6) * 16 + (kk & 15);
        dma16(rw, c * 8 < H ? (uint32_t)((grow * H + c * 8) * 2) : DMA_OFF_NONE, stg + kl * 1024);
      }
      dma_wait_all();
      __syncthreads();
#pragma unroll
      for (int ksl = 0; ksl < 4; ++ksl)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int mn = (w + 8 * j) * 16 + 4 * (r & 3);
          bf16x4 h[2];
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const int k = ksl * 32 + 8 * gq + 4 * hh + (r >> 2);
            const char* pa = stg + k * 1024 + ((mn >> 3) ^ wswz(k)) * 16 + (mn & 7) * 2;
            h[hh] = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((__attribute__((address_space(3))) bf16x4*)(pa));
          }
          bw[4 * p + ksl][j] = bf16x8{h[0][0], h[0][1], h[0][2], h[0][3], h[1][0], h[1][1], h[1][2], h[1][3]};
        }
      __syncthreads();   // the next rows (then the step buffers) reuse this LDS
    }
  }

  // LDS during the steps: own da as the A operand [32 k groups][R + 1][8]
  // (k = own row), gathered dh_rec [2][R][64] (member halves when SPLIT)
  bf16* al = (bf16*)lds_raw;
  float* dhl = (float*)(al + (size_t)32 * (R + 1) * 8);

  const int rend = a.b0 + a.rows;
  const int rowbase = a.b0 + s * R;
  const int rquads = (a.rows + 3) / 4;             // row quads of this launch
  const int64_t slot_stride = (int64_t)2 * rquads * NM * H;
  // cell items: unit cu = tid % 64, rows tid/64 + 8*i
  const int cu = tid & 63;
  float dcreg[ITEMS];
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) dcreg[i] = 0.f;
  // da^T and bias partials: thread t takes own gate row t/2 and 8 of the 16
  // rows of each 16-row block; the bias partial of a block is summed over the
  // steps in order and written once
  const int dkk = tid >> 1, dh8 = (tid & 1) * 8;
  const int64_t dgrow = (int64_t)d * 4 * H + (int64_t)((dkk >> 4) & 3) * H + u0 + (dkk >> 6) * 16 + (dkk & 15);
  float dbacc[MB];
#pragma unroll
  for (int m = 0; m < MB; ++m) dbacc[m] = 0.f;

  // everything the cell derivative needs besides dh_rec: dy, the gate
  // pre-activations and c at t, c at the step's predecessor in forward time
  // (which is the next step's t).  Fetched one step ahead, right after the
  // previous step's gather, so that no gather waits for them; c at t is the
  // previous step's predecessor value.
  float dyn[ITEMS], cpn[ITEMS], cc[ITEMS];
  bf16x4 gtn[ITEMS];
  auto fetch = [&](int tau_) {
    const int t_ = d ? tau_ : Tn - 1 - tau_;
    const int tp_ = d ? t_ + 1 : t_ - 1;
    const bool hp = tp_ >= 0 && tp_ < Tn;
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      int row = rowbase + (tid >> 6) + 8 * i;
      row = row < rend ? row : a.b0;
      const int64_t fr = (int64_t)t_ * B + row;
      const int unit = u0 + cu;
      dyn[i] = a.DY[fr * 2 * H + (int64_t)d * H + unit];
      cpn[i] = hp ? a.C[((int64_t)tp_ * B + row) * 2 * H + (int64_t)d * H + unit] : 0.f;
      // the unit's four gates are adjacent: one 8-byte load
      gtn[i] = *(const bf16x4*)(a.G + fr * 8 * H + (int64_t)d * 4 * H + (int64_t)unit * 4);
    }
  };
  {
    const int t0 = d ? 0 : Tn - 1;
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      int row = rowbase + (tid >> 6) + 8 * i;
      row = row < rend ? row : a.b0;
      cc[i] = a.C[((int64_t)t0 * B + row) * 2 * H + (int64_t)d * H + u0 + cu];
    }
  }
  fetch(0);

  // gathered (row quad, unit) items: MB == 1: 256 items, two threads each
  // (member halves [0, hm) and [hm, NM)); MB > 1: 256 MB items, MB / 2 per thread
  constexpr int GI = SPLIT ? 1 : MB / 2;    // items per thread
  constexpr int GM = SPLIT ? 4 : 8;         // members per thread at most (NM <= 8)
  const int hm = (NM + 1) / 2;

  for (int tau = 0; tau < Tn; ++tau) {
    const int t = d ? tau : Tn - 1 - tau;
    float dy[ITEMS], cp[ITEMS];
    // the step's gate activations from the prefetched pre-activations,
    // before the gather (whose polls wait for the other members anyway)
    float ga[ITEMS][4];
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      ga[i][0] = sigmoidf_((float)gtn[i][0]);
      ga[i][1] = sigmoidf_((float)gtn[i][1]);
      ga[i][2] = tanhf_((float)gtn[i][2]);
      ga[i][3] = sigmoidf_((float)gtn[i][3]);
    }

    if (tau > 0) {
      const uint64_t* xs = a.X + ((tau - 1) & 1) * slot_stride;
      const uint64_t want = h4_tag(a.seq, tau);
#pragma unroll
      for (int gi = 0; gi < GI; ++gi) {
        const int item = SPLIT ? (tid & 255) : tid + NTH * gi;
        const int qd = item >> 6, u = item & 63;   // row quad within the slice, own unit
        const int mh = SPLIT ? tid >> 8 : 0;
        const int m0 = SPLIT ? mh * hm : 0, mcount = SPLIT ? (mh ? NM - hm : hm) : NM;
        float sum[4] = {0.f, 0.f, 0.f, 0.f};
        if (rowbase + 4 * qd < rend) {
          const uint64_t* src = xs + ((int64_t)d * rquads + (rowbase - a.b0) / 4 + qd) * NM * H + u0 + u;
          const uint64_t* base = src + (int64_t)m0 * H;
          uint64_t wv[GM];
#pragma unroll
          for (int k = 0; k < GM; ++k) wv[k] = k < mcount ? ll_load(base + (int64_t)k * H) : want;
          poll_words<GM>(wv, base, H, want, a.status);
#pragma unroll
          for (int k = 0; k < GM; ++k) {
            if (k >= mcount) break;
#pragma unroll
            for (int r = 0; r < 4; ++r) sum[r] += p15_decode((uint32_t)(wv[k] >> (16 * r)) & 0xffffu);
          }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) dhl[mh * R * PU + (4 * qd + r) * PU + u] = sum[r];
      }
    } else {
      for (int i = tid; i < (SPLIT ? 2 : 1) * R * PU; i += NTH) dhl[i] = 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      dy[i] = dyn[i];
      cp[i] = cpn[i];
    }
    if (tau + 1 < Tn) fetch(tau + 1);

    // cell derivatives; da goes to global memory (weight gradients) and to
    // LDS (next partial product)
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      const int r = (tid >> 6) + 8 * i;
      const int row = rowbase + r;
      const float ig = ga[i][0], fg = ga[i][1], gg = ga[i][2], og = ga[i][3];
      const float dh = (SPLIT ? dhl[r * PU + cu] + dhl[R * PU + r * PU + cu] : dhl[r * PU + cu]) + dy[i];
      const float tc = tanhf_(cc[i]);
      const float dc = dh * og * (1.f - tc * tc) + dcreg[i];
      dcreg[i] = dc * fg;
      float da[4];
      da[0] = dc * gg * ig * (1.f - ig);
      da[1] = dc * cp[i] * fg * (1.f - fg);
      da[2] = dc * ig * (1.f - gg * gg);
      da[3] = dh * tc * og * (1.f - og);
      const bool ok = row < rend;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const bf16 v = ok ? (bf16)da[q] : (bf16)0.f;
        // own row kk = (cu >> 4)*64 + q*16 + (cu & 15)
        const int kk = (cu >> 4) * 64 + q * 16 + (cu & 15);
        al[((kk >> 3) * (R + 1) + r) * 8 + (kk & 7)] = v;
      }
      cc[i] = cp[i];   // c at the next step's t
    }
    __syncthreads();

    // P = da_own [R x 256] * W_own [256 x H]; unit blocks w + 8j of this
    // wave.  On the critical path, so before the global copies of da.
    if (tau + 1 < Tn) {
      uint64_t* xo = a.X + (tau & 1) * slot_stride;
      f32x4 acc[MB][4];
#pragma unroll
      for (int m = 0; m < MB; ++m)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[m][j] = f32x4{0.f, 0.f, 0.f, 0.f};
      // one k-step's A fragments at a time (the scheduling barrier keeps the
      // compiler from loading all of them ahead, which the registers holding
      // W_hh leave no room for)
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
#pragma unroll
        for (int m = 0; m < MB; ++m) {
          const bf16x8 af = *(const bf16x8*)&al[((ks * 4 + (lane >> 4)) * (R + 1) + m * 16 + (lane & 15)) * 8];
          // (unit blocks past H hold zero fragments; their sums are not published)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[m][j] = Mfma<bf16>::mma(af, bw[ks][j], acc[m][j]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      // publish: word (row quad, member, unit), the lane's four rows
      const uint64_t tg = h4_tag(a.seq, tau + 1);
#pragma unroll
      for (int m = 0; m < MB; ++m)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int rl = m * 16 + (lane >> 4) * 4;
          const int nb = w + 8 * j;
          const int unit = nb * 16 + (lane & 15);
          const uint64_t v = (uint64_t)p15_encode(acc[m][j][0]) | ((uint64_t)p15_encode(acc[m][j][1]) << 16) |
                             ((uint64_t)p15_encode(acc[m][j][2]) << 32) | ((uint64_t)p15_encode(acc[m][j][3]) << 48);
          if (rowbase + rl < rend && nb < NB)
            ll_store64(xo + (((int64_t)d * rquads + (rowbase - a.b0 + rl) / 4) * NM + mem) * H + unit, v | tg);
        }
    }

    // da in frame-major rows (DA, for dX): 16 bytes of LDS and of DA per
    // piece, 8 own gate rows of one row
    for (int c = tid; c < 32 * R; c += NTH) {
      const int kg = c & 31, r = c >> 5;
      const int row = rowbase + r;
      if (row < rend) {
        const int kk = kg * 8;
        const int64_t col = (int64_t)d * 4 * H + (int64_t)((kk >> 4) & 3) * H + u0 + (kk >> 6) * 16 + (kk & 15);
        *(uint4*)(a.DA + ((int64_t)t * B + row) * 8 * H + col) = *(const uint4*)&al[(kg * (R + 1) + r) * 8];
      }
    }
    // the own da block (R rows x 256 gate rows, in LDS) also goes out
    // frame-contiguous (DAT) and as bias-gradient partial sums per 16-row
    // block (DBP): thread t takes gate row t/2 and 8 of the 16 rows of a block
    if (a.DAT || a.DBP) {
#pragma unroll
      for (int m = 0; m < MB; ++m) {
        bf16 v[8];
        float sum = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          v[j] = al[((dkk >> 3) * (R + 1) + m * 16 + dh8 + j) * 8 + (dkk & 7)];
          sum += (float)v[j];
        }
        const int row = rowbase + m * 16 + dh8;
        if (a.DAT && row < rend) *(uint4*)(a.DAT + dgrow * a.M + (int64_t)t * B + row) = *(const uint4*)v;
        sum += __shfl_xor(sum, 1);
        dbacc[m] += sum;   // steps in order
      }
    }
  }
  if (a.DBP && (tid & 1) == 0) {
#pragma unroll
    for (int m = 0; m < MB; ++m)
      if (rowbase + m * 16 < rend) a.DBP[(int64_t)((rowbase + m * 16) / 16) * 8 * H + dgrow] = dbacc[m];
  }
}

// The recurrence status block (at the end of the activation workspace): an
// int set to 1 by any exchange wait that gives up, and a 64-bit tag that
// says whether the block has been initialised.  The flag is sticky: only
// status_reset_kernel (blstm_recurrence_ok) clears it, and the forward pass
// initialises it only when the tag is missing (a fresh workspace), so one
// query covers every call since the previous query.
#define STATUS_TAG 0x5354415455535f31ull   // "STATUS_1"

__device__ __forceinline__ void status_init_if_fresh(int* status) {
  uint64_t* tag = (uint64_t*)(status + 2);
  if (*tag != STATUS_TAG) {
    *status = 0;
    *tag = STATUS_TAG;
  }
}

// exchange words cleared; status (if non-null) initialised when fresh
__global__ __launch_bounds__(256) void clear_exchange_kernel(uint4* p, int64_t n16, int* status) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride)
    p[i] = make_uint4(0u, 0u, 0u, 0u);
  if (status && blockIdx.x == 0 && threadIdx.x == 0) status_init_if_fresh(status);
}

__global__ void status_reset_kernel(int* status) {
  *status = 0;
  *(uint64_t*)(status + 2) = STATUS_TAG;
}

// ---------------------------------------------------------------------------
// Host side.
// ---------------------------------------------------------------------------
size_t persist_lds_bytes(int H, bool backward, int MB) {
  const size_t R = 16 * (size_t)MB;
  const size_t run = backward ? (size_t)32 * (R + 1) * 16 + 2 * R * PU * 4
                              : (size_t)(H / 8) * (R + 1) * 16 + (size_t)4 * MB * 4 * 64 * 16 +
                                    (MB == 1 ? (size_t)16 * PU * (4 + 2 + 8) : 0);
  return std::max(run, (size_t)STAGE_BYTES);
}

// Compute units: one persistent workgroup fits per CU (its 8 waves hold
// the W_hh slice in half of the register file and the rest in working
// registers).
static int persist_max_wg() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return cus;
}

bool persist_supported(int H, int T) {
  (void)T;   // any length: the tag holds only bit 1 of the step number
  return H % PU == 0 && H >= PU && H <= 512;
}

// Launch mode.  Every workgroup of a launch waits for the others, so all
// must be resident at once.  A cooperative launch guarantees that, at a
// measured cost of about 15 us per launch on MI355X (12 launches per learner
// step).  A plain launch is used instead when the occupancy query shows that
// the whole grid fits on the device at once (one workgroup per CU here):
// the stream's previous kernel has completed, so every CU is free unless
// other streams or processes occupy some.  In that case the waits give up
// after their bound, the kernel still ends, and the status flag (see
// blstm_recurrence_ok) reports it.  ADPSGD_BLSTM_COOPERATIVE=1 forces
// cooperative launches (for devices shared with other work).
static bool force_cooperative() {
  const char* e = getenv("ADPSGD_BLSTM_COOPERATIVE");
  return e && e[0] == '1';
}

template <int MB, bool BWD>
static hipError_t launch_one(PersistArgs a, hipStream_t s) {
  const void* fn;
  if constexpr (BWD) fn = (const void*)lstm_bwd_persist<MB>;
  else fn = (const void*)lstm_fwd_persist<MB>;
  const size_t lds = persist_lds_bytes(a.H, BWD, MB);
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const dim3 grid(2 * a.NS * (a.H / PU)), block(NTH);
  void* args[] = {&a};
  // the whole grid resident at once? (per device; the answer depends only
  // on the kernel and its resources)
  bool fits = false;
  if (!force_cooperative()) {
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, NTH, lds) == hipSuccess)
      fits = (int64_t)per_cu * persist_max_wg() >= (int64_t)grid.x;
    else
      (void)hipGetLastError();
  }
  const char* name = BWD ? "lstm_rec_bwd_persist" : "lstm_rec_fwd_persist";
  const int slot = g_timing_on ? timing_pre(name, s) : -1;
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  e = hipStreamIsCapturing(s, &cap);
  if (e != hipSuccess) return e;
  if (fits) {
    e = hipLaunchKernel(fn, grid, block, args, lds, s);
  } else if (cap == hipStreamCaptureStatusNone) {
    e = hipLaunchCooperativeKernel(fn, grid, block, args, (unsigned)lds, s);
  } else {
    // recorded into a graph as a kernel node with the cooperative attribute
    hipLaunchAttribute attr;
    memset(&attr, 0, sizeof(attr));
    attr.id = hipLaunchAttributeCooperative;
    attr.val.cooperative = 1;
    hipLaunchConfig_t cfg;
    memset(&cfg, 0, sizeof(cfg));
    cfg.gridDim = grid;
    cfg.blockDim = block;
    cfg.dynamicSmemBytes = lds;
    cfg.stream = s;
    cfg.attrs = &attr;
    cfg.numAttrs = 1;
    e = hipLaunchKernelExC(&cfg, fn, args);
  }
  if (slot >= 0) timing_post(slot, s);
  return e;
}

// Rows per workgroup (16*MB, MB <= PERSIST_MAX_MB) and rows per launch: as
// few row blocks per workgroup as fill the chip (one workgroup per CU);
// more rows by chunking.  False if no launch fits.
static bool persist_plan(int H, int B, int* MBo, int* chunko) {
  const int NM = H / PU;
  const int max_ns = std::min(persist_max_wg() / (2 * NM), PERSIST_MAX_SLICES);
  if (max_ns < 1) return false;
  int MB = 1;
  while (MB < PERSIST_MAX_MB && (B + 16 * MB - 1) / (16 * MB) > max_ns) MB *= 2;
  *MBo = MB;
  *chunko = std::min(B, max_ns * 16 * MB);
  return true;
}

bool persist_bwd_needs_wt(int, int) { return false; }

hipError_t persist_clear(bool backward, const PersistArgs& a, hipStream_t s) {
  int MB, chunk;
  if (!persist_plan(a.H, a.B, &MB, &chunk)) return hipErrorInvalidValue;
  // both exchange slots start without any valid tag; the forward's clear
  // also initialises the status block of a fresh workspace
  const int64_t words = backward ? (int64_t)2 * 2 * ((chunk + 3) / 4) * (a.H / PU) * a.H
                                 : (int64_t)2 * 2 * chunk * (a.H / 4);
  const int64_t n16 = words / 2;
  hipLaunchKernelGGL(clear_exchange_kernel, dim3((unsigned)std::min<int64_t>(cdiv(n16, 256), 2048)), dim3(256), 0,
                     s, (uint4*)a.X, n16, backward ? nullptr : a.status);
  return hipGetLastError();
}

hipError_t persist_status_init(int* status, hipStream_t s) {
  hipLaunchKernelGGL(clear_exchange_kernel, dim3(1), dim3(64), 0, s, (uint4*)nullptr, (int64_t)0, status);
  return hipGetLastError();
}

hipError_t persist_status_reset(int* status, hipStream_t s) {
  hipLaunchKernelGGL(status_reset_kernel, dim3(1), dim3(1), 0, s, status);
  return hipGetLastError();
}

hipError_t persist_layer(bool backward, PersistArgs a, hipStream_t s) {
  int MB, chunk;
  if (!persist_plan(a.H, a.B, &MB, &chunk)) return hipErrorInvalidValue;
  for (int b0 = 0; b0 < a.B; b0 += chunk) {
    PersistArgs c = a;
    c.b0 = b0;
    c.rows = std::min(chunk, a.B - b0);
    c.NS = (c.rows + 16 * MB - 1) / (16 * MB);
    // the launch's position in the call (the caller's tag numbers the layers
    // in the order the call runs them)
    c.seq = a.tag * (uint32_t)cdiv(a.B, chunk) + (uint32_t)(b0 / chunk);
    static_assert(PERSIST_MAX_MB == 1, "one 16-row block per workgroup: the only instantiated kernels");
    const hipError_t e = backward ? launch_one<1, true>(c, s) : launch_one<1, false>(c, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}
