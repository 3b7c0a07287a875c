// Persistent recurrent kernels (bf16 operands): one launch runs all T steps
// of one layer, for both directions at once, with each workgroup's slice of
// W_hh on chip for the whole chunk (in registers at one 16-row block per
// workgroup, staged there through LDS; in LDS for more rows).
//
// Work split.  The batch is cut into slices of 16*MB rows; a group of
// H/32 workgroups owns one (direction, slice) pair and each member owns 32
// hidden units (two blocks of 16).  Its four waves are (unit block, half):
// the half splits the reduction dimension when MB == 1 and the m-blocks
// otherwise.  Per step a member
//   forward : gathers h_prev of its slice (all H units), multiplies by its
//             W_hh rows (4 gates x 32 units), adds the precomputed input
//             projection and applies the cell; c stays in registers, h/c/gates
//             are written for BPTT;
//   backward: applies the gate derivatives for its units (dc stays in
//             registers), multiplies its own da block by its W_hh rows to get
//             partial dh_rec for all H units, publishes them, and sums the
//             partials of all members for its own units.
//
// Step-to-step exchange without barriers or cache maintenance.  The values
// one member needs from the others (h, or partial dh) are published in an
// exchange buffer as 8-byte words holding four 15-bit values and a 4-bit
// tag (see h4_tag), written and read with agent-scope relaxed atomic
// stores and loads.  Atomic accesses to one location are coherent across the
// whole GPU, so a reader that sees the expected step number in a word also
// sees that word's payload; readers poll the words they need (bounded; the
// status word is set if a poll ever gives up).  Two slots alternate by step
// parity: a member overwrites a slot only after it has consumed the next
// step from every member, which those members produce only after they have
// consumed the slot's current contents.  The buffer is cleared once per
// forward or backward call, and the tag tells a word of the expected step
// from one of step n - 2 and from one left by either of the two previous
// launches of the call.  Every member of a
// group must be resident at once: the launch is plain when the occupancy
// query shows the whole grid fits on the device, cooperative otherwise (see
// launch_one).
#include <stdlib.h>
#include <string.h>

#include "common.hpp"
#include "lstm_persist.hpp"
#include "xpose.hpp"
#include "dma.hpp"

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

#define PU 32
#define SPIN_LIMIT (1u << 18)
#define H_MAX_MEMBERS 16   // H / 32 for the largest H whose W_hh slice fits in LDS

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

// MFMA A-fragments for k-steps ks0 .. ks0+nk-1 (nk <= KC) of MBW m-blocks,
// gathered from exchange rows rp[m] (nullptr: row outside the batch, zeros).
// Lane l takes row l % 16 and 8 k values = 2 words at word (ks*8 + (l/16)*2).
template <int MBW, int KC>
__device__ __forceinline__ void ll_fragments(const uint64_t* const (&rp)[MBW], int ks0, int nk,
                                             uint64_t want, int lane, bf16x8 (&af)[MBW][KC],
                                             int* status) {
  uint64_t w[MBW][KC][2];
  const int woff = (lane >> 4) * 2;
#pragma unroll
  for (int m = 0; m < MBW; ++m)
#pragma unroll
    for (int kk = 0; kk < KC; ++kk)
#pragma unroll
      for (int i = 0; i < 2; ++i)
        w[m][kk][i] = (rp[m] && kk < nk) ? ll_load(rp[m] + (ks0 + kk) * 8 + woff + i) : want;
  for (unsigned it = 0;; ++it) {
    bool bad = false;
#pragma unroll
    for (int m = 0; m < MBW; ++m)
#pragma unroll
      for (int kk = 0; kk < KC; ++kk)
#pragma unroll
        for (int i = 0; i < 2; ++i) bad |= (w[m][kk][i] & H4_TAG_BITS) != want;
    if (!bad) break;
    // give up after SPIN_LIMIT polls, or at once when any lane anywhere has
    // given up before (then every later poll returns immediately too)
    if (it > SPIN_LIMIT ||
        ((it & 63) == 63 && __hip_atomic_load(status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))) {
      __hip_atomic_store(status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      break;
    }
    __builtin_amdgcn_s_sleep(1);
#pragma unroll
    for (int m = 0; m < MBW; ++m)
#pragma unroll
      for (int kk = 0; kk < KC; ++kk)
#pragma unroll
        for (int i = 0; i < 2; ++i)
          if ((w[m][kk][i] & H4_TAG_BITS) != want) w[m][kk][i] = ll_load(rp[m] + (ks0 + kk) * 8 + woff + i);
  }
#pragma unroll
  for (int m = 0; m < MBW; ++m)
#pragma unroll
    for (int kk = 0; kk < KC; ++kk) {
      const uint64_t lo = w[m][kk][0] & ~H4_TAG_BITS, hi = w[m][kk][1] & ~H4_TAG_BITS;
      const uint4 v = make_uint4((uint32_t)lo, (uint32_t)(lo >> 32), (uint32_t)hi, (uint32_t)(hi >> 32));
      af[m][kk] = __builtin_bit_cast(bf16x8, v);
    }
}

// ---------------------------------------------------------------------------
// Forward.
// ---------------------------------------------------------------------------
template <int MB>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void lstm_fwd_persist(const PersistArgs a) {
  extern __shared__ __attribute__((aligned(16))) bf16 lds[];
  constexpr bool KSPLIT = MB == 1;
  constexpr int MBW = KSPLIT ? 1 : MB / 2;
  constexpr int KC = MBW >= 4 ? 2 : 8 / MBW;   // k-steps gathered per poll (all of a half when MB == 1)
  constexpr int LDN = 128 + 1;   // LDS rows per k-group (128 gate rows + pad)
  const int H = a.H, B = a.B, Tn = a.Tn;
  const int NG = 2 * a.NS;
  const int g = blockIdx.x % NG, mem = blockIdx.x / NG;
  const int d = g & 1, s = g >> 1;
  const int u0 = mem * PU;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int ub = w & 1, wx = w >> 1;

  // W_hh rows of this member.  MB > 1: in LDS, row n = ub*64 + gate*16 + u,
  // stored as [k/8][n][8]; staged with direct-to-LDS loads (one load fills
  // 64 consecutive rows of one 8-wide k chunk), all in flight at once.
  // MB == 1: in registers (below), each wave holding the fragments of its
  // unit block and k half, so the products read no W from LDS.
  const bf16* Wd = a.W + (d ? a.whh1 : a.whh0);
  const int kcn = H / 8;
  if constexpr (!KSPLIT) {
    const __amdgpu_buffer_rsrc_t rw = dma_rsrc(Wd);
    const int n = (w & 1) * 64 + lane;   // row of this lane
    const int64_t row = (int64_t)((n >> 4) & 3) * H + u0 + (n >> 6) * 16 + (n & 15);
    for (int kc = w >> 1; kc < kcn; kc += 2)
      dma16(rw, (uint32_t)((row * H + kc * 8) * 2), lds + (kc * LDN + (w & 1) * 64) * 8);
    dma_wait_all();
  }
  f32x4* red = (f32x4*)(lds + (KSPLIT ? (size_t)0 : (size_t)kcn * LDN * 8));
  bf16* hl = (bf16*)(red + 8 * 64);   // MB == 1: gathered h [H/8][16 + 1][8]
  // MB == 1: a step's c [16][32] (float), h [16][32] and gate pre-activations [16][32][4]
  // (bf16) of the own units, staged for 16-byte stores
  float* sC = (float*)(hl + (size_t)(H / 8) * 17 * 8);
  bf16* sY = (bf16*)(sC + 16 * 32);
  bf16* sG = sY + 16 * 32;
  __syncthreads();

  const int rend = a.b0 + a.rows;
  const int rowbase = a.b0 + s * 16 * MB;
  const int mb0 = KSPLIT ? 0 : wx * MBW;
  const bool epi = !KSPLIT || wx == 0;
  const int unit = u0 + ub * 16 + (lane & 15);
  const int nks = H / 32;
  const int ks_beg = KSPLIT ? (wx ? nks / 2 : 0) : 0;
  const int ks_end = KSPLIT ? (wx ? nks : nks / 2) : nks;
  // MB == 1: B fragments of the k half (at most H_MAX_MEMBERS / 2 k-steps;
  // lane l: gate row q*H + unit, k = ks*32 + (l/16)*8 .. +8); k-steps past
  // the half's end hold a valid k-step and meet a zero A fragment.  The 128
  // own gate rows (gate q, unit u0 + i at local row q*32 + i) are staged by
  // direct-to-LDS loads, 1 KB rows (units past H read as zeros), the 16-byte
  // chunk c of local row lr in slot c ^ (lr & 15) so that the 16 rows of one
  // fragment read land in distinct bank groups.
  constexpr int KH = H_MAX_MEMBERS / 2;
  bf16x8 bw[KSPLIT ? KH : 1][4];
  if constexpr (KSPLIT) {
    char* stg = (char*)lds;
    const __amdgpu_buffer_rsrc_t rw = dma_rsrc(Wd);
#pragma unroll
    for (int q = 0; q < 32; ++q) {
      const int lr = q * 4 + w;   // one 1 KB row per load instruction
      const int c = lane ^ (lr & 15);
      const int64_t grow = (int64_t)(lr >> 5) * H + u0 + (lr & 31);
      dma16(rw, c * 8 < H ? (uint32_t)((grow * H + c * 8) * 2) : DMA_OFF_NONE, stg + lr * 1024);
    }
    dma_wait_all();
    __syncthreads();
#pragma unroll
    for (int i = 0; i < KH; ++i) {
      const int ks = max(0, min(ks_beg + i, ks_end - 1));
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int lr = q * 32 + ub * 16 + (lane & 15);
        const int c = ks * 4 + (lane >> 4);
        bw[i][q] = *(const bf16x8*)(stg + lr * 1024 + (c ^ (lr & 15)) * 16);
      }
    }
    __syncthreads();   // the reduction buffer and gathered h reuse this LDS
  }
  const int wpr = H / 4;                        // exchange words per row
  constexpr int NJ4 = H_MAX_MEMBERS * PU / 64;  // MB == 1: words per thread and row (16 threads)
  const int64_t slot_stride = (int64_t)2 * a.rows * wpr;

  float creg[MBW][4];
#pragma unroll
  for (int m = 0; m < MBW; ++m)
#pragma unroll
    for (int r = 0; r < 4; ++r) creg[m][r] = 0.f;

  // input projection of a step (independent of h), loaded one step ahead so
  // that its latency hides behind the previous step's exchange
  bf16 gx[MBW][4][4], gxn[MBW][4][4];
  auto load_gx = [&](int tt) {
#pragma unroll
    for (int m = 0; m < MBW; ++m)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = rowbase + (mb0 + m) * 16 + (lane >> 4) * 4 + r;
        const bf16* p = a.Gx + ((int64_t)tt * B + (row < rend ? row : a.b0)) * 8 * H + (int64_t)d * 4 * H + unit;
#pragma unroll
        for (int q = 0; q < 4; ++q) gxn[m][r][q] = p[q * H];
      }
  };
  if (epi) load_gx(d ? Tn - 1 : 0);

  for (int tau = 0; tau < Tn; ++tau) {
    const int t = d ? Tn - 1 - tau : tau;
    if (epi) {
#pragma unroll
      for (int m = 0; m < MBW; ++m)
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int q = 0; q < 4; ++q) gx[m][r][q] = gxn[m][r][q];
    }

    f32x4 acc[MBW][4];
#pragma unroll
    for (int m = 0; m < MBW; ++m)
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[m][q] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (KSPLIT && tau > 0) {
      // h of the previous step (16 rows x H/2 words, published with step
      // number tau) is polled by all 256 threads in whole cache lines (thread
      // t: row t/16, words t%16 + 16j) and staged in LDS in the MFMA A layout
      const int tr = tid >> 4, tw = tid & 15;
      const int row = rowbase + tr;
      const bool rok = row < rend;
      const uint64_t* src = a.X + ((tau - 1) & 1) * slot_stride + ((int64_t)d * a.rows + (rok ? row - a.b0 : 0)) * wpr + tw;
      const uint64_t want = h4_tag(a.seq, tau);
      uint64_t wv[NJ4];
#pragma unroll
      for (int j = 0; j < NJ4; ++j) wv[j] = (rok && tw + 16 * j < wpr) ? ll_load(src + 16 * j) : want;
      for (unsigned it = 0;; ++it) {
        bool bad = false;
#pragma unroll
        for (int j = 0; j < NJ4; ++j) bad |= (wv[j] & H4_TAG_BITS) != want;
        if (!bad) break;
        if (it > SPIN_LIMIT ||
            ((it & 63) == 63 && __hip_atomic_load(a.status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))) {
          __hip_atomic_store(a.status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          break;
        }
        __builtin_amdgcn_s_sleep(1);
#pragma unroll
        for (int j = 0; j < NJ4; ++j)
          if ((wv[j] & H4_TAG_BITS) != want) wv[j] = ll_load(src + 16 * j);
      }
#pragma unroll
      for (int j = 0; j < NJ4; ++j) {
        if (tw + 16 * j >= wpr) break;
        const int k = 4 * (tw + 16 * j);   // units k .. k+3
        *(uint64_t*)&hl[((k >> 3) * 17 + tr) * 8 + (k & 7)] = rok ? (wv[j] & ~H4_TAG_BITS) : 0ull;
      }
      __syncthreads();
      // A fragments of the half (W is in registers), then the products
      bf16x8 af[KH];
#pragma unroll
      for (int i = 0; i < KH; ++i) {
        const int ks = max(0, min(ks_beg + i, ks_end - 1));
        const int kg = ks * 4 + (lane >> 4);
        af[i] = *(const bf16x8*)&hl[(kg * 17 + (lane & 15)) * 8];
        if (ks_beg + i >= ks_end) af[i] = bf16x8{};
      }
#pragma unroll
      for (int i = 0; i < KH; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[0][q] = Mfma<bf16>::mma(af[i], bw[i][q], acc[0][q]);
    } else if (tau > 0) {
      // h of the previous step, published with step number tau
      const uint64_t* rp[MBW];
#pragma unroll
      for (int m = 0; m < MBW; ++m) {
        const int row = rowbase + (mb0 + m) * 16 + (lane & 15);
        rp[m] = row < rend ? a.X + ((tau - 1) & 1) * slot_stride + ((int64_t)d * a.rows + (row - a.b0)) * wpr
                           : nullptr;
      }
      for (int ks0 = ks_beg; ks0 < ks_end; ks0 += KC) {
        const int nk = min(KC, ks_end - ks0);
        bf16x8 af[MBW][KC];
        ll_fragments<MBW, KC>(rp, ks0, nk, h4_tag(a.seq, tau), lane, af, a.status);
#pragma unroll
        for (int kk = 0; kk < KC; ++kk) {
          if (kk >= nk) break;
          const int kg = (ks0 + kk) * 4 + (lane >> 4);
          bf16x8 bfr[4];
#pragma unroll
          for (int q = 0; q < 4; ++q)
            bfr[q] = *(const bf16x8*)&lds[(kg * LDN + ub * 64 + q * 16 + (lane & 15)) * 8];
#pragma unroll
          for (int m = 0; m < MBW; ++m)
#pragma unroll
            for (int q = 0; q < 4; ++q) acc[m][q] = Mfma<bf16>::mma(af[m][kk], bfr[q], acc[m][q]);
        }
      }
    }
    if (KSPLIT) {
      if (wx == 1) {
#pragma unroll
        for (int q = 0; q < 4; ++q) red[(ub * 4 + q) * 64 + lane] = acc[0][q];
      }
      __syncthreads();
      if (wx == 0) {
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[0][q] += red[(ub * 4 + q) * 64 + lane];
      }
    }
    if (epi) {
      // cell math of all rows, then h published (the other members wait for
      // it), then the saved activations (only read after the launch)
      uint64_t* xo = a.X + (tau & 1) * slot_stride;
      float hv[MBW][4], gv[MBW][4][4];
#pragma unroll
      for (int m = 0; m < MBW; ++m)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          // gv: pre-activations, saved for the backward
#pragma unroll
          for (int q = 0; q < 4; ++q) gv[m][r][q] = acc[m][q][r] + (float)gx[m][r][q];
          const float ig = sigmoidf_(gv[m][r][0]), fg = sigmoidf_(gv[m][r][1]);
          const float gg = tanhf_(gv[m][r][2]), og = sigmoidf_(gv[m][r][3]);
          const float c = fg * creg[m][r] + ig * gg;
          creg[m][r] = c;
          hv[m][r] = og * tanhf_(c);
        }
      // every row's h before the first publish (the empty asm pins the
      // values here, so the compiler cannot sink their math past a publish)
#pragma unroll
      for (int m = 0; m < MBW; ++m)
#pragma unroll
        for (int r = 0; r < 4; ++r) __asm__ volatile("" : "+v"(hv[m][r]));
#pragma unroll
      for (int m = 0; m < MBW; ++m)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = rowbase + (mb0 + m) * 16 + (lane >> 4) * 4 + r;
          const float h_next_unit = lane_xor1(hv[m][r]);   // lanes of one row, units u and u^1
          // lane 4i stores units 4i .. 4i+3 (the pairs of lanes 4i and 4i+2)
          const uint32_t p2 = pack_bf16x2(hv[m][r], h_next_unit);
          const uint32_t p4 = lane_xor2(p2);
          if (row < rend && (lane & 3) == 0)
            ll_store64(xo + ((int64_t)d * a.rows + (row - a.b0)) * wpr + unit / 4,
                       ((((uint64_t)p4 << 32) | p2) & ~H4_TAG_BITS) | h4_tag(a.seq, tau + 1));
        }
      if constexpr (KSPLIT) {
        // into LDS; the whole workgroup writes them out after the barrier
        const int ul = ub * 16 + (lane & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int rl = (lane >> 4) * 4 + r;
          sC[rl * 32 + ul] = creg[0][r];
          sY[rl * 32 + ul] = (bf16)hv[0][r];
          bf16x4 g4;
#pragma unroll
          for (int q = 0; q < 4; ++q) g4[q] = (bf16)gv[0][r][q];
          *(bf16x4*)&sG[(rl * 32 + ul) * 4] = g4;
        }
      } else {
#pragma unroll
        for (int m = 0; m < MBW; ++m)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int row = rowbase + (mb0 + m) * 16 + (lane >> 4) * 4 + r;
            if (row >= rend) continue;
            const int64_t fr = (int64_t)t * B + row;
            a.C[fr * 2 * H + (int64_t)d * H + unit] = creg[m][r];
            a.Y[fr * 2 * H + (int64_t)d * H + unit] = (bf16)hv[m][r];
            bf16* gs = a.G + fr * 8 * H + (int64_t)d * 4 * H + (int64_t)unit * 4;
#pragma unroll
            for (int q = 0; q < 4; ++q) gs[q] = (bf16)gv[m][r][q];
          }
      }
    }
    if (epi && tau + 1 < Tn) load_gx(d ? Tn - 2 - tau : tau + 1);
    __syncthreads();   // the reduction buffer is reused by the next step
    if constexpr (KSPLIT) {
      // c, h and the gates of the step in 16-byte pieces (448 per step
      // instead of 24 two- or four-byte stores per lane of the two cell
      // waves): gates by every thread (a row's 32 units x 4 gates are 256
      // contiguous bytes), c by threads 0-127, h by 128-191.  The next step's
      // gather barrier comes before the LDS is rewritten.
      {
        const int rl = tid >> 4, c = tid & 15;
        const int row = rowbase + rl;
        if (row < rend)
          *(uint4*)(a.G + ((int64_t)t * B + row) * 8 * H + (int64_t)d * 4 * H + (int64_t)u0 * 4 + c * 8) =
              *(const uint4*)&sG[rl * 128 + c * 8];
      }
      if (tid < 128) {
        const int rl = tid >> 3, c = tid & 7;
        const int row = rowbase + rl;
        if (row < rend)
          *(float4*)(a.C + ((int64_t)t * B + row) * 2 * H + (int64_t)d * H + u0 + c * 4) =
              *(const float4*)&sC[rl * 32 + c * 4];
      } else if (tid < 192) {
        const int rl = (tid - 128) >> 2, c = (tid - 128) & 3;
        const int row = rowbase + rl;
        if (row < rend)
          *(uint4*)(a.Y + ((int64_t)t * B + row) * 2 * H + (int64_t)d * H + u0 + c * 8) =
              *(const uint4*)&sY[rl * 32 + c * 8];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Backward (BPTT).
//
// dh_rec[b][j] = sum over all 4H gate rows g of da[b][g] W_hh[g][j].  Member
// m owns the 128 gate rows of its 32 units, so it computes the partial sums
// P_m = da[:, own rows] W_hh[own rows, :] for ALL H units from data it
// already holds (its own da, kept in LDS, and its W_hh rows, LDS-resident),
// publishes P_m as exchange words, and gathers for its own 32 units the
// partials of all members, summed in member order.  Per step a member thus
// reads rows x 32 x H/32 values instead of rows x 4H.  An exchange word
// holds one unit's partials for two adjacent rows; words are ordered (row
// pair, member, unit), so a member publishes whole cache lines and a reader
// takes 256 contiguous bytes of each member.
// ---------------------------------------------------------------------------
template <int MB>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void lstm_bwd_persist(const PersistArgs a) {
  extern __shared__ __attribute__((aligned(16))) bf16 lds[];
  constexpr int R = 16 * MB;            // rows of this member's slice
  constexpr int ITEMS = 2 * MB;         // (row, unit) cell items per thread
  const int H = a.H, B = a.B, Tn = a.Tn;
  const int NM = H / PU, NG = 2 * a.NS;
  const int g = blockIdx.x % NG, mem = blockIdx.x / NG;
  const int d = g & 1, s = g >> 1;
  const int u0 = mem * PU;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;

  // LDS: W_hh of the 128 own gate rows, as the B operand [k/8][unit][8]
  // (k = own row kk: gate (kk>>4)&3, unit u0 + (kk>>6)*16 + (kk&15)), for
  // MB > 1 (MB == 1 holds it in registers, below); own da as the A operand
  // [k/8][row][8]; gathered dh_rec [row][32] fp32.
  constexpr bool WREG = MB == 1;
  bf16* wl = lds;
  bf16* al = wl + (WREG ? (size_t)0 : (size_t)16 * (H + 1) * 8);
  float* dhl = (float*)(al + (size_t)16 * (R + 1) * 8);
  const int NB = H / 16;
  // MB == 1: B fragments of the unit blocks nb = 16*bi + w + 4*j of this
  // wave, k-step ks (lane l: own rows ks*32 + (l/16)*8 .. +8, unit
  // nb*16 + l%16), read from W_hh as it lies: the own rows are staged into
  // LDS by direct-to-LDS loads ([kk][512 units], 1 KB rows, the 16-byte chunk
  // c of row kk in slot c ^ wswz(kk); units past H read as zeros), and each
  // lane takes its fragments with transposing LDS reads (ds_read_b64_tr_b16:
  // in a 16-lane group lane r addresses 4 consecutive units of k row r/4 and
  // receives unit column r's values over those 4 rows; two reads give the 8
  // consecutive k of the MFMA B operand).  The swizzle spreads the 16 rows of
  // one read over distinct chunk pairs.
  bf16x8 bw[WREG ? 2 : 1][4][4];
  if constexpr (WREG) {
    auto wswz = [](int k) { return 2 * ((k & 3) | (((k >> 3) & 1) << 2)); };
    char* stg = (char*)lds;
    const __amdgpu_buffer_rsrc_t rw = dma_rsrc(a.W + (d ? a.whh1 : a.whh0));
#pragma unroll
    for (int q = 0; q < 32; ++q) {
      const int kk = q * 4 + w;   // one 1 KB row per load instruction
      const int c = lane ^ wswz(kk);
      const int64_t grow = (int64_t)((kk >> 4) & 3) * H + u0 + (kk >> 6) * 16 + (kk & 15);
      dma16(rw, c * 8 < H ? (uint32_t)((grow * H + c * 8) * 2) : DMA_OFF_NONE, stg + kk * 1024);
    }
    dma_wait_all();
    __syncthreads();
    const int gq = lane >> 4, r = lane & 15;
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int mn = (bi * 16 + w + 4 * j) * 16 + 4 * (r & 3);
          bf16x4 h[2];
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const int k = ks * 32 + 8 * gq + 4 * hh + (r >> 2);
            const char* pa = stg + k * 1024 + ((mn >> 3) ^ wswz(k)) * 16 + (mn & 7) * 2;
            h[hh] = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((__attribute__((address_space(3))) bf16x4*)(pa));
          }
          bw[bi][ks][j] = bf16x8{h[0][0], h[0][1], h[0][2], h[0][3], h[1][0], h[1][1], h[1][2], h[1][3]};
        }
  } else if (a.WT && H % 64 == 0) {
    // from W_hh^T [H][4H] (made by the caller): the 8 own rows of k group kg
    // are 16 contiguous bytes of W_hh^T row j; one direct-to-LDS load fills
    // 64 consecutive j of one k group (a load always writes all 64 slots, so
    // H must be a multiple of 64)
    const __amdgpu_buffer_rsrc_t rw = dma_rsrc(a.WT + (int64_t)d * H * 4 * H);
    for (int c = w; c < 16 * (H / 64); c += 4) {
      const int kg = c % 16, j = (c / 16) * 64 + lane;
      const int kk = kg * 8;
      const int64_t grow = (int64_t)((kk >> 4) & 3) * H + u0 + (kk >> 6) * 16 + (kk & 15);
      dma16(rw, (uint32_t)(((int64_t)j * 4 * H + grow) * 2), wl + (kg * (H + 1) + (c / 16) * 64) * 8);
    }
    dma_wait_all();
  } else if constexpr (!WREG) {
    const bf16* Wd = a.W + (d ? a.whh1 : a.whh0);
    for (int b = tid; b < 16 * (H / 8); b += 256) {
      const int kg = b % 16, jb = b / 16;
      uint4 in[8], out[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int kk = kg * 8 + i;
        const int64_t grow = (int64_t)((kk >> 4) & 3) * H + u0 + (kk >> 6) * 16 + (kk & 15);
        in[i] = *(const uint4*)(Wd + grow * H + jb * 8);
      }
      transpose8x8(in, out);
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) *(uint4*)&wl[(kg * (H + 1) + jb * 8 + jj) * 8] = out[jj];
    }
  }
  __syncthreads();

  const int rend = a.b0 + a.rows;
  const int rowbase = a.b0 + s * R;
  const int rquads = (a.rows + 3) / 4;             // row quads of this launch
  const int64_t slot_stride = (int64_t)2 * rquads * NM * H;
  // cell items: unit cu = tid % 32, rows tid/32 + 8*i
  const int cu = tid & 31;
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

  // everything the cell derivative needs besides dh_rec: dy, the gate pre-activations and
  // c at t, c at the step's predecessor in forward time (which is the next
  // step's t).  Fetched one step ahead, right after the previous step's
  // gather, so that no gather waits for them; c at t is the previous step's
  // predecessor value.
  float dyn[ITEMS], cpn[ITEMS], cc[ITEMS];
  bf16 gtn[ITEMS][4];
  auto fetch = [&](int tau_) {
    const int t_ = d ? tau_ : Tn - 1 - tau_;
    const int tp_ = d ? t_ + 1 : t_ - 1;
    const bool hp = tp_ >= 0 && tp_ < Tn;
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      int row = rowbase + (tid >> 5) + 8 * i;
      row = row < rend ? row : a.b0;
      const int64_t fr = (int64_t)t_ * B + row;
      const int unit = u0 + cu;
      dyn[i] = a.DY[fr * 2 * H + (int64_t)d * H + unit];
      cpn[i] = hp ? a.C[((int64_t)tp_ * B + row) * 2 * H + (int64_t)d * H + unit] : 0.f;
      // the unit's four gates are adjacent: one 8-byte load
      const bf16x4 g4 = *(const bf16x4*)(a.G + fr * 8 * H + (int64_t)d * 4 * H + (int64_t)unit * 4);
#pragma unroll
      for (int q = 0; q < 4; ++q) gtn[i][q] = g4[q];
    }
  };
  {
    const int t0 = d ? 0 : Tn - 1;
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      int row = rowbase + (tid >> 5) + 8 * i;
      row = row < rend ? row : a.b0;
      cc[i] = a.C[((int64_t)t0 * B + row) * 2 * H + (int64_t)d * H + u0 + cu];
    }
  }
  fetch(0);

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

    // gather dh_rec for the own units.  MB == 1: items (row quad, unit,
    // member parity), unit = tid % 32, quad (tid / 32) % 4; each thread sums
    // the members of its parity in order into its half of the LDS sums.
    // MB > 1: items (row pair, unit); the 32 threads of a row pair read 32
    // adjacent words (256 bytes) per member.
    if (WREG && tau > 0) {
      const uint64_t* xs = a.X + ((tau - 1) & 1) * slot_stride;
      const int qd = (tid >> 5) & 3, mh = tid >> 7;
      float sum[4] = {0.f, 0.f, 0.f, 0.f};
      if (rowbase + 4 * qd < rend) {
        const uint64_t want = h4_tag(a.seq, tau);
        const uint64_t* src = xs + ((int64_t)d * rquads + (rowbase - a.b0) / 4 + qd) * NM * H + u0 + cu;
        constexpr int KM = H_MAX_MEMBERS / 2;
        uint64_t wv[KM];
#pragma unroll
        for (int k = 0; k < KM; ++k) wv[k] = 2 * k + mh < NM ? ll_load(src + (int64_t)(2 * k + mh) * H) : want;
        for (unsigned it = 0;; ++it) {
          bool bad = false;
#pragma unroll
          for (int k = 0; k < KM; ++k) bad |= (wv[k] & H4_TAG_BITS) != want;
          if (!bad) break;
          if (it > SPIN_LIMIT ||
              ((it & 63) == 63 && __hip_atomic_load(a.status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))) {
            __hip_atomic_store(a.status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            break;
          }
          __builtin_amdgcn_s_sleep(1);
#pragma unroll
          for (int k = 0; k < KM; ++k)
            if ((wv[k] & H4_TAG_BITS) != want) wv[k] = ll_load(src + (int64_t)(2 * k + mh) * H);
        }
#pragma unroll
        for (int k = 0; k < KM; ++k) {
          if (2 * k + mh >= NM) break;
#pragma unroll
          for (int r = 0; r < 4; ++r) sum[r] += p15_decode((uint32_t)(wv[k] >> (16 * r)) & 0xffffu);
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) dhl[mh * R * PU + (4 * qd + r) * PU + cu] = sum[r];
    } else if (tau > 0) {
      const uint64_t* xs = a.X + ((tau - 1) & 1) * slot_stride;
      const uint64_t want = h4_tag(a.seq, tau);
#pragma unroll
      for (int i = 0; i < (MB + 1) / 2; ++i) {
        const int qd = (tid >> 5) + 8 * i;   // row quad within this member's rows
        float sum[4] = {0.f, 0.f, 0.f, 0.f};
        if (qd < 4 * MB && rowbase + 4 * qd < rend) {
          const uint64_t* src = xs + ((int64_t)d * rquads + (rowbase - a.b0) / 4 + qd) * NM * H + u0 + cu;
          uint64_t wv[H_MAX_MEMBERS];
#pragma unroll
          for (int k = 0; k < H_MAX_MEMBERS; ++k) wv[k] = k < NM ? ll_load(src + (int64_t)k * H) : want;
          for (unsigned it = 0;; ++it) {
            bool bad = false;
#pragma unroll
            for (int k = 0; k < H_MAX_MEMBERS; ++k) bad |= (wv[k] & H4_TAG_BITS) != want;
            if (!bad) break;
            if (it > SPIN_LIMIT ||
                ((it & 63) == 63 && __hip_atomic_load(a.status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))) {
              __hip_atomic_store(a.status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              break;
            }
            __builtin_amdgcn_s_sleep(1);
#pragma unroll
            for (int k = 0; k < H_MAX_MEMBERS; ++k)
              if ((wv[k] & H4_TAG_BITS) != want) wv[k] = ll_load(src + (int64_t)k * H);
          }
#pragma unroll
          for (int k = 0; k < H_MAX_MEMBERS; ++k) {
            if (k >= NM) break;
#pragma unroll
            for (int r = 0; r < 4; ++r) sum[r] += p15_decode((uint32_t)(wv[k] >> (16 * r)) & 0xffffu);
          }
        }
        if (qd < 4 * MB) {
#pragma unroll
          for (int r = 0; r < 4; ++r) dhl[(4 * qd + r) * PU + cu] = sum[r];
        }
      }
    } else {
      for (int i = tid; i < (WREG ? 2 : 1) * R * PU; i += 256) dhl[i] = 0.f;
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
      const int r = (tid >> 5) + 8 * i;
      const int row = rowbase + r;
      const float ig = ga[i][0], fg = ga[i][1], gg = ga[i][2], og = ga[i][3];
      const float dh = (WREG ? dhl[r * PU + cu] + dhl[R * PU + r * PU + cu] : dhl[r * PU + cu]) + dy[i];
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

    // P = da_own [R x 128] * W_own [128 x H]; 16-unit block nb goes to wave
    // nb % 4.  On the critical path, so before the global copies of da.
    if (tau + 1 < Tn) {
      uint64_t* xo = a.X + (tau & 1) * slot_stride;
      // the A fragments (own da, 4 k-steps) serve every unit block
      bf16x8 af[MB][4];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int m = 0; m < MB; ++m)
          af[m][ks] = *(const bf16x8*)&al[((ks * 4 + (lane >> 4)) * (R + 1) + m * 16 + (lane & 15)) * 8];
      // unit blocks per pass and wave: all (up to 8) with W in registers,
      // else 4 per pass (two passes cover H_MAX_MEMBERS * 32 units)
      constexpr int JP = WREG ? 8 : 4;
#pragma unroll
      for (int bi = 0; bi < (WREG ? 1 : H_MAX_MEMBERS / 8); ++bi) {
        const int base = bi * 16;
        if (base >= NB) break;
        f32x4 acc[MB][JP];
#pragma unroll
        for (int m = 0; m < MB; ++m)
#pragma unroll
          for (int j = 0; j < JP; ++j) acc[m][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        // all B fragments of this pass first (registers, or one LDS round
        // trip), then the products
        bf16x8 bfr[4][JP];
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
#pragma unroll
          for (int j = 0; j < JP; ++j) {
            const int nb = base + w + 4 * j;
            if constexpr (WREG)
              bfr[ks][j] = bw[j / 4][ks][j % 4];
            else
              bfr[ks][j] = nb < NB ? *(const bf16x8*)&wl[((ks * 4 + (lane >> 4)) * (H + 1) + nb * 16 + (lane & 15)) * 8]
                                   : bf16x8{};
          }
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
#pragma unroll
          for (int m = 0; m < MB; ++m)
#pragma unroll
            for (int j = 0; j < JP; ++j) acc[m][j] = Mfma<bf16>::mma(af[m][ks], bfr[ks][j], acc[m][j]);
        // publish: word (row quad, member, unit), the lane's four rows
        const uint64_t tg = h4_tag(a.seq, tau + 1);
#pragma unroll
        for (int m = 0; m < MB; ++m)
#pragma unroll
          for (int j = 0; j < JP; ++j) {
            const int rl = m * 16 + (lane >> 4) * 4;
            const int nb = base + w + 4 * j;
            const int unit = nb * 16 + (lane & 15);
            const uint64_t v = (uint64_t)p15_encode(acc[m][j][0]) | ((uint64_t)p15_encode(acc[m][j][1]) << 16) |
                               ((uint64_t)p15_encode(acc[m][j][2]) << 32) | ((uint64_t)p15_encode(acc[m][j][3]) << 48);
            if (rowbase + rl < rend && nb < NB)
              ll_store64(xo + (((int64_t)d * rquads + (rowbase - a.b0 + rl) / 4) * NM + mem) * H + unit, v | tg);
          }
      }
    }

    // da in frame-major rows (DA, for dX): thread t copies 8 own gate rows
    // (16 contiguous bytes of LDS and of DA) of one row
#pragma unroll
    for (int m = 0; m < MB; ++m) {
      const int kg = tid & 15, r = m * 16 + (tid >> 4);
      const int row = rowbase + r;
      if (row < rend) {
        const int kk = kg * 8;
        const int64_t col = (int64_t)d * 4 * H + (int64_t)((kk >> 4) & 3) * H + u0 + (kk >> 6) * 16 + (kk & 15);
        *(uint4*)(a.DA + ((int64_t)t * B + row) * 8 * H + col) = *(const uint4*)&al[(kg * (R + 1) + r) * 8];
      }
    }
    // the own da block (R rows x 128 gate rows, in LDS) also goes out
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
  if (backward) {   // MB == 1 keeps W_hh in registers, staged through 128 KB of LDS
    const size_t run = (MB == 1 ? (size_t)0 : (size_t)16 * (H + 1) * 16) + (size_t)16 * (16 * MB + 1) * 16 +
                       (size_t)2 * 16 * MB * PU * 4;
    return MB == 1 ? std::max(run, (size_t)128 * 1024) : run;
  }
  // MB == 1 keeps W_hh in registers (staged through 128 KB of LDS at the
  // start): reduction buffer, gathered h and the step's staged c/h/gates
  // (7 KB) after that
  if (MB == 1) return std::max((size_t)8 * 64 * 16 + (size_t)(H / 8) * 17 * 16 + 7 * 1024, (size_t)128 * 1024);
  return (size_t)(H / 8) * (128 + 1) * 16 + 8 * 64 * 16;
}

// Workgroups that can be co-resident: one per compute unit (the LDS slice
// of the paper's H = 512 takes most of a CU's 160 KB).
static int persist_max_wg() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return cus;
}

bool persist_supported(int H, int T) {
  (void)T;   // any length: the tag holds only bit 1 of the step number
  return H % PU == 0 && H / PU <= H_MAX_MEMBERS && persist_lds_bytes(H, false, 2) <= 160 * 1024 &&
         persist_lds_bytes(H, true, 2) <= 160 * 1024;
}

// Launch mode.  Every workgroup of a launch waits for the others, so all
// must be resident at once.  A cooperative launch guarantees that, at a
// measured cost of about 15 us per launch on MI355X (12 launches per learner
// step).  A plain launch is used instead when the occupancy query shows that
// the whole grid fits on the device at once (one workgroup per CU here):
// the stream's previous kernel has completed, so every CU is free unless
// other streams or processes occupy some.  In that case the waits give up
// after their bound, the kernel still ends, and the status word (see
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
  const dim3 grid(2 * a.NS * (a.H / PU)), block(256);
  void* args[] = {&a};
  // the whole grid resident at once? (per device; the answer depends only
  // on the kernel and its resources)
  bool fits = false;
  if (!force_cooperative()) {
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, 256, lds) == hipSuccess)
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

// Runs all steps of one layer (both directions); returns hipSuccess or the
// launch error (nothing was enqueued for the failing chunk in that case).
// Rows per workgroup (16*MB) and rows per launch: as few rows as fill the
// chip, up to 8 row blocks (4 in the backward, whose LDS also holds its own
// da), more rows by chunking.  False if no launch fits.
static bool persist_plan(bool backward, int H, int B, int* MBo, int* chunko) {
  const int NM = H / PU;
  const int max_ns = std::min(persist_max_wg() / (2 * NM), PERSIST_MAX_SLICES);
  if (max_ns < 1) return false;
  const int mb_cap = backward ? 4 : 8;
  int MB = 1;
  while (MB < mb_cap && (B + 16 * MB - 1) / (16 * MB) > max_ns) MB *= 2;
  while (MB > 1 && persist_lds_bytes(H, backward, MB) > 160 * 1024) MB /= 2;
  *MBo = MB;
  *chunko = std::min(B, max_ns * 16 * MB);
  return true;
}

bool persist_bwd_needs_wt(int H, int B) {
  int MB, chunk;
  return !persist_plan(true, H, B, &MB, &chunk) || MB > 1;
}

hipError_t persist_clear(bool backward, const PersistArgs& a, hipStream_t s) {
  int MB, chunk;
  if (!persist_plan(backward, a.H, a.B, &MB, &chunk)) return hipErrorInvalidValue;
  // both exchange slots start without any valid step number; the forward's
  // clear also initialises the status block of a fresh workspace
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
  if (!persist_plan(backward, a.H, a.B, &MB, &chunk)) return hipErrorInvalidValue;
  for (int b0 = 0; b0 < a.B; b0 += chunk) {
    PersistArgs c = a;
    c.b0 = b0;
    c.rows = std::min(chunk, a.B - b0);
    c.NS = (c.rows + 16 * MB - 1) / (16 * MB);
    // the launch's position in the call (the caller's tag numbers the layers
    // in the order the call runs them)
    c.seq = a.tag * (uint32_t)cdiv(a.B, chunk) + (uint32_t)(b0 / chunk);
    hipError_t e;
    if (backward)
      e = MB == 1 ? launch_one<1, true>(c, s) : MB == 2 ? launch_one<2, true>(c, s) : launch_one<4, true>(c, s);
    else
      e = MB == 1 ? launch_one<1, false>(c, s) : MB == 2 ? launch_one<2, false>(c, s)
                  : MB == 4 ? launch_one<4, false>(c, s) : launch_one<8, false>(c, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}
