// Persistent recurrent kernels (bf16 operands): one cooperative launch runs
// all T steps of one layer, for both directions at once, with each
// workgroup's slice of W_hh held in LDS for the whole chunk.
//
// Work split.  The batch is cut into slices of 16*MB rows; a group of
// H/32 workgroups owns one (direction, slice) pair and each member owns 32
// hidden units (two blocks of 16).  Its four waves are (unit block, half):
// the half splits the reduction dimension when MB == 1 and the m-blocks
// otherwise.  Per step a member
//   forward : reads h_prev of its slice (all H units) from global memory,
//             multiplies by its LDS-resident W_hh rows (4 gates x 32 units),
//             adds the precomputed input projection and applies the cell;
//             c stays in registers, h/c/gates are written for BPTT;
//   backward: reads da of the previously processed step (all 4H gate
//             columns), multiplies by its LDS-resident W_hh columns to get
//             dh_rec for its units, applies the gate derivatives (dc stays in
//             registers) and writes da of this step.
// Steps are separated by a per-group barrier: each wave drains its stores,
// one thread per workgroup issues an agent-scope release fence and an atomic
// arrival, and one thread spins (bounded) on the group counter and issues the
// agent-scope acquire fence before the workgroup barrier releases the rest.  The launch is cooperative, so
// all workgroups are co-resident; the spin bound only guarantees that every
// wave exits even if that guarantee were broken (the status word is set).
// Group g's members are workgroups g, g+NG, g+2NG, ... with NG a multiple of
// 8, which keeps a group on one XCD when workgroups are dealt round-robin.
#include "common.hpp"
#include "lstm_persist.hpp"

#define PU 32
#define SPIN_LIMIT (1u << 22)
#define CTR_STRIDE 32

// Arrival: every wave first waits until its own stores are complete at the
// L2, the workgroup barrier joins the waves, and one thread then makes the
// workgroup's writes visible at agent scope and counts the arrival.
__device__ __forceinline__ void group_arrive(unsigned* ctr) {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Wait: one thread spins on the counter, then invalidates this CU's caches
// at agent scope before the barrier releases the other waves to read.
__device__ __forceinline__ void group_wait(unsigned* ctr, unsigned target, int* status) {
  if (threadIdx.x == 0) {
    unsigned it = 0;
    while (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      __builtin_amdgcn_s_sleep(1);
      if (++it > SPIN_LIMIT) {
        __hip_atomic_store(status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  }
  __syncthreads();
}

__device__ __forceinline__ bf16x8 ld16(const bf16* p) { return *(const bf16x8*)p; }

// 8x8 bf16 transpose: in[i] holds row i (8 values); out[j] gets column j.
__device__ __forceinline__ void transpose8x8(const uint4 (&in)[8], uint4 (&out)[8]) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    uint32_t o4[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t lo = ((const uint32_t*)&in[2 * w])[j / 2];
      const uint32_t hi = ((const uint32_t*)&in[2 * w + 1])[j / 2];
      o4[w] = (j & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
    }
    out[j] = make_uint4(o4[0], o4[1], o4[2], o4[3]);
  }
}

// ---------------------------------------------------------------------------
// Forward.
// ---------------------------------------------------------------------------
template <int MB>
__global__ __launch_bounds__(256) void lstm_fwd_persist(const PersistArgs a) {
  extern __shared__ __attribute__((aligned(16))) bf16 lds[];
  constexpr bool KSPLIT = MB == 1;
  constexpr int MBW = KSPLIT ? 1 : MB / 2;
  constexpr int LDN = 128 + 1;   // LDS rows per k-group (128 gate rows + pad)
  const int H = a.H, B = a.B, Tn = a.Tn;
  const int NM = H / PU, NG = 2 * a.NS;
  const int g = blockIdx.x % NG, mem = blockIdx.x / NG;
  const int d = g & 1, s = g >> 1;
  const int u0 = mem * PU;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int ub = w & 1, wx = w >> 1;

  // W_hh rows of this member: LDS row n = ub*64 + gate*16 + u
  const bf16* Wd = a.W + (d ? a.whh1 : a.whh0);
  const int kcn = H / 8;
  for (int c = tid; c < 128 * kcn; c += 256) {
    const int n = c / kcn, kc = c % kcn;
    const int64_t row = (int64_t)((n >> 4) & 3) * H + u0 + (n >> 6) * 16 + (n & 15);
    *(uint4*)&lds[(kc * LDN + n) * 8] = *(const uint4*)(Wd + row * H + kc * 8);
  }
  f32x4* red = (f32x4*)(lds + (size_t)kcn * LDN * 8);
  __syncthreads();

  const int rend = a.b0 + a.rows;
  const int rowbase = a.b0 + s * 16 * MB;
  const int mb0 = KSPLIT ? 0 : wx * MBW;
  const bool epi = !KSPLIT || wx == 0;
  const int unit = u0 + ub * 16 + (lane & 15);
  const int nks = H / 32;
  const int ks_beg = KSPLIT ? (wx ? nks / 2 : 0) : 0;
  const int ks_end = KSPLIT ? (wx ? nks : nks / 2) : nks;
  unsigned* ctr = a.ctr + g * CTR_STRIDE;

  float creg[MBW][4];
#pragma unroll
  for (int m = 0; m < MBW; ++m)
#pragma unroll
    for (int r = 0; r < 4; ++r) creg[m][r] = 0.f;

  for (int tau = 0; tau < Tn; ++tau) {
    const int t = d ? Tn - 1 - tau : tau;
    const int tp = d ? t + 1 : t - 1;
    // input projection of this step for the epilogue (independent of h)
    float gx[MBW][4][4];
    if (epi) {
#pragma unroll
      for (int m = 0; m < MBW; ++m)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = rowbase + (mb0 + m) * 16 + (lane >> 4) * 4 + r;
          const bf16* p = a.Gx + ((int64_t)t * B + (row < rend ? row : a.b0)) * 8 * H + (int64_t)d * 4 * H + unit;
#pragma unroll
          for (int q = 0; q < 4; ++q) gx[m][r][q] = (float)p[q * H];
        }
    }
    if (tau > 0) group_wait(ctr, (unsigned)(NM * tau), a.status);

    f32x4 acc[MBW][4];
#pragma unroll
    for (int m = 0; m < MBW; ++m)
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[m][q] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (tau > 0) {
      const bf16* arow[MBW];
      bool rowok[MBW];
#pragma unroll
      for (int m = 0; m < MBW; ++m) {
        const int row = rowbase + (mb0 + m) * 16 + (lane & 15);
        rowok[m] = row < rend;
        arow[m] = a.Y + ((int64_t)tp * B + (rowok[m] ? row : a.b0)) * 2 * H + (int64_t)d * H + (lane >> 4) * 8;
      }
#pragma unroll 4
      for (int ks = ks_beg; ks < ks_end; ++ks) {
        bf16x8 af[MBW];
#pragma unroll
        for (int m = 0; m < MBW; ++m) af[m] = rowok[m] ? ld16(arow[m] + ks * 32) : bf16x8{};
        const int kg = ks * 4 + (lane >> 4);
        bf16x8 bfr[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) bfr[q] = *(const bf16x8*)&lds[(kg * LDN + ub * 64 + q * 16 + (lane & 15)) * 8];
#pragma unroll
        for (int m = 0; m < MBW; ++m)
#pragma unroll
          for (int q = 0; q < 4; ++q) acc[m][q] = Mfma<bf16>::mma(af[m], bfr[q], acc[m][q]);
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
#pragma unroll
      for (int m = 0; m < MBW; ++m)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = rowbase + (mb0 + m) * 16 + (lane >> 4) * 4 + r;
          if (row >= rend) continue;
          const float ig = sigmoidf_(acc[m][0][r] + gx[m][r][0]);
          const float fg = sigmoidf_(acc[m][1][r] + gx[m][r][1]);
          const float gg = tanhf_(acc[m][2][r] + gx[m][r][2]);
          const float og = sigmoidf_(acc[m][3][r] + gx[m][r][3]);
          const float c = fg * creg[m][r] + ig * gg;
          creg[m][r] = c;
          const float h = og * tanhf_(c);
          const int64_t fr = (int64_t)t * B + row;
          a.C[fr * 2 * H + (int64_t)d * H + unit] = c;
          a.Y[fr * 2 * H + (int64_t)d * H + unit] = (bf16)h;
          bf16* gs = a.G + fr * 8 * H + (int64_t)d * 4 * H + unit;
          gs[0] = (bf16)ig;
          gs[H] = (bf16)fg;
          gs[2 * H] = (bf16)gg;
          gs[3 * H] = (bf16)og;
        }
    }
    group_arrive(ctr);
  }
}

// ---------------------------------------------------------------------------
// Backward (BPTT).
// ---------------------------------------------------------------------------
template <int MB>
__global__ __launch_bounds__(256) void lstm_bwd_persist(const PersistArgs a) {
  extern __shared__ __attribute__((aligned(16))) bf16 lds[];
  constexpr bool KSPLIT = MB == 1;
  constexpr int MBW = KSPLIT ? 1 : MB / 2;
  constexpr int LDN = PU + 1;    // LDS rows per k-group (32 units + pad)
  const int H = a.H, B = a.B, Tn = a.Tn;
  const int NM = H / PU, NG = 2 * a.NS;
  const int g = blockIdx.x % NG, mem = blockIdx.x / NG;
  const int d = g & 1, s = g >> 1;
  const int u0 = mem * PU;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int ub = w & 1, wx = w >> 1;

  // W_hh columns of this member, transposed: LDS element (k = gate row, n = unit)
  const bf16* Wd = a.W + (d ? a.whh1 : a.whh0);
  const int nblk = (4 * H / 8) * (PU / 8);
  for (int b = tid; b < nblk; b += 256) {
    const int kgrp = b / (PU / 8), nb = b % (PU / 8);
    uint4 in[8], out[8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
      in[i] = *(const uint4*)(Wd + (int64_t)(kgrp * 8 + i) * H + u0 + nb * 8);
    transpose8x8(in, out);
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) *(uint4*)&lds[(kgrp * LDN + nb * 8 + jj) * 8] = out[jj];
  }
  f32x4* red = (f32x4*)(lds + (size_t)(4 * H / 8) * LDN * 8);
  __syncthreads();

  const int rend = a.b0 + a.rows;
  const int rowbase = a.b0 + s * 16 * MB;
  const int mb0 = KSPLIT ? 0 : wx * MBW;
  const bool epi = !KSPLIT || wx == 0;
  const int unit = u0 + ub * 16 + (lane & 15);
  const int nks = 4 * H / 32;
  const int ks_beg = KSPLIT ? (wx ? nks / 2 : 0) : 0;
  const int ks_end = KSPLIT ? (wx ? nks : nks / 2) : nks;
  unsigned* ctr = a.ctr + g * CTR_STRIDE;

  float dcreg[MBW][4];
#pragma unroll
  for (int m = 0; m < MBW; ++m)
#pragma unroll
    for (int r = 0; r < 4; ++r) dcreg[m][r] = 0.f;

  for (int tau = 0; tau < Tn; ++tau) {
    const int t = d ? tau : Tn - 1 - tau;
    const int tn = d ? t - 1 : t + 1;
    const int tp = d ? t + 1 : t - 1;
    const bool has_prev = tp >= 0 && tp < Tn;
    // everything the cell derivative needs besides dh_rec
    float dy[MBW][4], gt[MBW][4][4], cc[MBW][4], cp[MBW][4];
    if (epi) {
#pragma unroll
      for (int m = 0; m < MBW; ++m)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          int row = rowbase + (mb0 + m) * 16 + (lane >> 4) * 4 + r;
          row = row < rend ? row : a.b0;
          const int64_t fr = (int64_t)t * B + row;
          dy[m][r] = a.DY[fr * 2 * H + (int64_t)d * H + unit];
          cc[m][r] = a.C[fr * 2 * H + (int64_t)d * H + unit];
          cp[m][r] = has_prev ? a.C[((int64_t)tp * B + row) * 2 * H + (int64_t)d * H + unit] : 0.f;
          const bf16* gs = a.G + fr * 8 * H + (int64_t)d * 4 * H + unit;
#pragma unroll
          for (int q = 0; q < 4; ++q) gt[m][r][q] = (float)gs[q * H];
        }
    }
    if (tau > 0) group_wait(ctr, (unsigned)(NM * tau), a.status);

    f32x4 acc[MBW];
#pragma unroll
    for (int m = 0; m < MBW; ++m) acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (tau > 0) {
      const bf16* arow[MBW];
      bool rowok[MBW];
#pragma unroll
      for (int m = 0; m < MBW; ++m) {
        const int row = rowbase + (mb0 + m) * 16 + (lane & 15);
        rowok[m] = row < rend;
        arow[m] = a.DA + ((int64_t)tn * B + (rowok[m] ? row : a.b0)) * 8 * H + (int64_t)d * 4 * H + (lane >> 4) * 8;
      }
#pragma unroll 4
      for (int ks = ks_beg; ks < ks_end; ++ks) {
        bf16x8 af[MBW];
#pragma unroll
        for (int m = 0; m < MBW; ++m) af[m] = rowok[m] ? ld16(arow[m] + ks * 32) : bf16x8{};
        const int kg = ks * 4 + (lane >> 4);
        const bf16x8 bfr = *(const bf16x8*)&lds[(kg * LDN + ub * 16 + (lane & 15)) * 8];
#pragma unroll
        for (int m = 0; m < MBW; ++m) acc[m] = Mfma<bf16>::mma(af[m], bfr, acc[m]);
      }
    }
    if (KSPLIT) {
      if (wx == 1) red[ub * 64 + lane] = acc[0];
      __syncthreads();
      if (wx == 0) acc[0] += red[ub * 64 + lane];
    }
    if (epi) {
#pragma unroll
      for (int m = 0; m < MBW; ++m)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = rowbase + (mb0 + m) * 16 + (lane >> 4) * 4 + r;
          if (row >= rend) continue;
          const float ig = gt[m][r][0], fg = gt[m][r][1], gg = gt[m][r][2], og = gt[m][r][3];
          const float dh = acc[m][r] + dy[m][r];
          const float tc = tanhf_(cc[m][r]);
          const float dc = dh * og * (1.f - tc * tc) + dcreg[m][r];
          dcreg[m][r] = dc * fg;
          bf16* da = a.DA + ((int64_t)t * B + row) * 8 * H + (int64_t)d * 4 * H + unit;
          da[0] = (bf16)(dc * gg * ig * (1.f - ig));
          da[H] = (bf16)(dc * cp[m][r] * fg * (1.f - fg));
          da[2 * H] = (bf16)(dc * ig * (1.f - gg * gg));
          da[3 * H] = (bf16)(dh * tc * og * (1.f - og));
        }
    }
    group_arrive(ctr);
  }
}

__global__ void zero_u32_kernel(unsigned* p, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0u;
}

// ---------------------------------------------------------------------------
// Host side.
// ---------------------------------------------------------------------------
size_t persist_lds_bytes(int H, bool backward) {
  if (backward) return (size_t)(4 * H / 8) * (PU + 1) * 16 + 2 * 64 * 16;
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

bool persist_supported(int H) {
  return H % PU == 0 && persist_lds_bytes(H, false) <= 160 * 1024 &&
         persist_lds_bytes(H, true) <= 160 * 1024;
}

template <int MB>
static hipError_t launch_one(bool backward, PersistArgs a, hipStream_t s) {
  const void* fn = backward ? (const void*)lstm_bwd_persist<MB> : (const void*)lstm_fwd_persist<MB>;
  const size_t lds = persist_lds_bytes(a.H, backward);
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  const dim3 grid(2 * a.NS * (a.H / PU)), block(256);
  void* args[] = {&a};
  const char* name = backward ? "lstm_rec_bwd_persist" : "lstm_rec_fwd_persist";
  const int slot = g_timing_on ? timing_pre(name, s) : -1;
  e = hipLaunchCooperativeKernel(fn, grid, block, args, (unsigned)lds, s);
  if (slot >= 0) timing_post(slot, s);
  return e;
}

// Runs all steps of one layer (both directions); returns hipSuccess or the
// launch error (nothing was enqueued for the failing chunk in that case).
hipError_t persist_layer(bool backward, PersistArgs a, hipStream_t s) {
  const int NM = a.H / PU;
  const int max_ns = std::min(persist_max_wg() / (2 * NM), 32);
  if (max_ns < 1) return hipErrorInvalidValue;
  int MB = 1;
  while (MB < 8 && (a.B + 16 * MB - 1) / (16 * MB) > max_ns) MB *= 2;
  const int chunk = std::min(a.B, max_ns * 16 * MB);
  for (int b0 = 0; b0 < a.B; b0 += chunk) {
    PersistArgs c = a;
    c.b0 = b0;
    c.rows = std::min(chunk, a.B - b0);
    c.NS = (c.rows + 16 * MB - 1) / (16 * MB);
    // counters and the status word are contiguous
    hipLaunchKernelGGL(zero_u32_kernel, dim3(1), dim3(256), 0, s, c.ctr, PERSIST_CTR_BYTES / 4 + 1);
    hipError_t e;
    switch (MB) {
      case 1: e = launch_one<1>(backward, c, s); break;
      case 2: e = launch_one<2>(backward, c, s); break;
      case 4: e = launch_one<4>(backward, c, s); break;
      default: e = launch_one<8>(backward, c, s); break;
    }
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}
