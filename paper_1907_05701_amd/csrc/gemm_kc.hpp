// bf16 GEMM with both operands K-contiguous (C[m][n] = sum_k A[m][k] B[n][k]),
// the layout every product of the learner step is brought into.
//
// Global -> LDS moves use gfx950's direct-to-LDS buffer loads
// (buffer_load_dwordx4 ... lds): each lane's 16 bytes land in LDS at the
// wave's base + 16 * lane, without passing through registers, so several
// k-tiles can be in flight (STAGES-deep LDS ring) at no register cost.  A
// k-tile is 64 deep: every tile row is 128 bytes = 8 chunks of 8 k values,
// and one load instruction fills 8 rows (lane i: row i/8, slot i%8).  Chunk c
// of row r sits in slot c ^ swz(r), so the 16 lanes that read one MFMA
// fragment (16 rows, one chunk) hit distinct bank groups.  Rows beyond the
// operand and k beyond the range end are fetched with an out-of-range buffer
// offset, which the hardware returns as zeros.
//
// Per k-tile each workgroup waits for its own oldest tile (vmcnt), meets at
// one barrier (which also retires the previous tile's LDS reads), refills the
// slot freed by the previous tile and multiplies the current one.
#pragma once

#include "gemm.hpp"
#include "dma.hpp"

struct KcArgs {
  const bf16* A;
  int64_t lda, azs, arows;   // A rows m (< arows valid), batch stride azs
  const bf16* B;
  int64_t ldb, bzs, brows;
  int64_t M, N, K, ksplit;   // k range of split s: [s*ksplit, min(K, (s+1)*ksplit))
  int splits, ntm, ntn;      // tiles along m and n
  int gm;                    // tile rows per group of the XCD-aware order
  int total;                 // workgroups = batches * splits * ntm * ntn
};

// Workgroup w runs on XCD w % 8.  The first 8*(total/8) workgroups are dealt
// so that XCD x takes logical tiles [x*q, (x+1)*q) in order; logical tiles
// run in groups of `gm` tile rows with the rows fastest, so the workgroups an
// XCD holds at once cover a compact block of A and B rows (L2 reuse).
__device__ __forceinline__ void kc_tile_of(const KcArgs& p, int w, int& zs, int& tm, int& tn) {
  const int q = p.total / 8;
  const int L = w < 8 * q ? (w % 8) * q + w / 8 : w;
  const int per = p.ntm * p.ntn;
  zs = L / per;
  const int t = L % per;
  const int grp = t / (p.gm * p.ntn);
  const int gm = min(p.gm, p.ntm - grp * p.gm);
  const int in = t - grp * p.gm * p.ntn;
  tm = grp * p.gm + in % gm;
  tn = in / gm;
}

template <int BM_, int BN_, int WM_, int WN_, int STAGES_, int BK_ = 64>
struct KcCfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, STAGES = STAGES_, BK = BK_;
  static constexpr size_t lds_bytes = (size_t)STAGES * (BM + BN) * BK * 2;
};

// Slot of 16-byte chunk c in tile row r.  The 16 lanes reading one fragment
// (rows r0..r0+15, one chunk) land in distinct bank groups both when the LDS
// serves 8 lanes of a b128 read per clock (128-byte window) and when it
// serves 16 (256-byte window).  64-deep tiles: 8 chunks per 128-byte row;
// 32-deep tiles: 4 chunks per 64-byte row.
template <int BK>
__device__ __forceinline__ int kc_slot(int c, int r) {
  if constexpr (BK == 64) return c ^ ((r >> 1) & 7) ^ ((r & 1) << 2);
  else return c ^ ((((r >> 1) ^ (r >> 3)) & 1) | (((r >> 2) & 1) << 1));
}

template <int N>
__device__ __forceinline__ void kc_wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

__device__ __forceinline__ void kc_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int BM, int BN, int WM, int WN, int STAGES, int BK, class Epi>
__global__ __launch_bounds__(WM * WN * 64) void gemm_kc_kernel(const KcArgs p, const Epi epi) {
  constexpr int NW = WM * WN;
  constexpr int ROWB = BK * 2, CPR = BK / 8, RPI = 64 / CPR;   // row bytes, chunks per row, rows per load
  constexpr int FM = BM / WM / 16, FN = BN / WN / 16;
  constexpr int LA = BM / RPI / NW, LB = BN / RPI / NW;   // load instructions per wave per k-tile
  static_assert(BK == 32 || BK == 64, "k-tile depth");
  static_assert(LA >= 1 && LB >= 1 && BM % (RPI * NW) == 0 && BN % (RPI * NW) == 0,
                "tile rows must split over the waves");
  constexpr int STAGE = (BM + BN) * ROWB;
  extern __shared__ __attribute__((aligned(1024))) char kc_lds[];

  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int wm = wid % WM, wn = wid / WM;
  int zs, tm, tn;
  kc_tile_of(p, blockIdx.x, zs, tm, tn);
  const int z = zs / p.splits, sp = zs % p.splits;
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  const int64_t kbeg = (int64_t)sp * p.ksplit;
  const int64_t kend = min(p.K, kbeg + p.ksplit);
  const int ntiles = kend > kbeg ? (int)((kend - kbeg + BK - 1) / BK) : 0;

  // buffer resources based at this tile's first row (offsets stay < 2 GiB)
  const bf16* abase = p.A + (int64_t)z * p.azs + m0 * p.lda;
  const bf16* bbase = p.B + (int64_t)z * p.bzs + n0 * p.ldb;
  const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc((void*)abase, (short)0, 0x7ffffff0, 0x00020000);
  const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc((void*)bbase, (short)0, 0x7ffffff0, 0x00020000);
  const int64_t arows = min((int64_t)BM, p.arows - m0), brows = min((int64_t)BN, p.brows - n0);

  // per lane: row within the rows of one load and the slot it fills
  const int lr = lane / CPR, ls = lane % CPR;
  auto issue = [&](int j) {
    const int64_t k0 = kbeg + (int64_t)j * BK;
    char* st = kc_lds + (j % STAGES) * STAGE;
#pragma unroll
    for (int q = 0; q < LA; ++q) {
      const int r = (q * NW + wid) * RPI + lr;
      const int c = kc_slot<BK>(ls, r);   // slot ls holds chunk c (kc_slot is an involution in c)
      const int64_t k = k0 + c * 8;
      const uint32_t off = (r < arows && k < kend) ? (uint32_t)((r * p.lda + k) * 2) : 0x80000000u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_ptr_t)(st + (q * NW + wid) * 1024), 16, off, 0, 0, 0);
    }
#pragma unroll
    for (int q = 0; q < LB; ++q) {
      const int r = (q * NW + wid) * RPI + lr;
      const int c = kc_slot<BK>(ls, r);
      const int64_t k = k0 + c * 8;
      const uint32_t off = (r < brows && k < kend) ? (uint32_t)((r * p.ldb + k) * 2) : 0x80000000u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_ptr_t)(st + BM * ROWB + (q * NW + wid) * 1024), 16, off, 0,
                                               0, 0);
    }
  };

  f32x4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int fr = lane & 15, fc = lane >> 4;   // fragment row, chunk within a 32-k step
  auto compute = [&](int j) {
    const char* st = kc_lds + (j % STAGES) * STAGE;
    const char* la = st + (wm * (BM / WM) + fr) * ROWB;
    const char* lb = st + BM * ROWB + (wn * (BN / WN) + fr) * ROWB;
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      const int slot = kc_slot<BK>(ks * 4 + fc, fr) * 16;   // row offsets below are multiples of 16
      bf16x8 a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) a[i] = *(const bf16x8*)(la + i * 16 * ROWB + slot);
#pragma unroll
      for (int jn = 0; jn < FN; ++jn) b[jn] = *(const bf16x8*)(lb + jn * 16 * ROWB + slot);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int jn = 0; jn < FN; ++jn) acc[i][jn] = Mfma<bf16>::mma(a[i], b[jn], acc[i][jn]);
    }
  };

#pragma unroll
  for (int j = 0; j < STAGES - 1; ++j)
    if (j < ntiles) issue(j);
  for (int it = 0; it < ntiles; ++it) {
    if (it + STAGES - 2 < ntiles)
      kc_wait_vm<(STAGES - 2) * (LA + LB)>();
    else
      kc_wait_vm<0>();
    kc_barrier();
    if (it + STAGES - 1 < ntiles) issue(it + STAGES - 1);
    compute(it);
  }
  epi.template apply<FM, FN>(z, sp, m0 + wm * (BM / WM), n0 + wn * (BN / WN), acc, lane);
}

// Whether an operand can go through the direct-to-LDS path: plain rows
// (no segments or gate interleave), 16-byte aligned rows and batch strides.
static inline bool kc_operand_ok(const Opnd& o, int64_t K) {
  return o.seg == 0 && o.ilH == 0 && o.ld % 8 == 0 && o.zstride % 8 == 0 &&
         ((uintptr_t)o.base & 15) == 0 && o.ext >= K;
}

static int kc_group_rows = 4;   // measured best at the learner-step shapes

template <class C, class Epi>
static inline void gemm_kc_launch(const char* name, hipStream_t s, const Opnd& A, const Opnd& B, int64_t M,
                                  int64_t N, int64_t K, int batches, int splits, const Epi& epi) {
  KcArgs p;
  p.A = (const bf16*)A.base; p.lda = A.ld; p.azs = A.zstride; p.arows = std::min(A.rows, M);
  p.B = (const bf16*)B.base; p.ldb = B.ld; p.bzs = B.zstride; p.brows = std::min(B.rows, N);
  p.M = M; p.N = N; p.K = K;
  p.ksplit = splits > 1 ? rup(cdiv(K, splits), C::BK) : (K > 0 ? K : 1);
  p.splits = splits;
  p.ntn = (int)cdiv(N, C::BN);
  p.ntm = (int)cdiv(M, C::BM);
  p.gm = kc_group_rows;
  p.total = batches * splits * p.ntm * p.ntn;
  auto fn = gemm_kc_kernel<C::BM, C::BN, C::WM, C::WN, C::STAGES, C::BK, Epi>;
  static bool attr_set = false;   // raising the LDS limit is per function, once
  if (!attr_set) {
    (void)hipFuncSetAttribute((const void*)fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)C::lds_bytes);
    attr_set = true;
  }
  BLSTM_LAUNCH(name, fn, dim3((unsigned)p.total), dim3(C::WM * C::WN * 64),
               C::lds_bytes, s, p, epi);
}

// Tile shape of the direct-to-LDS kernel (measured on MI355X at the
// learner-step shapes, against 256x256 blocks, 32-deep tiles and deeper
// rings): 128x128 blocks of 8 waves (64x32 each), two 64-deep stages, two
// blocks per CU.
typedef KcCfg<128, 128, 2, 4, 2> KcTile;

// GEMM dispatch: bf16 K-contiguous operands with 16-byte aligned rows go to
// the direct-to-LDS kernel, everything else to the generic kernel.
template <typename T, bool AKC, bool BKC, int VA, int VB, class Epi>
static inline void gemm_launch(const char* name, hipStream_t s, const Opnd& A, const Opnd& B,
                               int64_t M, int64_t N, int64_t K, int batches, int splits,
                               const Epi& epi) {
  if constexpr (std::is_same<T, bf16>::value && AKC && BKC) {
    if (K % 8 == 0 && kc_operand_ok(A, K) && kc_operand_ok(B, K)) {
      gemm_kc_launch<KcTile>(name, s, A, B, M, N, K, batches, splits, epi);
      return;
    }
    gemm_launch_cfg<T, GemmCfgK32, AKC, BKC, VA, VB>(name, s, A, B, M, N, K, batches, splits, epi);
    return;
  }
  gemm_launch_cfg<T, GemmCfg<T>, AKC, BKC, VA, VB>(name, s, A, B, M, N, K, batches, splits, epi);
}
