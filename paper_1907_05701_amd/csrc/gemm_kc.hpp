// bf16 GEMM C[m][n] = sum_k A(m, k) B(n, k) with each operand K-contiguous
// (element (mn, k) at mn*ld + k) or MN-contiguous (at k*ld + mn), so that the
// learner step's products read their operands as they lie.
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
// An MN-contiguous operand (element (mn, k) at k*ld + mn) is staged as it
// lies: LDS rows of one k, 256 bytes (128 mn) each, one load instruction
// filling 4 rows, chunk c of row k in slot c ^ mn_swz(k).  Its MFMA fragments
// come from gfx950's transposing LDS read (ds_read_b64_tr_b16): within each
// 16-lane group, lane r points at 4 consecutive mn of k row r/4 and the
// instruction hands lane i the 4 values of mn column i over those 4 k rows
// (lane i, element j = lane 4j + i/4's element i%4).  Two such reads give a
// lane its 8 consecutive k.  Such an operand may also come in k segments (a
// power of two of rows, whole k-tiles, at a fixed stride): the two direction
// blocks of W_ih.
//
// Per k-tile each workgroup waits for its own oldest tile (vmcnt), meets at
// one barrier (which also retires the previous tile's LDS reads), refills the
// slot freed by the previous tile and multiplies the current one.
#pragma once

#include <atomic>
#include <cstring>

#include "gemm.hpp"
#include "dma.hpp"

struct KcArgs {
  const bf16* A;
  int64_t lda, azs, arows;   // A rows m (< arows valid), batch stride azs
  int asegsh;                // MN-contiguous A: k rows in segments of 2^asegsh (0: one segment) ...
  int64_t asegs;             // ... whose starts are asegs elements apart
  const bf16* B;
  int64_t ldb, bzs, brows;
  int bsegsh;
  int64_t bsegs;
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

// Slot of 16-byte chunk c (8 mn) in k row r of an MN-contiguous tile (16
// chunks per 256-byte row): the 16 k rows one transposing read touches
// (r & 3 and bit 3 of r vary) take distinct chunk pairs.
__device__ __forceinline__ int mn_slot(int c, int r) { return c ^ (2 * ((r & 3) | (((r >> 3) & 1) << 2))); }

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

template <int N>
__device__ __forceinline__ void kc_wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

__device__ __forceinline__ void kc_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Transposing LDS read (ds_read_b64_tr_b16) as inline asm.  The compiler's
// own form of this read is made to wait for every direct-to-LDS load in
// flight (vmcnt(0)), since it cannot tell which LDS bytes they write; here
// that wait would take the next k-tile's loads out of the overlap.  The loop
// already orders the reads after the current tile's loads (its own vmcnt wait
// and the barrier); kc_lds_wait() gives the results back to the compiler.
__device__ __forceinline__ bf16x4 kc_read_tr(const char* p) {
  const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
  bf16x4 v;
  asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(v) : "v"(a));
  return v;
}

template <int N>
__device__ __forceinline__ void kc_lds_wait(bf16x8 (&f)[N]) {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : "+v"(f[i]));
}

// Staging and fragment reads of one operand (rows BMN of the tile's M or N
// side, BK deep), K-contiguous (KC) or MN-contiguous.
template <bool KC, int BMN, int BK, int NW>
struct KcOperand {
  static constexpr int ROWB = KC ? BK * 2 : BMN * 2;        // LDS row bytes
  static constexpr int CPR = ROWB / 16;                     // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;                      // rows per load instruction
  static constexpr int LOADS = (KC ? BMN : BK) / RPI / NW;  // load instructions per wave per k-tile
  static_assert(LOADS >= 1 && (KC ? BMN : BK) % (RPI * NW) == 0, "tile rows must split over the waves");
  static_assert(KC || BMN == 128, "MN-contiguous tiles are 128 wide");

  // base: the operand's batch base; mn0: tile's first MN row; ld: row pitch;
  // mnrows: valid MN rows of this tile (KC) / MN extent left (MNC); segsh,
  // segs: k rows of an MNC operand in segments of 2^segsh rows (at least BK,
  // so no k-tile straddles two) whose starts are segs apart, or segsh = 0
  __device__ __forceinline__ static void issue(const bf16* base, int64_t ld, int segsh, int64_t segs, int64_t mn0,
                                               int64_t mnrows, int64_t k0, int64_t kend, char* tile, int wid,
                                               int lane) {
    if constexpr (KC) {
      const __amdgpu_buffer_rsrc_t r = dma_rsrc(base + mn0 * ld);
      const int lr = lane / CPR, ls = lane % CPR;
#pragma unroll
      for (int q = 0; q < LOADS; ++q) {
        const int row = (q * NW + wid) * RPI + lr;
        const int c = kc_slot<BK>(ls, row);   // slot ls holds chunk c (kc_slot is an involution in c)
        const int64_t k = k0 + c * 8;
        const uint32_t off = (row < mnrows && k < kend) ? (uint32_t)((row * ld + k) * 2) : DMA_OFF_NONE;
        dma16(r, off, tile + (q * NW + wid) * 1024);
      }
    } else {
      // per-k-tile base keeps the offsets small for long operands
      const int64_t kb = segsh ? (k0 >> segsh) * segs + (k0 & ((1LL << segsh) - 1)) * ld : k0 * ld;
      const __amdgpu_buffer_rsrc_t r = dma_rsrc(base + kb + mn0);
      const int lr = lane / CPR, ls = lane % CPR;
#pragma unroll
      for (int q = 0; q < LOADS; ++q) {
        const int row = (q * NW + wid) * RPI + lr;   // k row within the tile
        const int c = mn_slot(ls, row);
        const bool ok = k0 + row < kend && c * 8 + 8 <= mnrows;
        dma16(r, ok ? (uint32_t)((row * ld + c * 8) * 2) : DMA_OFF_NONE, tile + (q * NW + wid) * 1024);
      }
    }
  }

  // MFMA fragment (16 MN rows from mnb, 8 consecutive k of 32-k step ks)
  __device__ __forceinline__ static bf16x8 frag(const char* tile, int mnb, int ks, int lane) {
    if constexpr (KC) {
      const int fr = lane & 15, fc = lane >> 4;
      return *(const bf16x8*)(tile + (mnb + fr) * ROWB + kc_slot<BK>(ks * 4 + fc, fr) * 16);
    } else {
      const int g = lane >> 4, r = lane & 15;
      const int mn = mnb + 4 * (r & 3);
      bf16x4 h[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int k = ks * 32 + 8 * g + 4 * hh + (r >> 2);
        const char* pa = tile + k * ROWB + mn_slot(mn >> 3, k) * 16 + (mn & 7) * 2;
        h[hh] = kc_read_tr(pa);
      }
      return bf16x8{h[0][0], h[0][1], h[0][2], h[0][3], h[1][0], h[1][1], h[1][2], h[1][3]};
    }
  }
};

// One output tile of one product; w is the workgroup's index within the
// product's workgroups (those at or past p.total have no tile).
template <int BM, int BN, int WM, int WN, int STAGES, int BK, bool AKC, bool BKC, class Epi>
__device__ __forceinline__ void kc_gemm_tile(const KcArgs& p, const Epi& epi, int w) {
  constexpr int NW = WM * WN;
  constexpr int FM = BM / WM / 16, FN = BN / WN / 16;
  typedef KcOperand<AKC, BM, BK, NW> OA;
  typedef KcOperand<BKC, BN, BK, NW> OB;
  static_assert(BK == 32 || BK == 64, "k-tile depth");
  constexpr int TA = BM * BK * 2, STAGE = (BM + BN) * BK * 2;
  extern __shared__ __attribute__((aligned(1024))) char kc_lds[];

  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int wm = wid % WM, wn = wid / WM;
  if (w >= p.total) return;
  int zs, tm, tn;
  kc_tile_of(p, w, zs, tm, tn);
  const int z = zs / p.splits, sp = zs % p.splits;
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  const int64_t kbeg = (int64_t)sp * p.ksplit;
  const int64_t kend = min(p.K, kbeg + p.ksplit);
  const int ntiles = kend > kbeg ? (int)((kend - kbeg + BK - 1) / BK) : 0;

  const bf16* abase = p.A + (int64_t)z * p.azs;
  const bf16* bbase = p.B + (int64_t)z * p.bzs;
  const int64_t arows = p.arows - m0, brows = p.brows - n0;   // valid MN rows from the tile start
  auto issue = [&](int j) {
    const int64_t k0 = kbeg + (int64_t)j * BK;
    char* st = kc_lds + (j % STAGES) * STAGE;
    OA::issue(abase, p.lda, p.asegsh, p.asegs, m0, arows, k0, kend, st, wid, lane);
    OB::issue(bbase, p.ldb, p.bsegsh, p.bsegs, n0, brows, k0, kend, st + TA, wid, lane);
  };

  f32x4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int j) {
    const char* st = kc_lds + (j % STAGES) * STAGE;
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      bf16x8 a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) a[i] = OA::frag(st, wm * (BM / WM) + i * 16, ks, lane);
#pragma unroll
      for (int jn = 0; jn < FN; ++jn) b[jn] = OB::frag(st + TA, wn * (BN / WN) + jn * 16, ks, lane);
      if constexpr (!AKC) kc_lds_wait(a);
      if constexpr (!BKC) kc_lds_wait(b);
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
      kc_wait_vm<(STAGES - 2) * (OA::LOADS + OB::LOADS)>();
    else
      kc_wait_vm<0>();
    kc_barrier();
    if (it + STAGES - 1 < ntiles) issue(it + STAGES - 1);
    compute(it);
  }
  if constexpr (EpiIsWorkgroup<Epi>::value)
    epi.template apply_wg<BM, WM, WN, FM, FN>(m0 + wm * (BM / WM), n0 + wn * (BN / WN), acc, lane, kc_lds, tn);
  else
    epi.template apply<FM, FN>(z, sp, m0 + wm * (BM / WM), n0 + wn * (BN / WN), acc, lane);
}

template <int BM, int BN, int WM, int WN, int STAGES, int BK, bool AKC, bool BKC, class Epi>
__global__ __launch_bounds__(WM * WN * 64, WM * WN / 2) void gemm_kc_kernel(const KcArgs p, const Epi epi) {
  kc_gemm_tile<BM, BN, WM, WN, STAGES, BK, AKC, BKC, Epi>(p, epi, blockIdx.x);
}

// Several independent products in one launch (fills the chip when each alone
// would not): product i owns workgroups [start[i], start[i+1]); every start is
// a multiple of 8 so that the XCD-aware tile order of each product holds.
#define KC_MAX_GROUP 12
template <class Epi>
struct KcGroup {
  KcArgs p[KC_MAX_GROUP];
  Epi e[KC_MAX_GROUP];
  int start[KC_MAX_GROUP + 1];
  int n;
};

template <int BM, int BN, int WM, int WN, int STAGES, int BK, bool AKC, bool BKC, class Epi>
__global__ __launch_bounds__(WM * WN * 64, WM * WN / 2) void gemm_kc_group_kernel(const KcGroup<Epi> g) {
  // the product index: every start compared at once (the loads are
  // independent, so they issue together)
  int i = 0;
#pragma unroll
  for (int k = 1; k < KC_MAX_GROUP; ++k) i += (k < g.n && (int)blockIdx.x >= g.start[k]);
  kc_gemm_tile<BM, BN, WM, WN, STAGES, BK, AKC, BKC, Epi>(g.p[i], g.e[i], (int)blockIdx.x - g.start[i]);
}

// Two independent products with different operand layouts in one launch
// (each alone would leave part of its last round of the chip idle): the
// first owns workgroups [0, n1) (n1 a multiple of 8), the second the rest.
template <int BM, int BN, int WM, int WN, int STAGES, int BK, bool AKC1, bool BKC1, bool AKC2, bool BKC2, class Epi>
__global__ __launch_bounds__(WM * WN * 64, WM * WN / 2) void gemm_kc_pair_kernel(const KcArgs p1, const Epi e1,
                                                                             const KcArgs p2, const Epi e2, int n1) {
  if ((int)blockIdx.x < n1)
    kc_gemm_tile<BM, BN, WM, WN, STAGES, BK, AKC1, BKC1, Epi>(p1, e1, (int)blockIdx.x);
  else
    kc_gemm_tile<BM, BN, WM, WN, STAGES, BK, AKC2, BKC2, Epi>(p2, e2, (int)blockIdx.x - n1);
}

// Whether an operand can go through the direct-to-LDS path: no gate
// interleave, 16-byte aligned rows and batch strides, the whole k range inside
// the operand; MN-contiguous operands also need an MN extent that is a
// multiple of 8 (whole 16-byte chunks), and may come in k segments of a power
// of two of at least 64 rows (whole k-tiles); K-contiguous ones may not be
// segmented.
static inline bool kc_operand_ok(const Opnd& o, int64_t K, bool kc) {
  const bool plain = o.ilH == 0 && o.ld % 8 == 0 && o.zstride % 8 == 0 && ((uintptr_t)o.base & 15) == 0;
  if (kc) return plain && o.seg == 0 && o.ext >= K;
  const bool segok = o.seg == 0 || (o.seg >= 64 && (o.seg & (o.seg - 1)) == 0 && o.segstride % 8 == 0);
  return plain && o.rows >= K && o.ext % 8 == 0 && segok;
}

static inline int kc_seg_shift(const Opnd& o) { return o.seg > 0 ? __builtin_ctzll((unsigned long long)o.seg) : 0; }

static constexpr int kc_group_rows = 4;   // measured best at the learner-step shapes

template <class C, bool AKC, bool BKC>
static inline KcArgs kc_args(const Opnd& A, const Opnd& B, int64_t M, int64_t N, int64_t K, int batches, int splits) {
  KcArgs p;
  // MN extent: the row count of a K-contiguous operand (at most the output
  // extent), the contiguous extent of an MN-contiguous one (whole 16-byte
  // chunks up to it are loaded even past the output extent, whose rows the
  // epilogue drops)
  p.A = (const bf16*)A.base; p.lda = A.ld; p.azs = A.zstride; p.arows = AKC ? std::min<int64_t>(A.rows, M) : A.ext;
  p.B = (const bf16*)B.base; p.ldb = B.ld; p.bzs = B.zstride; p.brows = BKC ? std::min<int64_t>(B.rows, N) : B.ext;
  p.asegsh = AKC ? 0 : kc_seg_shift(A); p.asegs = A.segstride;
  p.bsegsh = BKC ? 0 : kc_seg_shift(B); p.bsegs = B.segstride;
  p.M = M; p.N = N; p.K = K;
  p.ksplit = splits > 1 ? rup(cdiv(K, splits), C::BK) : (K > 0 ? K : 1);
  p.splits = splits;
  p.ntn = (int)cdiv(N, C::BN);
  p.ntm = (int)cdiv(M, C::BM);
  p.gm = kc_group_rows;
  p.total = batches * splits * p.ntm * p.ntn;
  return p;
}

// Raises a kernel's dynamic LDS limit once per device (raised: that
// kernel's own mask of devices done so far).
static inline void kc_raise_lds_limit(const void* fn, size_t bytes, std::atomic<uint64_t>& raised) {
  int dev = 0;
  const bool known = hipGetDevice(&dev) == hipSuccess && dev >= 0 && dev < 64;
  if (known && (raised.load(std::memory_order_relaxed) >> dev & 1u)) return;
  (void)hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  if (known) raised.fetch_or((uint64_t)1 << dev, std::memory_order_relaxed);
}

template <class C, bool AKC, bool BKC, class Epi>
static inline void gemm_kc_launch(const char* name, hipStream_t s, const Opnd& A, const Opnd& B, int64_t M,
                                  int64_t N, int64_t K, int batches, int splits, const Epi& epi) {
  const KcArgs p = kc_args<C, AKC, BKC>(A, B, M, N, K, batches, splits);
  auto fn = gemm_kc_kernel<C::BM, C::BN, C::WM, C::WN, C::STAGES, C::BK, AKC, BKC, Epi>;
  static std::atomic<uint64_t> lds_raised{0};
  kc_raise_lds_limit((const void*)fn, C::lds_bytes, lds_raised);
  BLSTM_LAUNCH(name, fn, dim3((unsigned)p.total), dim3(C::WM * C::WN * 64),
               C::lds_bytes, s, p, epi);
}

// Tile shape of the direct-to-LDS kernel (measured on MI355X at the
// learner-step shapes, against 256x256 blocks, 32-deep tiles and deeper
// rings): 128x128 blocks of 8 waves (64x32 each), two 64-deep stages, two
// blocks per CU.
typedef KcCfg<128, 128, 2, 4, 2> KcTile;
// 192-row blocks (two per CU fill 160 KB of LDS): fewer, larger tiles for
// products with more 128x128 tiles than one round of two blocks per CU
// (the gate projection, 448 instead of 672 blocks, and the logits)
typedef KcCfg<192, 128, 2, 4, 2> KcTileTall;
static constexpr int64_t kc_round_blocks = 2 * 256;   // two blocks on each of 256 CUs

// Whether a product with K-contiguous A goes to the 192-row blocks.
static inline bool kc_tall(int64_t M, int64_t N, int batches, int splits) {
  return M >= KcTileTall::BM && cdiv(M, 128) * cdiv(N, 128) * batches * splits > kc_round_blocks;
}
// Whether a product can take the direct-to-LDS kernel.
static inline bool kc_eligible(const Opnd& A, const Opnd& B, int64_t K, bool akc, bool bkc) {
  return K % 8 == 0 && kc_operand_ok(A, K, akc) && kc_operand_ok(B, K, bkc);
}

// GEMM dispatch: bf16 operands with 16-byte aligned rows go to the
// direct-to-LDS kernel, everything else to the generic kernel.
template <typename T, bool AKC, bool BKC, int VA, int VB, class Epi>
static inline void gemm_launch(const char* name, hipStream_t s, const Opnd& A, const Opnd& B,
                               int64_t M, int64_t N, int64_t K, int batches, int splits,
                               const Epi& epi) {
  if constexpr (std::is_same<T, bf16>::value) {
    if (kc_eligible(A, B, K, AKC, BKC)) {
      if constexpr (AKC) {
        if (kc_tall(M, N, batches, splits)) {
          gemm_kc_launch<KcTileTall, AKC, BKC>(name, s, A, B, M, N, K, batches, splits, epi);
          return;
        }
      }
      gemm_kc_launch<KcTile, AKC, BKC>(name, s, A, B, M, N, K, batches, splits, epi);
      return;
    }
    if constexpr (AKC && BKC) {
      gemm_launch_cfg<T, GemmCfgK32, AKC, BKC, VA, VB>(name, s, A, B, M, N, K, batches, splits, epi);
      return;
    }
  }
  gemm_launch_cfg<T, GemmCfg<T>, AKC, BKC, VA, VB>(name, s, A, B, M, N, K, batches, splits, epi);
}

// The pair kernel above for two products (128x128 blocks); false and nothing
// launched if either cannot take the direct-to-LDS path.
template <bool AKC1, bool BKC1, bool AKC2, bool BKC2, class Epi>
static inline bool gemm_kc_pair_launch(const char* name, hipStream_t s, const Opnd& A1, const Opnd& B1, int64_t M1,
                                       int64_t N1, int64_t K1, int splits1, const Epi& e1, const Opnd& A2,
                                       const Opnd& B2, int64_t M2, int64_t N2, int64_t K2, int splits2,
                                       const Epi& e2) {
  typedef KcTile C;
  if (!kc_eligible(A1, B1, K1, AKC1, BKC1) || !kc_eligible(A2, B2, K2, AKC2, BKC2)) return false;
  const KcArgs p1 = kc_args<C, AKC1, BKC1>(A1, B1, M1, N1, K1, 1, splits1);
  const KcArgs p2 = kc_args<C, AKC2, BKC2>(A2, B2, M2, N2, K2, 1, splits2);
  const int n1 = (int)rup(p1.total, 8);
  auto fn = gemm_kc_pair_kernel<C::BM, C::BN, C::WM, C::WN, C::STAGES, C::BK, AKC1, BKC1, AKC2, BKC2, Epi>;
  static std::atomic<uint64_t> lds_raised{0};
  kc_raise_lds_limit((const void*)fn, C::lds_bytes, lds_raised);
  BLSTM_LAUNCH(name, fn, dim3((unsigned)(n1 + p2.total)), dim3(C::WM * C::WN * 64), C::lds_bytes, s, p1, e1, p2, e2,
               n1);
  return true;
}

// One product of a grouped launch.
struct KcItem {
  Opnd A, B;
  int64_t M, N, K;
  int batches, splits;
};

// Launches products with the same operand layouts as one grid; false (and
// nothing launched) if any of them cannot take the direct-to-LDS path.
template <class C, bool AKC, bool BKC, class Epi>
static inline bool gemm_kc_group_launch_cfg(const char* name, hipStream_t s, int n, const KcItem* it,
                                            const Epi* epi) {
  if (n < 1 || n > KC_MAX_GROUP) return false;
  KcGroup<Epi> g;
  std::memset((void*)&g, 0, sizeof g);
  g.n = n;
  int start = 0;
  for (int i = 0; i < n; ++i) {
    if (it[i].K % 8 != 0 || !kc_operand_ok(it[i].A, it[i].K, AKC) || !kc_operand_ok(it[i].B, it[i].K, BKC))
      return false;
    g.p[i] = kc_args<C, AKC, BKC>(it[i].A, it[i].B, it[i].M, it[i].N, it[i].K, it[i].batches, it[i].splits);
    g.e[i] = epi[i];
    g.start[i] = start;
    start += (int)rup(g.p[i].total, 8);
  }
  g.start[n] = start;
  auto fn = gemm_kc_group_kernel<C::BM, C::BN, C::WM, C::WN, C::STAGES, C::BK, AKC, BKC, Epi>;
  static std::atomic<uint64_t> lds_raised{0};
  kc_raise_lds_limit((const void*)fn, C::lds_bytes, lds_raised);
  BLSTM_LAUNCH(name, fn, dim3((unsigned)start), dim3(C::WM * C::WN * 64), C::lds_bytes, s, g);
  return true;
}

// A grouped launch with more 128x128 blocks than one round of two per CU
// takes 192-row blocks when every product has at least 192 rows (as a
// single product does) and a k range of at most 16384 (measured: the
// weight gradients over 2688 frames 225 -> 204 us, dX at 65536 frames
// 3.11 -> 2.75 ms; but the weight gradients over 65536 frames 5.5 -> 6.1 ms).
template <bool AKC, bool BKC, class Epi>
static inline bool gemm_kc_group_launch(const char* name, hipStream_t s, int n, const KcItem* it, const Epi* epi) {
  int64_t blocks = 0;
  bool tall = n >= 1 && n <= KC_MAX_GROUP;
  for (int i = 0; tall && i < n; ++i) {
    blocks += cdiv(it[i].M, 128) * cdiv(it[i].N, 128) * it[i].batches * it[i].splits;
    tall = it[i].M >= KcTileTall::BM && it[i].K <= 16384;
  }
  if (tall && blocks > kc_round_blocks) return gemm_kc_group_launch_cfg<KcTileTall, AKC, BKC>(name, s, n, it, epi);
  return gemm_kc_group_launch_cfg<KcTile, AKC, BKC>(name, s, n, it, epi);
}
