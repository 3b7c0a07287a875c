// LDS-tiled MFMA GEMM used for every all-frames contraction of the step:
// the gate input projection, the bottleneck and softmax-layer products and
// all weight-gradient / input-gradient products.
//
// C[z][m][n] = sum_k A[z][m][k] * B[z][k][n], accumulated in float32, with
//   - each operand either K-contiguous ("KC": element (mn, k) at row(mn) + k)
//     or MN-contiguous ("MNC": element (mn, k) at row(k) + mn), so that
//     transposed products (dW = da^T x, dx = da W) need no transposed copies;
//   - a row-address map per operand (plain, segmented for the two LSTM
//     directions stored apart, or gate-interleaved);
//   - optional split-K over blockIdx.z (partial sums reduced afterwards in a
//     fixed order, so results are deterministic);
//   - an epilogue functor that receives the wave's accumulator tile.
//
// Block tile BM x BN x BK, WM x WN waves of 64 lanes, each wave owning a
// (BM/WM) x (BN/WN) tile of 16x16 MFMA blocks.  Global tiles are staged in
// registers, written to a double-buffered LDS tile laid out as
// [BK/KPL][BMN + pad][KPL] so that one MFMA fragment is one aligned LDS read.
#pragma once

#include <type_traits>

#include "common.hpp"

struct Opnd {
  const void* base;
  int64_t ld;         // elements between consecutive index rows
  int64_t zstride;    // elements between batch entries
  int64_t seg;        // > 0: rows come in segments of `seg` rows ...
  int64_t segstride;  // ... whose starts are `segstride` elements apart
  int32_t ilH;        // > 0: gate-interleaved rows (16 units x 4 gates per 64 rows)
  int32_t ext;        // extent of the contiguous dimension (elements)
  int64_t rows;       // extent of the row index; rows beyond it read as zero
};

static inline Opnd opnd(const void* base, int64_t ld, int32_t ext, int64_t rows,
                        int64_t zstride = 0) {
  Opnd o;
  o.base = base; o.ld = ld; o.zstride = zstride; o.seg = 0; o.segstride = 0;
  o.ilH = 0; o.ext = ext; o.rows = rows;
  return o;
}

template <typename T>
__device__ __forceinline__ const T* opnd_row(const Opnd& o, int z, int64_t r) {
  const T* p = (const T*)o.base + (int64_t)z * o.zstride;
  if (o.ilH > 0) r = ((r >> 4) & 3) * (int64_t)o.ilH + (r >> 6) * 16 + (r & 15);
  if (o.seg > 0) return p + (r / o.seg) * o.segstride + (r % o.seg) * o.ld;
  return p + r * o.ld;
}

template <int BYTES> struct VecOf;
template <> struct VecOf<16> { typedef uint4 type; };
template <> struct VecOf<8> { typedef uint2 type; };

template <typename T> struct LdsPad { static constexpr int rows = 1; };
template <> struct LdsPad<float> { static constexpr int rows = 4; };

// Global -> register -> LDS staging of one operand tile.
//
// K-contiguous operands (and every float32 operand) move in VEC-element
// chunks.  MN-contiguous bf16 operands move in 8x8 blocks (8 k rows of 8
// consecutive mn): each thread loads the block's 8 rows, transposes it in
// registers (pairs of bf16 per dword) and writes 8 aligned 16-byte LDS rows,
// so the LDS tile has the same [k/8][mn][8] layout in both cases.  Block b
// goes to thread b (k group = b % (BK/8)), which spreads one store
// instruction over all LDS banks.  TOFF rotates the thread numbering so two
// transposed operands are staged by different halves of the workgroup.
template <typename T, int BMN, int BK, int NT, bool KC, int VEC, int TOFF = 0>
struct TileLoader {
  static constexpr int KPL = Mfma<T>::KPL;
  static constexpr int PADR = LdsPad<T>::rows;
  static constexpr bool XPOSE = !KC && KPL == 8;
  typedef typename VecOf<VEC * (int)sizeof(T)>::type V;
  static constexpr int CPR = KC ? BK / VEC : BMN / VEC;   // chunks per global row
  static constexpr int CH = XPOSE ? (BK / 8) * (BMN / 8) * 8 : (KC ? BMN * CPR : BK * CPR);
  static constexpr int NB = (BK / 8) * (BMN / 8);          // 8x8 blocks (XPOSE)
  static constexpr int NA = NB < NT ? NB : NT;              // threads with a block
  static constexpr int BPT = NB < NT ? 1 : NB / NT;         // blocks per thread
  static constexpr int PER = XPOSE ? 8 * BPT : (CH + NT - 1) / NT;
  static_assert(KPL == 1 || VEC <= KPL || !KC, "bf16 K-contiguous chunk must fit a k-group");
  static_assert(!XPOSE || (VEC == 8 && NB % NA == 0), "transposed staging needs 8-wide chunks");
  V r[PER];

  __device__ __forceinline__ void load(const Opnd& o, int z, int64_t mn0, int64_t k0,
                                       int64_t kend, int tid) {
    if (XPOSE) {
      const int t = (tid + TOFF) % NT;
#pragma unroll
      for (int p = 0; p < BPT; ++p) {
        const int b = t + p * NA;
        const int kg = b % (BK / 8), mc = b / (BK / 8);
        const int64_t mn = mn0 + (int64_t)mc * 8;
        const bool mnok = t < NA && mn + 8 <= o.ext;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int64_t k = k0 + kg * 8 + i;
          V v = {};
          if (mnok && k < kend && k < o.rows) v = *(const V*)(opnd_row<T>(o, z, k) + mn);
          r[p * 8 + i] = v;
        }
      }
      return;
    }
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int c = tid + p * NT;
      V v = {};
      if (CH % NT == 0 || c < CH) {
        const int rr = c / CPR, cc = c % CPR;
        if (KC) {
          const int64_t row = mn0 + rr, k = k0 + (int64_t)cc * VEC;
          const int64_t kmax = min((int64_t)o.ext, (kend + VEC - 1) / VEC * VEC);
          if (row < o.rows && k + VEC <= kmax) v = *(const V*)(opnd_row<T>(o, z, row) + k);
        } else {
          const int64_t k = k0 + rr, mn = mn0 + (int64_t)cc * VEC;
          if (k < kend && k < o.rows && mn + VEC <= o.ext) v = *(const V*)(opnd_row<T>(o, z, k) + mn);
        }
      }
      r[p] = v;
    }
  }

  __device__ __forceinline__ void store(T* lds, int tid) const {
    if (XPOSE) {
      const int t = (tid + TOFF) % NT;
      if (t >= NA) return;
#pragma unroll
      for (int p = 0; p < BPT; ++p) {
        const int b = t + p * NA;
        const int kg = b % (BK / 8), mc = b / (BK / 8);
        const uint4* in = (const uint4*)&r[p * 8];
        // out row j (mn = 8*mc + j) holds k = 8*kg .. 8*kg+7; dword w packs
        // k = 2w (low half) and 2w+1 (high half)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          uint32_t o4[4];
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const uint32_t lo = ((const uint32_t*)&in[2 * w])[j / 2];
            const uint32_t hi = ((const uint32_t*)&in[2 * w + 1])[j / 2];
            o4[w] = (j & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
          }
          *(uint4*)&lds[(kg * (BMN + PADR) + mc * 8 + j) * 8] = make_uint4(o4[0], o4[1], o4[2], o4[3]);
        }
      }
      return;
    }
#pragma unroll
    for (int p = 0; p < PER; ++p) {
      const int c = tid + p * NT;
      if (CH % NT != 0 && c >= CH) continue;
      const int rr = c / CPR, cc = c % CPR;
      if (KC) {
        const int kl = cc * VEC;
        if (KPL == 8) {
          *(V*)&lds[((kl / 8) * (BMN + PADR) + rr) * 8 + (kl % 8)] = r[p];
        } else {
          const T* e = (const T*)&r[p];
#pragma unroll
          for (int i = 0; i < VEC; ++i) lds[(kl + i) * (BMN + PADR) + rr] = e[i];
        }
      } else {
        const int ml = cc * VEC;
        *(V*)&lds[rr * (BMN + PADR) + ml] = r[p];   // float32: [k][mn]
      }
    }
  }
};

// Epilogues that combine the waves of a workgroup declare
// `static constexpr bool workgroup = true` and take apply_wg<BM, WM, WN>(...,
// lds, tm, tn) instead of apply: every thread of the workgroup calls it once,
// and the kernel's LDS is theirs after a barrier.
template <class E, class = void> struct EpiIsWorkgroup : std::false_type {};
template <class E>
struct EpiIsWorkgroup<E, std::void_t<decltype(E::workgroup)>> : std::integral_constant<bool, E::workgroup> {};

template <typename T, int BM, int BN, int BK, int WM, int WN, bool AKC, bool BKC, int VA, int VB,
          class Epi, int STAGES = 1>
__global__ __launch_bounds__(WM * WN * 64) void gemm_kernel(const Opnd A, const Opnd B, int64_t M,
                                                            int64_t N, int64_t K, int64_t ksplit,
                                                            int splits, const Epi epi) {
  typedef Mfma<T> MT;
  constexpr int NT = WM * WN * 64;
  constexpr int KPL = MT::KPL;
  constexpr int PADR = LdsPad<T>::rows;
  constexpr int SA = (BK / KPL) * (BM + PADR) * KPL;
  constexpr int SB = (BK / KPL) * (BN + PADR) * KPL;
  constexpr int FM = BM / WM / 16, FN = BN / WN / 16;
  __shared__ __attribute__((aligned(16))) T lds[2][SA + SB];

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm = wid % WM, wn = wid / WM;
  const int z = blockIdx.z / splits, sp = blockIdx.z % splits;
  const int64_t m0 = (int64_t)blockIdx.y * BM, n0 = (int64_t)blockIdx.x * BN;
  const int64_t kbeg = (int64_t)sp * ksplit;
  const int64_t kend = min(K, kbeg + ksplit);
  const int ntiles = kend > kbeg ? (int)((kend - kbeg + BK - 1) / BK) : 0;

  f32x4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  typedef TileLoader<T, BM, BK, NT, AKC, VA, 0> LA;
  typedef TileLoader<T, BN, BK, NT, BKC, VB, (!AKC && !BKC) ? NT / 2 : 0> LB;
  auto compute = [&](const T* lA, const T* lB) {
#pragma unroll
    for (int ks = 0; ks < BK / MT::KSTEP; ++ks) {
      const int kg = ks * (MT::KSTEP / KPL) + (lane >> 4);
      typename MT::frag a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        a[i] = *(const typename MT::frag*)&lA[(kg * (BM + PADR) + wm * (BM / WM) + i * 16 + (lane & 15)) * KPL];
#pragma unroll
      for (int j = 0; j < FN; ++j)
        b[j] = *(const typename MT::frag*)&lB[(kg * (BN + PADR) + wn * (BN / WN) + j * 16 + (lane & 15)) * KPL];
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = MT::mma(a[i], b[j], acc[i][j]);
    }
  };
  auto kat = [&](int j) { return kbeg + (int64_t)j * BK; };
  if (STAGES == 1 && ntiles > 0) {
    // one register stage: the global loads of tile i+1 are in flight while
    // tile i is multiplied from LDS
    LA la;
    LB lb;
    la.load(A, z, m0, kat(0), kend, tid);
    lb.load(B, z, n0, kat(0), kend, tid);
    la.store(&lds[0][0], tid);
    lb.store(&lds[0][SA], tid);
    __syncthreads();
    for (int it = 0; it < ntiles; ++it) {
      const int cur = it & 1;
      const bool more = it + 1 < ntiles;
      if (more) {
        la.load(A, z, m0, kat(it + 1), kend, tid);
        lb.load(B, z, n0, kat(it + 1), kend, tid);
      }
      compute(&lds[cur][0], &lds[cur][SA]);
      if (more) {
        la.store(&lds[cur ^ 1][0], tid);
        lb.store(&lds[cur ^ 1][SA], tid);
      }
      __syncthreads();
    }
  }
  // two register stages: the global loads of tile i+2 are in flight while
  // tile i is multiplied from LDS and tile i+1 is written to the other LDS
  // buffer (two iterations of memory latency hidden, more registers)
  if (STAGES == 2 && ntiles > 0) {
    LA la0, la1;
    LB lb0, lb1;
    la0.load(A, z, m0, kat(0), kend, tid);
    lb0.load(B, z, n0, kat(0), kend, tid);
    la0.store(&lds[0][0], tid);
    lb0.store(&lds[0][SA], tid);
    if (ntiles > 1) {
      la1.load(A, z, m0, kat(1), kend, tid);
      lb1.load(B, z, n0, kat(1), kend, tid);
    }
    if (ntiles > 2) {
      la0.load(A, z, m0, kat(2), kend, tid);
      lb0.load(B, z, n0, kat(2), kend, tid);
    }
    __syncthreads();
    for (int it = 0; it < ntiles; it += 2) {
      // tile it is in LDS buffer 0; registers: stage 1 = tile it+1, stage 0 = tile it+2
      compute(&lds[0][0], &lds[0][SA]);
      if (it + 1 < ntiles) {
        la1.store(&lds[1][0], tid);
        lb1.store(&lds[1][SA], tid);
      }
      if (it + 3 < ntiles) {
        la1.load(A, z, m0, kat(it + 3), kend, tid);
        lb1.load(B, z, n0, kat(it + 3), kend, tid);
      }
      __syncthreads();
      if (it + 1 >= ntiles) break;
      // tile it+1 is in LDS buffer 1; stage 0 = tile it+2, stage 1 = tile it+3
      compute(&lds[1][0], &lds[1][SA]);
      if (it + 2 < ntiles) {
        la0.store(&lds[0][0], tid);
        lb0.store(&lds[0][SA], tid);
      }
      if (it + 4 < ntiles) {
        la0.load(A, z, m0, kat(it + 4), kend, tid);
        lb0.load(B, z, n0, kat(it + 4), kend, tid);
      }
      __syncthreads();
    }
  }
  if constexpr (EpiIsWorkgroup<Epi>::value)
    epi.template apply_wg<BM, WM, WN, FM, FN>(m0 + wm * (BM / WM), n0 + wn * (BN / WN), acc, lane, (char*)&lds[0][0],
                                              (int)blockIdx.x);
  else
    epi.template apply<FM, FN>(z, sp, m0 + wm * (BM / WM), n0 + wn * (BN / WN), acc, lane);
}

// Plain store epilogue: out[z][sp][m][n] = acc + bias[z][n] + bias2[z][n].
template <typename TO>
struct EpiStore {
  TO* out;
  int64_t ld, zstride, sstride;
  const float* bias;
  const float* bias2;
  int64_t bias_zstride;
  int64_t M, N;
  template <int FM, int FN>
  __device__ __forceinline__ void apply(int z, int sp, int64_t mw, int64_t nw, f32x4 (&acc)[FM][FN],
                                        int lane) const {
    TO* o = out + (int64_t)z * zstride + (int64_t)sp * sstride;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int64_t n = nw + j * 16 + (lane & 15);
      if (n >= N) continue;
      float bv = 0.f;
      if (bias) bv += bias[(int64_t)z * bias_zstride + n];
      if (bias2) bv += bias2[(int64_t)z * bias_zstride + n];
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t m = mw + i * 16 + (lane >> 4) * 4 + r;
          if (m < M) o[m * ld + n] = from_f32<TO>(acc[i][j][r] + bv);
        }
    }
  }
};

template <typename TO>
static inline EpiStore<TO> epi_store(TO* out, int64_t ld, int64_t M, int64_t N, int64_t zstride = 0,
                                     int64_t sstride = 0, const float* bias = nullptr,
                                     const float* bias2 = nullptr, int64_t bias_zstride = 0) {
  EpiStore<TO> e;
  e.out = out; e.ld = ld; e.zstride = zstride; e.sstride = sstride;
  e.bias = bias; e.bias2 = bias2; e.bias_zstride = bias_zstride; e.M = M; e.N = N;
  return e;
}

// Tile configurations.  bf16: 128x128 blocks with 64x64 wave tiles (66 KB of
// LDS, two workgroups per CU so one hides the other's barrier stalls);
// float32: 64x64 blocks.
template <typename T> struct GemmCfg;
template <> struct GemmCfg<bf16> {
  static constexpr int BM = 128, BN = 128, BK = 64, WM = 2, WN = 2;
};
template <> struct GemmCfg<float> {
  static constexpr int BM = 64, BN = 64, BK = 16, WM = 2, WN = 2;
};
template <typename T, class C, bool AKC, bool BKC, int VA, int VB, class Epi, int STAGES = 1>
static inline void gemm_launch_cfg(const char* name, hipStream_t s, const Opnd& A, const Opnd& B,
                                   int64_t M, int64_t N, int64_t K, int batches, int splits,
                                   const Epi& epi) {
  const int64_t ksplit = splits > 1 ? rup(cdiv(K, splits), C::BK) : (K > 0 ? K : 1);
  dim3 grid((unsigned)cdiv(N, C::BN), (unsigned)cdiv(M, C::BM), (unsigned)(batches * splits));
  BLSTM_LAUNCH(name, (gemm_kernel<T, C::BM, C::BN, C::BK, C::WM, C::WN, AKC, BKC, VA, VB, Epi, STAGES>),
               grid, dim3(C::WM * C::WN * 64), 0, s, A, B, M, N, K, ksplit, splits, epi);
}

// K-contiguous x K-contiguous bf16 products that the direct-to-LDS kernel
// cannot take (unaligned rows) run 32-deep k-tiles.
struct GemmCfgK32 {
  static constexpr int BM = 128, BN = 128, BK = 32, WM = 2, WN = 2;
};

// Fixed-order split-K reduction: dst[z][m][n] = sum_s part[z][s][m][n]
// (part rows are N wide), optionally also a low-precision copy.
template <typename TC>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* part, int splits, int batches,
                                                            int64_t M, int64_t N, float* dst,
                                                            int64_t ld, int64_t dst_zstride,
                                                            TC* dstc, int64_t ldc) {
  const int64_t total = (int64_t)batches * M * N;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t z = idx / (M * N), rem = idx % (M * N), m = rem / N, n = rem % N;
    const float* p = part + (z * splits) * M * N + rem;
    float s = p[0];
    for (int k = 1; k < splits; ++k) s += p[(int64_t)k * M * N];
    dst[z * dst_zstride + m * ld + n] = s;
    if (dstc) dstc[m * ldc + n] = from_f32<TC>(s);
  }
}
