// Deterministic reductions shared by the LSTM and head passes: column sums
// (bias gradients) and the float32-output GEMM wrapper with optional split-K.
#pragma once

#include <cstring>

#include "common.hpp"
#include "gemm_kc.hpp"

// Column sums of an [M][N] matrix (row pitch ld) in two fixed-order passes:
// `chunks` row ranges each summed in order (VEC adjacent columns per thread,
// one 16-byte load per row when the rows allow it), then the ranges in order.
template <typename T, int VEC>
__global__ __launch_bounds__(256) void colsum_partial_kernel(const T* __restrict__ X, int64_t M,
                                                             int64_t N, int64_t ld, int chunks,
                                                             float* __restrict__ part) {
  const int64_t c = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * VEC;
  if (c >= N) return;
  const int64_t rpc = cdiv(M, chunks);
  const int64_t r0 = (int64_t)blockIdx.y * rpc, r1 = min(M, r0 + rpc);
  float s[VEC];
#pragma unroll
  for (int v = 0; v < VEC; ++v) s[v] = 0.f;
  if constexpr (VEC == 1) {
    for (int64_t r = r0; r < r1; ++r) s[0] += to_f32(X[r * ld + c]);
  } else {
    typedef typename VecOf<VEC * (int)sizeof(T)>::type V;
#pragma unroll 4
    for (int64_t r = r0; r < r1; ++r) {
      const V x = *(const V*)(X + r * ld + c);
      const T* e = (const T*)&x;
#pragma unroll
      for (int v = 0; v < VEC; ++v) s[v] += to_f32(e[v]);
    }
  }
#pragma unroll
  for (int v = 0; v < VEC; ++v) part[(int64_t)blockIdx.y * N + c + v] = s[v];
}

// Sum of `nparts` partial rows per column, in part order: four threads per
// column each add a contiguous quarter, the quarters are added in order.
// out1/out2 are written at (c / seg) * segstride + c % seg.
__global__ __launch_bounds__(256) static void colsum_final_kernel(const float* __restrict__ part,
                                                                  int nparts, int64_t N, int64_t seg,
                                                                  int64_t segstride, float* out1,
                                                                  float* out2) {
  __shared__ float q4[4][64];
  const int cl = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int64_t c = (int64_t)blockIdx.x * 64 + cl;
  const int per = (nparts + 3) / 4;
  const int p0 = q * per, p1 = min(nparts, p0 + per);
  float s = 0.f;
  if (c < N) {
#pragma unroll 8
    for (int k = p0; k < p1; ++k) s += part[(int64_t)k * N + c];
  }
  q4[q][cl] = s;
  __syncthreads();
  if (q != 0 || c >= N) return;
  const float t = ((q4[0][cl] + q4[1][cl]) + q4[2][cl]) + q4[3][cl];
  const int64_t o = (c / seg) * segstride + c % seg;
  out1[o] = t;
  if (out2) out2[o] = t;
}

static inline void colsum_parts(const char* name, hipStream_t s, const float* part, int nparts, int64_t N,
                                int64_t seg, int64_t segstride, float* out1, float* out2) {
  BLSTM_LAUNCH(name, colsum_final_kernel, dim3((unsigned)cdiv(N, 64)), dim3(256), 0, s, part, nparts, N, seg,
               segstride, out1, out2);
}

template <typename T>
static inline void colsum(const char* name, hipStream_t s, const T* X, int64_t M, int64_t N,
                          int64_t ld, float* part, int64_t seg, int64_t segstride, float* out1,
                          float* out2) {
  constexpr int VEC = 16 / (int)sizeof(T);
  const bool vec = N % VEC == 0 && ld % VEC == 0 && ((uintptr_t)X & 15) == 0;
  const int64_t xb = cdiv(N, 256 * (vec ? VEC : 1));
  // about one workgroup per CU (measured at the logits' 32000 columns: 16
  // row ranges, fewer partials to combine, slightly ahead of 128)
  int chunks = (int)std::min<int64_t>(COLSUM_MAX_CHUNKS, std::max<int64_t>(16, cdiv(256, xb)));
  chunks = (int)std::max<int64_t>(1, std::min<int64_t>(chunks, M));
  if (vec)
    BLSTM_LAUNCH(name, (colsum_partial_kernel<T, VEC>), dim3((unsigned)xb, (unsigned)chunks), dim3(256), 0, s, X,
                 M, N, ld, chunks, part);
  else
    BLSTM_LAUNCH(name, (colsum_partial_kernel<T, 1>), dim3((unsigned)xb, (unsigned)chunks), dim3(256), 0, s, X, M,
                 N, ld, chunks, part);
  colsum_parts("colsum_final", s, part, chunks, N, seg, segstride, out1, out2);
}

// The same reduction, 4 adjacent columns per thread: block (m, column block
// of 256, batch), 64 threads.  Needs N, ld, ldc multiples of 4 and aligned
// destinations.  Optional: a per-column bias added to the sum, and no
// float32 destination (dst null) when only the low-precision copy is wanted.
template <typename TC>
__global__ __launch_bounds__(64) void splitk_reduce4_kernel(const float* __restrict__ part, int splits, int64_t M,
                                                            int64_t N, float* dst, int64_t ld, int64_t dst_zstride,
                                                            TC* dstc, int64_t ldc, const float* __restrict__ bias) {
  const int64_t m = blockIdx.x, n = ((int64_t)blockIdx.y * 64 + threadIdx.x) * 4;
  const int z = blockIdx.z;
  if (n >= N) return;
  const float* p = part + ((int64_t)z * splits * M + m) * N + n;
  // the first eight summands loaded together, then added in order
  constexpr int U = 8;
  float4 v[U];
#pragma unroll
  for (int k = 0; k < U; ++k)
    if (k < splits) v[k] = *(const float4*)(p + (int64_t)k * M * N);
  float4 acc = v[0];
#pragma unroll
  for (int k = 1; k < U; ++k)
    if (k < splits) { acc.x += v[k].x; acc.y += v[k].y; acc.z += v[k].z; acc.w += v[k].w; }
  for (int k = U; k < splits; ++k) {
    const float4 w = *(const float4*)(p + (int64_t)k * M * N);
    acc.x += w.x; acc.y += w.y; acc.z += w.z; acc.w += w.w;
  }
  if (bias) { acc.x += bias[n]; acc.y += bias[n + 1]; acc.z += bias[n + 2]; acc.w += bias[n + 3]; }
  if (dst) *(float4*)(dst + z * dst_zstride + m * ld + n) = acc;
  if (dstc) {
    TC* c = dstc + m * ldc + n;
    c[0] = from_f32<TC>(acc.x); c[1] = from_f32<TC>(acc.y); c[2] = from_f32<TC>(acc.z); c[3] = from_f32<TC>(acc.w);
  }
}

// The split-K reduction of a product whose partials gemm_f32 left in part
// (dst, and a low-precision copy dstc if given).
template <typename T>
static inline void splitk_reduce_launch(hipStream_t s, float* part, int splits, int batches, int64_t M, int64_t N,
                                        float* dst, int64_t ld, int64_t dst_zstride, T* dstc, int64_t ldc) {
  if (N % 4 == 0 && ld % 4 == 0 && dst_zstride % 4 == 0 && ((uintptr_t)dst & 15) == 0 &&
      (!dstc || (ldc % 4 == 0 && ((uintptr_t)dstc & 7) == 0))) {
    BLSTM_LAUNCH("splitk_reduce", splitk_reduce4_kernel<T>, dim3((unsigned)M, (unsigned)cdiv(N, 256), batches),
                 dim3(64), 0, s, part, splits, M, N, dst, ld, dst_zstride, dstc, ldc, (const float*)nullptr);
    return;
  }
  const int64_t total = (int64_t)batches * M * N;
  const unsigned grid = (unsigned)std::min<int64_t>(cdiv(total, 256), 8192);
  BLSTM_LAUNCH("splitk_reduce", splitk_reduce_kernel<T>, dim3(grid), dim3(256), 0, s, part, splits,
               batches, M, N, dst, ld, dst_zstride, dstc, ldc);
}

// C = A B with a float32 destination (ld, dst_zstride per batch).  With
// splits > 1 (or when a low-precision copy dstc is wanted) the product goes
// through split-K partials and the fixed-order reduction.
template <typename T, bool AKC, bool BKC, int VA, int VB>
static inline void gemm_f32(const char* name, hipStream_t s, const Opnd& A, const Opnd& B, int64_t M,
                            int64_t N, int64_t K, int batches, int splits, float* dst, int64_t ld,
                            int64_t dst_zstride, float* part, T* dstc = nullptr, int64_t ldc = 0) {
  if (splits == 1 && !dstc) {
    gemm_launch<T, AKC, BKC, VA, VB>(name, s, A, B, M, N, K, batches, 1,
                                     epi_store<float>(dst, ld, M, N, dst_zstride));
    return;
  }
  gemm_launch<T, AKC, BKC, VA, VB>(name, s, A, B, M, N, K, batches, splits,
                                   epi_store<float>(part, N, M, N, (int64_t)splits * M * N, M * N));
  splitk_reduce_launch<T>(s, part, splits, batches, M, N, dst, ld, dst_zstride, dstc, ldc);
}

// Several float32-destination products in one launch (see gemm_f32), then
// one launch of all their split-K reductions.
struct F32Job {
  Opnd A, B;
  int64_t M, N, K;
  int batches, splits;
  float* dst;
  int64_t ld, dst_zstride;
  float* part;   // splits x M x N floats per batch entry when splits > 1
};

// Column sums riding on a grouped launch's reduction: dst[z][n] (and dst2)
// = sum over r < rows of part[z * zin + r * kstride + n], n < N, in row order.
struct ColSumJob {
  const float* part;
  int rows, batches;
  int64_t N, kstride, zin;
  float* dst;
  float* dst2;   // optional second copy
  int64_t dst_zstride;
};

// One reduction of a grouped launch: float4 e of the job covers batch entry
// z = e / (M N/4), row m and columns 4c..4c+3 of what remains; the summands
// are kstride apart, batch entries zin apart in part.
struct ReduceJob {
  const float* part;
  float* dst;
  float* dst2;               // optional second copy
  uint32_t N4, per, count;   // N/4; M N/4; batches M N/4
  int64_t ld, dst_zstride;
  int64_t kstride, zin;
  int splits, start;         // splits: summands; start: first block of this job
};
struct ReduceGroup {
  ReduceJob j[KC_MAX_GROUP];
  int n;
};

static __global__ __launch_bounds__(256) void splitk_reduce_group_kernel(const ReduceGroup g) {
  int i = 0;
#pragma unroll
  for (int k = 1; k < KC_MAX_GROUP; ++k) i += (k < g.n && (int)blockIdx.x >= g.j[k].start);
  const ReduceJob& r = g.j[i];
  const uint32_t e = ((uint32_t)blockIdx.x - (uint32_t)r.start) * 256u + threadIdx.x;
  if (e >= r.count) return;
  const uint32_t z = e / r.per, rem = e - z * r.per;
  const uint32_t m = rem / r.N4, n = (rem - m * r.N4) * 4;
  const float* p = r.part + (int64_t)z * r.zin + (int64_t)m * r.N4 * 4 + n;
  // the first eight summands loaded together (one memory round trip), then
  // added in order; any further ones one by one after them
  constexpr int U = 8;
  float4 v[U];
#pragma unroll
  for (int k = 0; k < U; ++k)
    if (k < r.splits) v[k] = *(const float4*)(p + (int64_t)k * r.kstride);
  float4 acc = v[0];
#pragma unroll
  for (int k = 1; k < U; ++k)
    if (k < r.splits) { acc.x += v[k].x; acc.y += v[k].y; acc.z += v[k].z; acc.w += v[k].w; }
  for (int k = U; k < r.splits; ++k) {
    const float4 w = *(const float4*)(p + (int64_t)k * r.kstride);
    acc.x += w.x; acc.y += w.y; acc.z += w.z; acc.w += w.w;
  }
  const int64_t o = (int64_t)z * r.dst_zstride + (int64_t)m * r.ld + n;
  *(float4*)(r.dst + o) = acc;
  if (r.dst2) *(float4*)(r.dst2 + o) = acc;
}

static inline bool colsum_job_ok(const ColSumJob& c) {
  return c.N % 4 == 0 && c.kstride % 4 == 0 && c.zin % 4 == 0 && c.dst_zstride % 4 == 0 && c.rows >= 1 &&
         ((uintptr_t)c.part & 15) == 0 && ((uintptr_t)c.dst & 15) == 0 && ((uintptr_t)c.dst2 & 15) == 0 &&
         (int64_t)c.batches * c.N / 4 < ((int64_t)1 << 31);
}

// Launches the jobs of a reduction group (nothing if it has none).
static inline void reduce_group_launch(hipStream_t s, const ReduceGroup& rg) {
  if (rg.n < 1) return;
  const ReduceJob& last = rg.j[rg.n - 1];
  const unsigned blocks = (unsigned)(last.start + cdiv((int64_t)last.count, 256));
  BLSTM_LAUNCH("splitk_reduce_group", splitk_reduce_group_kernel, dim3(blocks), dim3(256), 0, s, rg);
}

// The reduction job of a column sum (rows summed in row order).
static inline ReduceJob colsum_reduce_job(const ColSumJob& cs, int start) {
  ReduceJob r;
  r.part = cs.part; r.dst = cs.dst; r.dst2 = cs.dst2;
  r.N4 = (uint32_t)(cs.N / 4); r.per = r.N4; r.count = (uint32_t)((int64_t)cs.batches * cs.N / 4);
  r.ld = 0; r.dst_zstride = cs.dst_zstride;
  r.kstride = cs.kstride; r.zin = cs.zin;
  r.splits = cs.rows; r.start = start;
  return r;
}

// A column sum alone, through the same reduction kernel (so the same
// summation order as when it rides on a grouped launch); false if the job
// does not qualify.
static inline bool colsum_job_launch(const char* name, hipStream_t s, const ColSumJob& cs) {
  if (!colsum_job_ok(cs)) return false;
  ReduceGroup rg;
  std::memset((void*)&rg, 0, sizeof rg);
  rg.n = 1;
  rg.j[0] = colsum_reduce_job(cs, 0);
  BLSTM_LAUNCH(name, splitk_reduce_group_kernel, dim3((unsigned)cdiv((int64_t)rg.j[0].count, 256)), dim3(256), 0, s,
               rg);
  return true;
}

// bf16 products only (the direct-to-LDS kernel); false and nothing launched
// if a product cannot take that path or its reduction needs unaligned rows.
// cs (optional): column sums added to the reduction launch.
// held (optional): the reduction is not launched but returned there, for
// the caller to launch later or to leave to a consumer of the partials.
template <bool AKC, bool BKC>
static inline bool gemm_f32_group(const char* name, hipStream_t s, int n, const F32Job* jb,
                                  const ColSumJob* cs = nullptr, ReduceGroup* held = nullptr) {
  if (n < 1 || n > KC_MAX_GROUP || (cs && (n == KC_MAX_GROUP || !colsum_job_ok(*cs)))) return false;
  KcItem it[KC_MAX_GROUP];
  EpiStore<float> e[KC_MAX_GROUP];
  ReduceGroup rg;
  std::memset((void*)&rg, 0, sizeof rg);
  rg.n = 0;
  int rblocks = 0;
  for (int i = 0; i < n; ++i) {
    const F32Job& j = jb[i];
    it[i] = KcItem{j.A, j.B, j.M, j.N, j.K, j.batches, j.splits};
    if (j.splits == 1) {
      e[i] = epi_store<float>(j.dst, j.ld, j.M, j.N, j.dst_zstride);
      continue;
    }
    const int64_t count = (int64_t)j.batches * j.M * j.N / 4;
    if (j.N % 4 != 0 || j.ld % 4 != 0 || j.dst_zstride % 4 != 0 || ((uintptr_t)j.dst & 15) != 0 ||
        ((uintptr_t)j.part & 15) != 0 || count >= ((int64_t)1 << 31))
      return false;
    e[i] = epi_store<float>(j.part, j.N, j.M, j.N, (int64_t)j.splits * j.M * j.N, j.M * j.N);
    ReduceJob& r = rg.j[rg.n++];
    r.part = j.part; r.dst = j.dst; r.dst2 = nullptr;
    r.N4 = (uint32_t)(j.N / 4); r.per = (uint32_t)(j.M * j.N / 4); r.count = (uint32_t)count;
    r.ld = j.ld; r.dst_zstride = j.dst_zstride;
    r.kstride = j.M * j.N; r.zin = (int64_t)j.splits * j.M * j.N;
    r.splits = j.splits; r.start = rblocks;
    rblocks += (int)cdiv(count, 256);
  }
  if (cs) {
    rg.j[rg.n] = colsum_reduce_job(*cs, rblocks);
    rblocks += (int)cdiv((int64_t)rg.j[rg.n++].count, 256);
  }
  if (!gemm_kc_group_launch<AKC, BKC>(name, s, n, it, e)) return false;
  if (held) *held = rg;
  else if (rg.n) reduce_group_launch(s, rg);
  return true;
}
