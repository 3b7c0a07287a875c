// Deterministic reductions shared by the LSTM and head passes: column sums
// (bias gradients) and the float32-output GEMM wrapper with optional split-K.
#pragma once

#include "common.hpp"
#include "gemm_kc.hpp"

#define COLSUM_CHUNKS 64

// Column sums of an [M][N] matrix (row pitch ld) in two fixed-order passes:
// COLSUM_CHUNKS row ranges each summed in order, then the ranges in order.
template <typename T>
__global__ __launch_bounds__(256) void colsum_partial_kernel(const T* __restrict__ X, int64_t M,
                                                             int64_t N, int64_t ld,
                                                             float* __restrict__ part) {
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= N) return;
  const int64_t rpc = cdiv(M, COLSUM_CHUNKS);
  const int64_t r0 = (int64_t)blockIdx.y * rpc, r1 = min(M, r0 + rpc);
  float s = 0.f;
  for (int64_t r = r0; r < r1; ++r) s += to_f32(X[r * ld + c]);
  part[(int64_t)blockIdx.y * N + c] = s;
}

// out1/out2 are written at (c / seg) * segstride + c % seg.
__global__ __launch_bounds__(256) static void colsum_final_kernel(const float* __restrict__ part,
                                                                  int64_t N, int64_t seg,
                                                                  int64_t segstride, float* out1,
                                                                  float* out2) {
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= N) return;
  float s = part[c];
  for (int k = 1; k < COLSUM_CHUNKS; ++k) s += part[(int64_t)k * N + c];
  const int64_t o = (c / seg) * segstride + c % seg;
  out1[o] = s;
  if (out2) out2[o] = s;
}

template <typename T>
static inline void colsum(const char* name, hipStream_t s, const T* X, int64_t M, int64_t N,
                          int64_t ld, float* part, int64_t seg, int64_t segstride, float* out1,
                          float* out2) {
  BLSTM_LAUNCH(name, colsum_partial_kernel<T>, dim3((unsigned)cdiv(N, 256), COLSUM_CHUNKS), dim3(256),
               0, s, X, M, N, ld, part);
  BLSTM_LAUNCH("colsum_final", colsum_final_kernel, dim3((unsigned)cdiv(N, 256)), dim3(256), 0, s,
               part, N, seg, segstride, out1, out2);
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
  const int64_t total = (int64_t)batches * M * N;
  const unsigned grid = (unsigned)std::min<int64_t>(cdiv(total, 256), 8192);
  BLSTM_LAUNCH("splitk_reduce", splitk_reduce_kernel<T>, dim3(grid), dim3(256), 0, s, part, splits,
               batches, M, N, dst, ld, dst_zstride, dstc, ldc);
}
