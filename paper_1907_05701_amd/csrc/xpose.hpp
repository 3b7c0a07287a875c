// bf16 matrix transposes for the operand copies of the backward products.
// A wave moves an 8x8 grid of 8x8-element blocks: each lane loads one
// block's 8 rows (16 bytes each), transposes it in registers (pairs of bf16
// per dword) and stores 8 rows of the transposed block; 8 lanes cover 128
// contiguous bytes on both the read and the write side.
#pragma once

#include "common.hpp"

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

// dst[c * ld_dst + r] = src[r * ld_src + c] for r < R, c < C (R, C, ld_src,
// ld_dst multiples of 8, pointers 16-byte aligned).
struct XposeJob {
  const bf16* src;
  bf16* dst;
  int64_t ld_src, ld_dst;
  int R, C;
};
#define XPOSE_MAX_JOBS 64
struct XposeJobs {
  XposeJob j[XPOSE_MAX_JOBS];
};

__global__ __launch_bounds__(256) static void transpose_bf16_kernel(const XposeJobs jobs) {
  const XposeJob& jb = jobs.j[blockIdx.z];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r0 = blockIdx.y * 64 + (lane >> 3) * 8;
  const int c0 = blockIdx.x * 256 + w * 64 + (lane & 7) * 8;
  if (r0 >= jb.R || c0 >= jb.C) return;
  uint4 in[8], out[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) in[i] = *(const uint4*)(jb.src + (int64_t)(r0 + i) * jb.ld_src + c0);
  transpose8x8(in, out);
#pragma unroll
  for (int j = 0; j < 8; ++j) *(uint4*)(jb.dst + (int64_t)(c0 + j) * jb.ld_dst + r0) = out[j];
}

static inline void transpose_bf16(const char* name, hipStream_t s, const XposeJobs& jobs, int n) {
  int maxR = 0, maxC = 0;
  for (int i = 0; i < n; ++i) {
    maxR = std::max(maxR, jobs.j[i].R);
    maxC = std::max(maxC, jobs.j[i].C);
  }
  if (n == 0) return;
  BLSTM_LAUNCH(name, transpose_bf16_kernel, dim3((unsigned)cdiv(maxC, 256), (unsigned)cdiv(maxR, 64), n),
               dim3(256), 0, s, jobs);
}
