// gfx950 direct-to-LDS buffer loads: a wave's 64 lanes each fetch 16 bytes
// from global memory into LDS at the wave-uniform destination + 16 * lane,
// without passing through registers.  An offset at or beyond the resource's
// range reads as zeros.
#pragma once

#include "common.hpp"

typedef __attribute__((address_space(3))) void* lds_ptr_t;

#define DMA_OFF_NONE 0x80000000u   // out of range: the lane's 16 bytes read as zero

__device__ __forceinline__ __amdgpu_buffer_rsrc_t dma_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, 0x7ffffff0, 0x00020000);
}

// lds_wave_base: this wave's 1 KB destination (same for all lanes)
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, uint32_t byte_off, void* lds_wave_base) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)lds_wave_base, 16, byte_off, 0, 0, 0);
}

__device__ __forceinline__ void dma_wait_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
