// Shared definitions of the learner-step library: element types, the gfx950
// MFMA wrappers, the flat parameter layout, workspace layout, error and
// kernel-timing plumbing.  Everything here is written for CDNA4 (gfx950,
// 64-lane wavefronts) only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "adpsgd_blstm.h"

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

#define MAX_LAYERS 16
#define MAX_REPLICAS 16
#define COLSUM_MAX_CHUNKS 256   // row ranges of the two-pass column sums

// ---------------------------------------------------------------------------
// Element conversion.  float -> bf16 is round-to-nearest-even (the compiler
// lowers the cast to gfx950's v_cvt_pk_bf16_f32, which rounds that way).
// ---------------------------------------------------------------------------
template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) { return (bf16)v; }
__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16 v) { return (float)v; }

// ---------------------------------------------------------------------------
// MFMA 16x16 tiles.  For both element types lane l supplies row (l % 16) of
// the A block and column (l % 16) of the B block, and the k values it
// supplies are the same set for A and B; lane l receives C rows
// 4*(l/16) .. 4*(l/16)+3 of column l % 16.
//   bf16 : v_mfma_f32_16x16x32_bf16, 8 consecutive k per lane (one 16-byte read)
//   float: v_mfma_f32_16x16x4_f32,   1 k per lane
// ---------------------------------------------------------------------------
template <typename T> struct Mfma;
template <> struct Mfma<bf16> {
  static constexpr int KPL = 8;
  static constexpr int KSTEP = 32;
  typedef bf16x8 frag;
  __device__ static __forceinline__ f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static __forceinline__ frag zero() { return frag{}; }
};
template <> struct Mfma<float> {
  static constexpr int KPL = 1;
  static constexpr int KSTEP = 4;
  typedef float frag;
  __device__ static __forceinline__ f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  __device__ static __forceinline__ frag zero() { return 0.0f; }
};

// Transcendental helpers for the LSTM cell (float32 throughout), on the
// hardware exponential and reciprocal (v_exp_f32, v_rcp_f32: about 1 ulp
// each): sigmoid(a) = 1 / (1 + e^-a), tanh(a) = 2 sigmoid(2a) - 1 (absolute
// error a few 1e-7; both saturate correctly when e^-a over- or underflows).
__device__ __forceinline__ float sigmoidf_(float a) { return __builtin_amdgcn_rcpf(1.0f + __expf(-a)); }
__device__ __forceinline__ float tanhf_(float a) {
  return 2.0f * __builtin_amdgcn_rcpf(1.0f + __expf(-2.0f * a)) - 1.0f;
}

// ---------------------------------------------------------------------------
// Host side: layout of the flat parameter vector and of the workspaces.
// ---------------------------------------------------------------------------
struct Layout {
  int L, D, H, P, K, T, B, prec;
  int64_t M;          // frames per mini-batch, T*B
  int Dp0;            // layer-0 input width padded to a multiple of 8
  int Kp;             // logits row pitch, K padded to a multiple of 8
  size_t es;          // bytes per activation element (2 for bf16, 4 for float)
  int64_t n;          // parameter count
  // parameter offsets in elements
  int64_t Wih[MAX_LAYERS][2], Whh[MAX_LAYERS][2], bih[MAX_LAYERS][2], bhh[MAX_LAYERS][2];
  int64_t Wl, bl, Ws, bs;
  // act_ws byte offsets
  size_t X0, Y[MAX_LAYERS], G[MAX_LAYERS], C[MAX_LAYERS], GX, DYa, DYb, DC, WT, DAT, DBP, CSP, SKP, SKP2, SYNC, XCH;
  size_t WP0, WP0_bytes;   // bf16 with D % 8 != 0: layer-0 W_ih padded to Dp0 columns (else 0 bytes)
  size_t dat_bytes, dbp_bytes;   // one of the two alternating da^T / bias-partial buffers
  bool write_dat;     // bf16 with B % 8 == 0: BPTT also writes da^T [8H][M] for the weight gradients
  size_t act_bytes;
  // head_ws byte offsets
  size_t Z, S, LST, LSE, LDB, RL, DZ, DZT, HCSP, HSKP, DBLP;
  size_t head_bytes;
  size_t ytop_bytes;
  // split-K factors of the weight/input-gradient GEMMs (1 = direct store)
  int sp_dWih[MAX_LAYERS], sp_dWhh[MAX_LAYERS], sp_dX[MAX_LAYERS], sp_z, sp_dz, sp_dWs, sp_dWl, sp_dy;
  size_t skp_hh[MAX_LAYERS], skp_dx[MAX_LAYERS];   // byte offsets of the dW_hh / dX partials in SKP
  int layer_in(int l) const { return l == 0 ? D : 2 * H; }
  int layer_in_pitch(int l) const { return l == 0 ? Dp0 : 2 * H; }
};

// Fills *lo; returns BLSTM_OK or an error code (message set).
int make_layout(const blstm_dims* d, Layout* lo);

// Split-K factor for an output of Mo x No tiles of BMt x BNt with a reduction
// of Kr over BK-deep tiles: 1 when the grid already fills the chip.
int plan_splits(int64_t Mo, int64_t No, int64_t Kr, int BMt, int BNt, int BK, int batches, bool lp, bool alone);

// Error reporting (thread-local message).
int blstm_fail(int code, const char* fmt, ...);
int blstm_check_launch(const char* what);

// Kernel timing hooks; see blstm_timing_begin in the public header.
int timing_pre(const char* name, hipStream_t s);
extern bool g_timing_on;
// one event pair around `launches` consecutive launches of one kernel
int timing_pre_n(const char* name, hipStream_t s, int launches);
void timing_post(int slot, hipStream_t s);

// Times a run of consecutive launches of one kernel as a single event pair
// (per-launch events would add their own gaps between back-to-back kernels).
struct TimedRun {
  int slot;
  bool saved;
  hipStream_t s;
  TimedRun(const char* name, hipStream_t st, int launches) : s(st) {
    extern bool g_timing_on;
    saved = g_timing_on;
    slot = g_timing_on ? timing_pre_n(name, st, launches) : -1;
    g_timing_on = false;
  }
  ~TimedRun() {
    extern bool g_timing_on;
    g_timing_on = saved;
    if (slot >= 0) timing_post(slot, s);
  }
};

#define BLSTM_LAUNCH(name, kernel, grid, block, shmem, stream, ...)                     \
  do {                                                                                 \
    int _slot = g_timing_on ? timing_pre(name, stream) : -1;                           \
    hipLaunchKernelGGL(kernel, grid, block, shmem, stream, __VA_ARGS__);               \
    if (_slot >= 0) timing_post(_slot, stream);                                        \
  } while (0)

__host__ __device__ static inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
__host__ __device__ static inline int64_t rup(int64_t a, int64_t b) { return cdiv(a, b) * b; }
