// Persistent recurrent kernels: interface used by the layer drivers.
#pragma once

#include "common.hpp"

struct PersistArgs {
  bf16* Y;            // layer output [M][2H] (forward: read h_prev, write h)
  const bf16* W;      // bf16 parameter copy (flat layout)
  int64_t whh0, whh1; // element offsets of W_hh for the two directions
  const bf16* WT;     // unused by the persistent kernels (W_hh^T of the layer, [2][H][4H])
  bf16* Gx;           // forward: input projection incl. both biases [M][8H] (written by the
                      // kernel itself when Xin is set, else read only)
  // forward, optional: the layer input and W_ih, so that each workgroup
  // computes the input projection of its own rows and gate columns before
  // the steps (instead of a separate product launch); null Xin: Gx is given
  const bf16* Xin;    // layer input [M][ldx] (bf16, 16-byte aligned rows)
  int64_t ldx;
  const bf16* Wih;    // W_ih of direction 0 [4H][ldw]; direction 1 at Wih + wih_d
  int64_t ldw, wih_d;
  const float* bih;   // b_ih and b_hh of direction 0 [4H]; direction 1 at + b_d
  const float* bhh;
  int64_t b_d;
  int Kin;            // input width (a multiple of 8; zero k past the operands' ends)
  // backward, optional: dy as ndy split-K partial sums (partial s of frame f,
  // unit column c at DYP[s * dy_kstride + f * 2H + c]) instead of DY; the
  // kernel sums its own rows' and units' entries in split order (the order
  // of the separate reduction) before the steps, into LDS
  const float* DYP;
  int ndy;
  int64_t dy_kstride;
  float* C;           // cell states [M][2H] (forward writes, backward reads)
  bf16* G;            // gate pre-activations [M][2][H][4] (direction, unit, gate i/f/g/o; forward writes, backward reads)
  bf16* DA;           // backward: gate pre-activation gradients [M][8H]
  const float* DY;    // backward: gradient reaching the layer output [M][2H]
  uint64_t* X;        // step-exchange words (see lstm_persist.hip), PERSIST_XCH_BYTES
  bf16* DAT;          // backward, optional: da also frame-contiguous [8H][M] (needs B % 8 == 0)
  float* DBP;         // backward, optional: sums of da over each workgroup's rows and all steps
                      // [cdiv(B, rows per workgroup)][8H] (see persist_rows_per_workgroup)
  int64_t M;          // frames, T*B (DAT row length)
  int* status;        // recurrence status block (sticky flag, see persist_status_reset)
  uint32_t tag;       // caller: the layer's position in the order the call runs the layers
  int Tn, B, H;
  int b0, rows, NS;   // batch chunk handled by one launch (filled in by persist_layer)
  uint32_t seq;       // the launch's position among the call's launches (filled in by persist_layer)
};

// At most this many batch slices of 8 or 16 rows per launch, so one launch
// covers at most PERSIST_MAX_ROWS rows.
#define PERSIST_MAX_SLICES 32
#define PERSIST_MAX_ROWS (PERSIST_MAX_SLICES * 16)
// Exchange buffer: 2 slots x 2 directions x row quads x (H/64 members) x H
// units words of 8 bytes (the backward's partial sums, four rows per word;
// the forward uses H/4 words per row, never more).
static inline size_t persist_xch_bytes(int B, int H) {
  const size_t rows = B < PERSIST_MAX_ROWS ? B : PERSIST_MAX_ROWS;
  const size_t members = H / 64 > 0 ? H / 64 : 1;
  const size_t bwd = (size_t)2 * 2 * ((rows + 3) / 4) * members * H * 8;
  const size_t fwd = (size_t)2 * 2 * rows * (H / 4 > 0 ? H / 4 : 1) * 8;
  return bwd > fwd ? bwd : fwd;
}

// Whether the backward can take dy as split-K partials (its summed dy of all
// steps must fit the LDS beside the step buffers).
bool persist_bwd_dy_partials_ok(int H, int B, int T);
// True if the persistent kernels handle this H (a multiple of 64, at most
// 512: a member's 256 W_hh rows fit in its registers); any T.
bool persist_supported(int H, int T);
// Batch rows per persistent workgroup (8 or 16) for this H and B: the row
// block of the BPTT's bias partial sums (PersistArgs::DBP).
int persist_rows_per_workgroup(int H, int B);
// Whether the persistent BPTT of a layer reads W_hh^T (PersistArgs::WT):
// never (its W_hh rows are read as they lie).
bool persist_bwd_needs_wt(int H, int B);
// Status block (PERSIST_STATUS_BYTES at the end of the activation
// workspace): an int flag set by any exchange wait that gives up, and a tag
// that marks the block initialised.  The flag is sticky across calls.
#define PERSIST_STATUS_BYTES 256
// Clears the exchange words (and, for the forward, initialises the status
// block of a fresh workspace); once per forward or backward call, before
// its first persist_layer.
hipError_t persist_clear(bool backward, const PersistArgs& a, hipStream_t s);
// Initialises the status block if it is fresh (a forward call that does not
// take the persistent path, or whose exchange clear failed).
hipError_t persist_status_init(int* status, hipStream_t s);
// Clears the flag (after blstm_recurrence_ok has read it).
hipError_t persist_status_reset(int* status, hipStream_t s);
// Runs every step of one layer, both directions; hipSuccess or the error of
// the launch that failed.  The layers of one call carry tags 0, 1, 2, ...
// in the order they run (an exchange word tells its launch from the two
// before it by the launch's position modulo 4).
hipError_t persist_layer(bool backward, PersistArgs a, hipStream_t s);
