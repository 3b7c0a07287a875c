// Persistent recurrent kernels: interface used by the layer drivers.
#pragma once

#include "common.hpp"

struct PersistArgs {
  bf16* Y;            // layer output [M][2H] (forward: read h_prev, write h)
  const bf16* W;      // bf16 parameter copy (flat layout)
  int64_t whh0, whh1; // element offsets of W_hh for the two directions
  const bf16* Gx;     // forward: input projection [M][8H]
  float* C;           // cell states [M][2H] (forward writes, backward reads)
  bf16* G;            // activated gates [M][8H] (forward writes, backward reads)
  bf16* DA;           // backward: gate pre-activation gradients [M][8H]
  const float* DY;    // backward: gradient reaching the layer output [M][2H]
  unsigned* ctr;      // group counters (zeroed before each launch)
  int* status;        // set to 1 if a barrier wait ever timed out
  int Tn, B, H;
  int b0, rows, NS;   // batch chunk handled by one launch (filled in by persist_layer)
};

// Largest number of groups' counters a launch uses (times CTR stride).
#define PERSIST_CTR_BYTES (64 * 32 * 4)

// True if the persistent kernels can hold a W_hh slice for this H in LDS.
bool persist_supported(int H);
// Runs every step of one layer, both directions; hipSuccess or the error of
// the cooperative launch that failed.
hipError_t persist_layer(bool backward, PersistArgs a, hipStream_t s);
