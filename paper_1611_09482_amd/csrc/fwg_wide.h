// Wide step-kernel family (fwg_wide.hip): float32 ReLU stacks with 512 channels, each layer spread
// over the 32 blocks of a group (one group per XCD, four streams per group).  Not part of the public
// ABI.
#pragma once

#include "fwg_internal.h"

namespace fwg {

constexpr int kWideC = 512;       // channels
constexpr int kWideBlocks = 32;   // blocks per group (16 output channels each)
constexpr int kWideStreams = 4;   // streams per group
constexpr int kWideGroups = 8;    // groups of a launch (one per XCD)

// Workspace arrays of the family (device pointers) and the queue entries per block.
struct WideArgs {
  void *wl;        // packed layer weights
  void *wo;        // packed output 1x1
  float *embT;     // embedding transposed [Q][C]
  float *embb;     // [C]
  float *convb;    // [L][C]
  float *outb;     // [Q]
  int entries;     // sum of the dilations
  int nslots;      // weight chunks the LDS ring of a block holds
  size_t wl_bytes, wo_bytes;
};
// Whether a model fits the family (fills the array sizes, the launch's LDS bytes and its exchange
// region's bytes).
bool wide_layout(int kind, int dtype, int C, int Q, int L, int w, int bmax, const int32_t *dil, WideArgs *g,
                 size_t *lds, size_t *comm_bytes);
size_t wide_comm_bytes(int L);
hipError_t wide_setup(size_t lds, int *coresident_ok);
hipError_t launch_wide_step(const StepArgs &a, const WideArgs &g, size_t lds, hipStream_t s);
hipError_t launch_wide_pack(const void *embed, const float *embed_b, const void *const *conv,
                            const float *const *conv_b, const void *out, const float *out_b, int L, const WideArgs &g,
                            hipStream_t s);

}  // namespace fwg
