// Chain step-kernel family (fwg_chain.hip): small float32 ReLU stacks, one block per stream, every
// weight and queue in LDS.  Not part of the public ABI.
#pragma once

#include "fwg_internal.h"

namespace fwg {

constexpr int kChainC = 32;         // channels the chain kernel is built for
constexpr int kChainMaxLayers = 6;  // layers whose weights its waves hold in registers

// The weight image (offsets in floats): embedding [Q][C] and bias, per layer W_r^T [C][C], W_e^T
// [C][C] and bias, output 1x1 transposed [C][Q] and bias.
struct ChainArgs {
  const float *image;
  int image_floats, ring_floats;
  int o_emb, o_embb, o_layer, layer_floats, o_out, o_outb;
};
// Whether a model fits the family (fills g and the launch's LDS bytes).
bool chain_layout(int kind, int dtype, int C, int Q, int L, int w, const int32_t *dil, ChainArgs *g, size_t *lds);
hipError_t set_chain_lds_limit(size_t bytes);
hipError_t launch_chain_step(const StepArgs &a, const ChainArgs &g, size_t lds, hipStream_t s);
hipError_t launch_chain_image(const void *embed, const float *embed_b, const void *const *conv,
                              const float *const *conv_b, const void *out, const float *out_b, int L,
                              const ChainArgs &g, float *img, hipStream_t s);

}  // namespace fwg
