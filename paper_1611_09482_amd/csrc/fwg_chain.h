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

namespace fwg {

// Gated variant (fwg_chain.hip): float32 gated stacks with R = 32 residual channels, S = H = 256,
// filter width 2 or 3, at most 64 layers: one block per stream, the weights streamed from the workspace
// per step, the queues in the workspace.
constexpr int kChainGR = 32, kChainGS = 256;
constexpr int kChainGMaxLayers = 64;  // per-layer queue tables live in one lane each
constexpr int kChainGMaxWidth = 3;    // filter widths 2 and 3
struct ChainGatedArgs {
  const float4 *wchain;  // [L][12][64]: wave 0's W_e row chunks (8), then W_res half-row chunks (4)
  const float4 *wrec;    // [L][8 (w - 1)][64]: wave 1's row chunks of the recurrent taps, oldest first
  const float4 *wskip;   // [L][2][16][64]: the skip waves' two rows each (8 chunks per row)
  const float4 *whead;   // [4][64][64]: row t = 64 w + l of the first head 1x1, chunk c at [w][c][l]
  const float4 *wout;    // [4][64][64]: row t of the output 1x1, the same way
  const float4 *wm;      // pair variant: [L][8][64], slot l: rows of W_e^l W_res^{l-1} (slot 0 unused)
  const float *convb;    // [L][64] (pair variant: + W_e^l b_res^{l-1})
  const float *resb;     // [L][32]
  const float *skipb;    // [256]: the skip biases summed over the layers
  const float *headb, *outb;  // [256] each
  const float *embT;     // [Q][32]
  const float *embb;     // [32]
};
bool chain_gated_ok(int kind, int dtype, int C, int S, int H, int Q, int L, int w, size_t *img_bytes, size_t *lds);
hipError_t set_chain_gated_lds_limit(size_t bytes);
// The arrays of ChainGatedArgs laid out from `base` (the workspace region of img_bytes).
ChainGatedArgs chain_gated_arrays(void *base, int L, int w);
hipError_t launch_chain_gated_step(const StepArgs &a, const ChainGatedArgs &g, size_t lds, hipStream_t s);
hipError_t launch_chain_gated_pack(const void *embed, const float *embed_b, const void *const *conv,
                                   const float *const *conv_b, const void *const *res, const float *const *res_b,
                                   const void *const *skip, const float *const *skip_b, const void *head,
                                   const float *head_b, const void *out, const float *out_b, int L, int w, bool pair,
                                   const ChainGatedArgs &g, hipStream_t s);
// Pair variant (two blocks of one XCD per stream, exchanging tagged words; pack with pair = true):
// LDS bytes of a launch, exchange-region bytes for `batch` streams (zeroed before every launch;
// an abort word, then 736 + 32 L words per stream), grid blocks, set-up (LDS limit; whether every
// block of a launch of bmax streams can be resident at once) and launch (a.sp_comm, a.sp_sticky).
size_t chain_pair_lds_bytes(int L);
size_t chain_pair_comm_bytes(int L, int batch);
int chain_pair_grid(int batch);
hipError_t chain_pair_setup(size_t lds, int bmax, int *coresident_ok);
hipError_t launch_chain_pair_step(const StepArgs &a, const ChainGatedArgs &g, size_t lds, hipStream_t s);

}  // namespace fwg
