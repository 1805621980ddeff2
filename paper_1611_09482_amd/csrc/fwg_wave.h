// Wave-per-stream step-kernel family (fwg_wave.hip).
#pragma once

#include "fwg_internal.h"

namespace fwg {

// Wave-per-stream family (fwg_wave.hip): every weight in LDS as a float image, offsets in floats.
struct WaveArgs {
  const float *image;  // the image in the workspace (copied to LDS at launch)
  int image_floats;    // multiple of 4
  int scr_floats;      // per-wave scratch after the image
  int ain_floats, c_floats, s_floats, h_floats;
  int o_emb, o_embb, o_layer, layer_floats;
  int o_convb, o_res, o_resb, o_skip, o_skipb;  // inside a layer's block
  int o_head, o_headb, o_out, o_outb;
};
hipError_t launch_wave_step(const StepArgs &a, const WaveArgs &g, hipStream_t s);
hipError_t set_wave_lds_limit(size_t bytes);
hipError_t launch_wave_image(const void *src, float *dst, int dtype, int N, int K, int C, int conv, hipStream_t s);
hipError_t launch_wave_vec(const float *src, float *dst, int n, hipStream_t s);

}  // namespace fwg
