// Internal definitions shared by the host layer (fwg_host.cpp) and every step-kernel family: the
// layer table, the launch arguments, the step modes, the MFMA family's shape and the utility
// launchers.  Family-specific declarations sit in fwg_valu.h, fwg_wave.h and fwg_par.h.  Not part
// of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fwg {

constexpr int kThreads = 256;     // every step kernel runs 4 waves of 64 lanes
constexpr int kMaxLayers = 1024;  // per-layer slot counters live in LDS

// One dilated layer as the step kernels see it (device-resident table).
struct LayerDev {
  // general step kernels: conv, res and skip weights, then conv_b, res_b and skip_b, are one
  // contiguous block starting at conv (staged into LDS as a unit)
  const void *conv;     // packed conv weights (W_r stacked over W_e), layout per kernel family
  const float *conv_b;  // [Cout]
  const void *res;      // gated: packed [R][R]
  const float *res_b;   // [R]
  const void *skip;     // gated: packed [S][R]
  const float *skip_b;  // [S]
  long long ring_off;   // element offset of this layer's queue inside a queue region
  int dil;              // dilation d
  int depth;            // queue slots: (w - 1) d (= d for width 2)
};

// Arguments of one step-kernel launch (passed by value).
struct StepArgs {
  const LayerDev *layers;  // [L]
  int valu_wbytes;         // general step kernels: bytes of one layer's weights + biases staged in LDS
                           // one layer ahead (0: read from global memory)
  const void *embed;       // [Q][C] rows (embedding transposed for a row gather)
  const float *embed_b;    // [C]
  const void *head;        // gated: packed [H][S]
  const float *head_b;     // [H]
  const void *out;         // packed [Q][C or H]
  const float *out_b;      // [Q]
  void *ring;              // queue region (generation or teacher-forced)
  int32_t *last;           // [bmax] next input per stream (generation mode)
  const float *uniforms;   // [batch][n_steps]
  int32_t *samples;        // [batch][n_steps]
  const int32_t *inputs;   // forced modes [batch][n_steps]
  float *logits;           // forced modes [batch][n_steps][Q]
  long long t0;            // time index of the first step of this launch
  int n_steps, batch, bmax;
  int kind, dtype, C, S, H, Q, L;
  int w;                   // filter width (taps per dilated product)
  int mode;                // StepMode
  // MFMA family only
  const void *mf_frags;    // per-wave packed weight fragment streams
  const void *mf_embT;     // embedding table [Q][R] (bf16)
  const float *mf_bias;    // bias block: conv [L][2R], res [L][R], skip sum [S], head [H], out [Q], embed [R]
  // split MFMA family only
  void *sp_comm;           // exchange words between cooperating blocks
  uint32_t *sp_sticky;     // set when a wait of a launch ran out (cleared by create and reset)
  int sp_nb;               // split family: chain blocks of this launch (ceil(batch / 16)); wide family:
                           // stream groups (ceil(batch / 4))
  uint32_t sp_tag0;        // split family: tag base of this launch, above every tag written to sp_comm
                           // since it was last zeroed (handshake and abort mark + 1, step s + 2 + s)
};

// What drives the input of each step.
enum StepMode {
  MODE_GENERATE = 0,  // the previous sample (or the stream's pending input) is fed back
  MODE_TEACHER = 1,   // step s consumes inputs[s]; queues of their own, from zero
  MODE_ONLINE = 2     // step s consumes the pending input, then inputs[s] becomes pending
};
// Offset, in steps, of the forced input that becomes the next step's input.
__host__ __device__ inline int forced_shift(int mode) { return mode == MODE_TEACHER ? 1 : 0; }

// Kernel families.
enum Regime { REGIME_VALU = 0, REGIME_MFMA = 1, REGIME_WAVE = 2, REGIME_SPLIT = 3, REGIME_CHAIN = 4, REGIME_WIDE = 5,
             REGIME_CHAIN_GATED = 6, REGIME_CHAIN_PAIR = 7 };

// MFMA family shape (gated, bf16 operands): R residual, S skip, H head channels,
// 16 streams per block of 8 waves, weight fragments per wave and stage.
constexpr int kMfR = 64, kMfS = 512, kMfH = 512, kMfRows = 16;
constexpr int kMfWaves = 8, kMfThreads = 64 * kMfWaves;
constexpr int kMfFrags = 13;       // fragments per wave and stage (8 waves x 13 = one layer's 104)
constexpr int kMfHeadStages = 8;   // head: 96 fragments per wave (+ padding), 8 stages of 13
constexpr int kMfMaxLayers = 128;
constexpr size_t kMfStageBytes = (size_t)kMfWaves * kMfFrags * 1024;
__host__ __device__ inline size_t mfma_frag_bytes(int L) { return kMfStageBytes * ((size_t)L + kMfHeadStages); }
// Width 3: the oldest tap's recurrent fragments of each layer follow the stage streams, 4 per B wave
// (tanh and sigmoid tile, two k-steps each).
constexpr size_t kMfTapBytes = (size_t)4 * 4 * 1024;
__host__ __device__ inline size_t mfma_all_frag_bytes(int L, int w) {
  return mfma_frag_bytes(L) + (w == 3 ? kMfTapBytes * (size_t)L : 0);
}
__host__ __device__ inline size_t mfma_bias_floats(int L) { return (size_t)L * 3 * kMfR + kMfS + kMfH + 256 + kMfR; }

// Split MFMA family (the MFMA family's model shape, L a multiple of 6 and at least 12): per 16
// streams one chain block (the layers), kSpHelpers helper blocks, each owning S / kSpHelpers skip
// channels and H / kSpHelpers hidden channels, and one class block (output 1x1 and sampling).
// Fragments per layer of chain waves A and B, and per layer and helper wave.
constexpr int kSpHelpers = 8;
constexpr int kSpFA = 6, kSpFB = 4, kSpFS = 8;
inline bool split_layers_ok(int L) { return L % 6 == 0 && L >= 12; }
size_t split_frag_bytes(int L);
size_t split_comm_bytes(int L, int nb);
size_t split_lds_bytes(int L);
hipError_t split_setup(int L, int nb, int *coresident_ok);
hipError_t launch_split_step(const StepArgs &a, hipStream_t s);
hipError_t launch_split_repack_layer(const void *conv, const void *res, const void *skip, int l, int L, void *frags,
                                     hipStream_t s);
hipError_t launch_split_repack_head(const void *head, const void *out, int L, void *frags, hipStream_t s);
// Allocation-free generation: the split family's per-launch exchange words in a static device array
// of this many bytes (one per device, held until the process ends) instead of the workspace.
constexpr size_t kStaticScratchBytes = (size_t)4 << 20;
// Device address of that array on the current device (looked up once per device; never the host-side
// name of the array, which is not a device address).
hipError_t split_static_scratch(void **ptr);

// Utility and MFMA-family launchers (fwg_kernels.hip, fwg_mfma.hip).
hipError_t launch_repack(const void *src, void *dst, int mode, int dtype, int K, int N, int C, hipStream_t s);
hipError_t launch_fill_zero(void *dst, size_t bytes, hipStream_t s);
hipError_t launch_fill_i32(int32_t *dst, int32_t value, int n, hipStream_t s);
hipError_t launch_copy_bias(const float *src, float *dst, int n, hipStream_t s);
size_t mfma_lds_bytes(int L, int w);
hipError_t launch_mfma_step(const StepArgs &a, hipStream_t s);
hipError_t set_mfma_lds_limit(size_t bytes);
hipError_t launch_mfma_repack_layer(const void *conv, const void *res, const void *skip, int l, int L, int w,
                                    void *frags, hipStream_t s);
hipError_t launch_mfma_repack_head(const void *head, const void *out, int L, void *frags, hipStream_t s);
hipError_t launch_mfma_embed_table(const void *embed, void *dst, hipStream_t s);
hipError_t launch_mfma_bias_block(const float *const *conv_b, const float *const *res_b, const float *const *skip_b,
                                  const float *head_b, const float *out_b, const float *emb_b, int L, float *dst,
                                  hipStream_t s);

// Repack modes: how W^T[k][n] is read from the caller's PyTorch layout.
enum RepackMode {
  REPACK_LINEAR = 0,  // src [N][K] (out, in)
  REPACK_CONV = 1,    // src [N][C][w]; k -> tap k / C, channel k % C; K = wC
  REPACK_EMBED = 2    // src [C][Q] -> dst [Q][C] row gather table (K = Q rows, N = C)
};

}  // namespace fwg
