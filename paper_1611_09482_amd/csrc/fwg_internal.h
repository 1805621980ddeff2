// Internal definitions shared by the host layer (fwg_host.cpp) and the HIP
// kernels (fwg_kernels.hip).  Not part of the public ABI.
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
enum Regime { REGIME_VALU = 0, REGIME_MFMA = 1, REGIME_WAVE = 2 };

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

// MFMA family shape (gated, bf16 operands): R residual, S skip, H head channels,
// 16 streams per block of 8 waves, weight fragments per wave and stage.
constexpr int kMfR = 64, kMfS = 512, kMfH = 512, kMfRows = 16;
constexpr int kMfWaves = 8, kMfThreads = 64 * kMfWaves;
constexpr int kMfFrags = 13;       // fragments per wave and stage (8 waves x 13 = one layer's 104)
constexpr int kMfHeadStages = 8;   // head: 96 fragments per wave (+ padding), 8 stages of 13
constexpr int kMfMaxLayers = 128;
constexpr size_t kMfStageBytes = (size_t)kMfWaves * kMfFrags * 1024;
__host__ __device__ inline size_t mfma_frag_bytes(int L) { return kMfStageBytes * ((size_t)L + kMfHeadStages); }
inline size_t mfma_bias_floats(int L) { return (size_t)L * 3 * kMfR + kMfS + kMfH + 256 + kMfR; }

// Packed-weight layout of the VALU family: W^T blocked by 16 bytes along K,
// Wp[kb][n][kb_elems], with W^T[k][n] the weight from input k to output n.
inline int valu_kb_elems(int dtype) { return dtype == 1 ? 8 : 4; }

// The layer fields the general step kernel reads in its loop, copied to LDS at launch.
struct ValuLayer {
  const void *block;    // the layer's weight + bias block
  long long ring_off;   // element offset of the layer's queue
  int dil, depth;
  int pad_[2];
};
static_assert(sizeof(ValuLayer) == 32, "eight floats per layer in the LDS table");

// LDS layout (in floats) of the VALU step kernel for rows-per-block `rpw`: two buffers of popped
// states and, when a layer's weights are staged (wfloats > 0), two weight buffers.
struct ValuLds {
  int xf, xo, vo, vo2, ao, zo, so, ho, h2, lg, partA, partB, wb0, wb1, ltab, slots, ins, total_floats;
};
constexpr int kValuPrefPops = 8;   // popped elements per thread and layer held in registers
// Weight staging: a layer's block, at most kValuStagePieces 16-byte pieces per thread (64 KB).
constexpr int kValuStagePieces = 16;
__host__ __device__ inline int valu_part_cols(int N) { return N >= 256 ? N : 256; }
__host__ __device__ inline ValuLds valu_lds_layout(int kind, int C, int S, int H, int Q, int L, int rpw, int w,
                                                   int wfloats) {
  ValuLds o;
  int p = 0;
  auto take = [&](int n) { int at = p; p += (n + 3) & ~3; return at; };
  const int Co = kind == 2 ? 2 * C : C;
  o.xf = take(rpw * C);
  o.xo = take(rpw * C);
  o.vo = take(rpw * (w - 1) * C);  // the w - 1 popped states per stream, oldest first
  o.vo2 = take(rpw * (w - 1) * C);
  o.ao = take(rpw * Co);
  o.zo = take(kind == 2 ? rpw * C : 0);
  o.so = take(kind == 2 ? rpw * S : 0);
  o.ho = take(kind == 2 ? rpw * S : 0);
  o.h2 = take(kind == 2 ? rpw * H : 0);
  o.lg = take(rpw * Q);
  int partN = valu_part_cols(Co);
  if (kind == 2) {
    partN = partN > valu_part_cols(S) ? partN : valu_part_cols(S);
    partN = partN > valu_part_cols(H) ? partN : valu_part_cols(H);
  }
  partN = partN > valu_part_cols(Q) ? partN : valu_part_cols(Q);
  o.partA = take(rpw * partN);
  o.partB = take(kind == 2 ? rpw * valu_part_cols(C) : 0);
  o.wb0 = take(wfloats);
  o.wb1 = take(wfloats);
  o.ltab = take(8 * L);  // per layer: weight block address, queue offset, dilation, depth (ValuLayer)
  o.slots = take(L);   // int
  o.ins = take(rpw);   // int
  o.total_floats = p;
  return o;
}

// Launchers (fwg_kernels.hip).
hipError_t launch_valu_step(const StepArgs &a, int rpw, size_t lds_bytes, hipStream_t s);
hipError_t launch_repack(const void *src, void *dst, int mode, int dtype, int K, int N, int C, hipStream_t s);
hipError_t launch_fill_zero(void *dst, size_t bytes, hipStream_t s);
hipError_t launch_fill_i32(int32_t *dst, int32_t value, int n, hipStream_t s);
hipError_t launch_copy_bias(const float *src, float *dst, int n, hipStream_t s);
hipError_t set_valu_lds_limit(size_t bytes);
size_t mfma_lds_bytes(int L);
hipError_t launch_mfma_step(const StepArgs &a, hipStream_t s);
hipError_t set_mfma_lds_limit(size_t bytes);
hipError_t launch_mfma_repack_layer(const void *conv, const void *res, const void *skip, int l, int L, void *frags,
                                    hipStream_t s);
hipError_t launch_mfma_repack_head(const void *head, const void *out, int L, void *frags, hipStream_t s);
hipError_t launch_mfma_embed_table(const void *embed, void *dst, hipStream_t s);
hipError_t launch_mfma_bias_block(const float *const *conv_b, const float *const *res_b, const float *const *skip_b,
                                  const float *head_b, const float *out_b, const float *emb_b, int L, float *dst,
                                  hipStream_t s);

// Time-parallel path (fwg_parallel.hip).  One GEMM launch: C = A . W^T over the rows of a
// chunk (m = b * Tcur + j for time t0 + j), W operand-typed [N][K] rows.
struct ParGemm {
  int M, N, K;
  const void *A;           // plain: operand rows with stride lda; conv: the layer input rows (stride C)
  long long lda;
  const void *ring;        // conv: this layer's queue, [depth][brows][C] operand-typed
  long long t0;            // time of row j = 0
  int dil, brows, Tcur, C;
  int w, depth;            // conv / tree: taps (K = w C) and queue slots ((w - 1) dil)
  const void *W;
  const float *bias;       // [N]
  const float *xres;       // residual epilogues: fp32 input rows (stride ldo)
  float *xout;             // residual epilogues: fp32 output rows (stride ldo)
  void *oout;              // operand-typed output rows (stride ldo); NULL when it aliases xout
  long long ldo;
  int zoff;                // gate: column offset of this layer in the z rows
  float *logits;           // logits epilogue: [batch][n_steps][N]
  long long n_steps, s0;
  // naive tree (PAR_A_TREE): row m = b * Tcur + i is the node at time tnow + toff[i]; tap k reads row
  // b * nprev + tsrc[k * Tcur + i] of the level below (the node at time - (w - 1 - k) dil), and a node
  // before time 0 reads as zero.  When tsrc1 is set, residual epilogues read x_in from the
  // level-below row b * nprev + tsrc1[i] (the same-time node) instead of row m.
  const int *toff, *tsrc, *tsrc1;
  int nprev;
  long long tnow;
  void *ztop;              // gate in tree mode: z of the node at offset 0 (i = Tcur - 1) also to ztop[b][zoff + c]
  // fused gated layer (launch_par_gated_layer): residual 1x1 weights [R][R] and bias, and the z rows
  const void *W2;
  const float *bias2;
  void *zout;
  long long ldz;
};
struct ParEmbed {
  int M, C, Tcur, mode;
  long long s0, n_steps;
  const int32_t *inputs;   // [batch][n_steps]
  const int32_t *last;     // pending input per stream (online prediction)
  const void *embed;       // [Q][C] operand-typed
  const float *embed_b;
  float *xout;             // fp32 rows (NULL when not kept)
  void *oout;              // operand rows
  // naive tree: row j of stream b embeds the input at time tnow + toff[j], read from the stream's
  // input history hist[b][time & hmask] (rows before time 0 are never read as operands)
  const int *toff;
  long long tnow;
  const int32_t *hist;
  int hmask;
};
struct ParRing {
  void *ring;              // this layer's queue [depth][brows][row_bytes]
  const void *src;         // the layer input rows of the chunk
  long long t0;
  int Tcur, depth, brows, batch, row_bytes;
};
enum ParRepack { PAR_REPACK_CONV = 0, PAR_REPACK_COPY = 1 };
enum ParAMode { PAR_A_PLAIN = 0, PAR_A_CONV = 1, PAR_A_TREE = 2 };
enum ParEMode { PAR_E_RELU = 0, PAR_E_RELU_RES = 1, PAR_E_RES_ADD = 2, PAR_E_GATE = 3, PAR_E_LOGITS = 4 };
constexpr int kParKTileBytes = 128;  // K of every product must be a multiple of 128 bytes of operands
hipError_t launch_par_gemm(const ParGemm &g, int dtype, int amode, int emode, hipStream_t s);
// One gated layer over a chunk: dilated product (A gathered as in PAR_A_CONV), gate, z rows out,
// residual 1x1 and add.  Needs R in {32, 64} with R operands filling at most one 128-byte k-tile
// (par_gated_layer_ok).
bool par_gated_layer_ok(int R, int dtype);
hipError_t launch_par_gated_layer(const ParGemm &g, int dtype, hipStream_t s);
hipError_t launch_par_embed(const ParEmbed &e, int dtype, hipStream_t s);
hipError_t launch_par_ring(const ParRing &r, hipStream_t s);
hipError_t launch_par_set_last(const int32_t *inputs, int32_t *last, int batch, int n_steps, hipStream_t s);
hipError_t launch_par_repack(const void *src, void *dst, int mode, int dtype, int N, int K, int C, int interleave,
                             long long ldd, long long doff, hipStream_t s);  // conv: K = w C
hipError_t launch_par_bias(const float *src, float *dst, int N, int interleave, int accumulate, hipStream_t s);
// Naive generator: sample each row of logits [batch][256] with uniforms[b][s], write samples[b][s] and
// append the sample to the stream's input history at time tnext.
hipError_t launch_par_sample(const float *logits, const float *uniforms, int32_t *samples, int32_t *hist, int hmask,
                             long long tnext, int batch, int n_steps, int s, hipStream_t st);

// Repack modes: how W^T[k][n] is read from the caller's PyTorch layout.
enum RepackMode {
  REPACK_LINEAR = 0,  // src [N][K] (out, in)
  REPACK_CONV = 1,    // src [N][C][w]; k -> tap k / C, channel k % C; K = wC
  REPACK_EMBED = 2    // src [C][Q] -> dst [Q][C] row gather table (K = Q rows, N = C)
};

}  // namespace fwg
