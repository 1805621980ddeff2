// Time-parallel kernels (fwg_parallel.hip): forced sequences over whole chunks and the naive
// generator's per-level products.
#pragma once

#include "fwg_internal.h"

namespace fwg {

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
  // fused gated layer: the previous layer's queue refresh rides along (qring NULL: none).  Row m =
  // b * Tcur + j of qsrc (the previous layer's input rows, C operands each) goes to slot
  // (t0 + j) mod qdepth, stream b, of qring when it is among the chunk's last qdepth steps.
  void *qring;
  const void *qsrc;
  int qdepth;
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
// (par_gated_layer_ok).  Also refreshes the previous layer's queue when g.qring is set.
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

}  // namespace fwg
