/*
 * fwg.h -- C ABI of the Fast Wavenet generation library (libfwg.so) for AMD
 * Instinct MI355X (gfx950).
 *
 * The library implements cached autoregressive generation through a stack of
 * dilated causal convolutions (width 2 as in Sections 2.1-2.2, wider filters
 * as in Section 3.1), the method of "Fast Wavenet Generation Algorithm"
 * (Paine et al., 2016):
 *   - one generation step behaves like one step of a multi-layer recurrent net:
 *     (input, states popped from the queues) -> (logits, states to push)
 *     (Section 2.2, Fig. 4);
 *   - there is one FIFO convolution queue per layer, its depth equal to the
 *     dilation of the layer it feeds (Section 2.1, Fig. 3; (w - 1) times the
 *     dilation for width w), initialised with zeros (Section 2.2);
 *   - each generated sample runs a pop phase, the computation and a push phase
 *     (Section 2.2, Fig. 5, Fig. 6), so a sample costs O(L) work instead of the
 *     O(2^L) of recomputing the tree of Fig. 1 (Section 3.1);
 *   - every prediction is fed back as the next input (Section 1).
 *
 * Layer kinds (the paper leaves the layer type open):
 *   FWG_RELU:           x^l = relu(W_r x^{l-1}_{t-d} + W_e x^{l-1}_t + b)
 *   FWG_RELU_RESIDUAL:  x^l = x^{l-1} + relu(W_r x^{l-1}_{t-d} + W_e x^{l-1}_t + b)
 *   FWG_GATED:          a = W_r x^{l-1}_{t-d} + W_e x^{l-1}_t + b (2R channels),
 *                       z = tanh(a[0:R]) * sigmoid(a[R:2R]),
 *                       x^l = x^{l-1} + W_res z + b_res,  s += W_skip z + b_skip
 *   output: relu kinds  logits = W_out x^L + b_out
 *           gated       logits = W_out relu(W_head relu(s) + b_head) + b_out
 *   sampling: softmax over the n_classes logits, inverse CDF with one caller
 *           uniform u per stream and step: the first class k with u*Z < S_k
 *           (S_k = running sum of exp(logit_j - max), Z = S_{n_classes-1}),
 *           else the last class.  Computed in float32.
 *
 * Precision: FWG_F32 computes in float32.  FWG_BF16 takes bf16 weights and
 * rounds every operand of a weight product (popped states, the current layer
 * input, z, relu(s), the head hidden vector, the output layer's input) to bf16
 * (round to nearest even); accumulation, biases, nonlinearities, the residual
 * stream, the skip sum, logits and softmax stay float32.  The queues store bf16.
 *
 * Memory and ownership:
 *   - The library never allocates device memory.  The caller provides one
 *     device workspace of fwg_workspace_size() bytes (256-byte aligned), which
 *     must stay allocated and untouched until fwg_destroy().
 *   - fwg_create() copies and repacks the caller's weights into the workspace;
 *     the caller's weight buffers may be freed once the stream has synchronised.
 *   - All device pointers are plain device addresses; all outputs are
 *     caller-owned.
 *   - Every call enqueues its work on the stream given to fwg_create() and
 *     returns without waiting (fwg_create() itself synchronises that stream
 *     once, after uploading its tables).  The caller synchronises before
 *     reading outputs.
 *
 * Errors: every argument and state check runs on the host before anything is
 * enqueued; on a non-OK status nothing was enqueued and fwg_last_error()
 * returns a message (per calling thread).  Device data are never validated:
 * inputs outside [0, n_classes) are undefined behaviour; a uniform >= 1 selects
 * the last class and a negative one class 0.  A handle is not thread-safe;
 * distinct handles are independent.
 */
#ifndef FWG_H
#define FWG_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
enum {
  FWG_OK = 0,
  FWG_EINVAL = -1,       /* NULL pointer, non-positive size, dilation < 1, batch out of range ... */
  FWG_ENOSPACE = -2,     /* workspace smaller than fwg_workspace_size() or misaligned */
  FWG_EHIP = -3,         /* a HIP runtime call failed (message has the HIP error string) */
  FWG_ESTATE = -4,       /* generate() with a batch other than the one used since the last reset */
  FWG_EUNSUPPORTED = -5, /* a valid shape this build has no kernel for */
  FWG_EDEVICE = -6       /* fwg_device_status: a launch ended without valid results (see there) */
};

/* layer kinds */
enum { FWG_RELU = 0, FWG_RELU_RESIDUAL = 1, FWG_GATED = 2 };
/* weight / operand types (accumulation is always float32) */
enum { FWG_F32 = 0, FWG_BF16 = 1 };

/* Model descriptor.  All fields are read during the call only. */
typedef struct {
  int32_t kind;           /* FWG_RELU, FWG_RELU_RESIDUAL or FWG_GATED */
  int32_t dtype;          /* FWG_F32 or FWG_BF16 */
  int32_t n_classes;      /* Q: size of the one-hot input and of the softmax; 256 supported */
  int32_t channels;       /* C (relu kinds) or R (gated residual channels) */
  int32_t skip_channels;  /* S, gated only (ignored otherwise) */
  int32_t head_channels;  /* H, gated only (ignored otherwise) */
  int32_t n_layers;       /* L >= 1 */
  int32_t max_batch;      /* largest batch of independent streams, >= 1 */
  int32_t seed_input;     /* input class fed at the first step after a reset, in [0, Q) */
  const int32_t *dilations; /* HOST array [n_layers], each >= 1: layer l reads x^{l-1}_{t-d_l} */
  int32_t filter_width;   /* w taps per dilated product, x^{l-1}_{t-(w-1)d_l} .. x^{l-1}_t
                             (Section 3.1); 0 means 2, the width of Sections 2.1-2.2.  Each
                             queue then holds (w-1) d_l states. */
} fwg_desc;

/* Weights: DEVICE pointers to row-major arrays in PyTorch layouts; the
 * per-layer tables are HOST arrays of n_layers DEVICE pointers.  Matrices have
 * the descriptor's dtype (bf16 = 16-bit bf16 bit patterns); biases are always
 * float32.  A NULL bias (or a NULL bias table) means zeros.
 *   embed   [C][Q]           1x1 convolution over the one-hot input
 *   conv[l] [Cout][C][w]     Cout = C (relu kinds) or 2R (gated); tap k multiplies
 *                            x_{t-(w-1-k)d}: for w = 2 tap 0 multiplies x_{t-d} (W_r),
 *                            tap 1 multiplies x_t (W_e)
 *   res[l]  [R][R]           gated only
 *   skip[l] [S][R]           gated only
 *   head    [H][S]           gated only
 *   out     [Q][C] or [Q][H] */
typedef struct {
  const void *embed;
  const float *embed_b;
  const void *const *conv;
  const float *const *conv_b;
  const void *const *res;
  const float *const *res_b;
  const void *const *skip;
  const float *const *skip_b;
  const void *head;
  const float *head_b;
  const void *out;
  const float *out_b;
} fwg_weights;

typedef struct fwg_handle fwg_handle;

/* Bytes of device workspace a model needs (pure host computation; no device
 * needed).  Returns FWG_EINVAL / FWG_EUNSUPPORTED for descriptors create()
 * would reject. */
int fwg_workspace_size(const fwg_desc *desc, size_t *bytes);

/* Validate the descriptor, lay out the workspace, repack the weights into it
 * and reset the queues (Section 2.2: queues start at zero).  hip_stream is a
 * hipStream_t (NULL = default stream) on the current device; it is used by
 * every later call on the handle.  On success *out receives the handle. */
int fwg_create(const fwg_desc *desc, const fwg_weights *weights, void *workspace, size_t ws_bytes,
               void *hip_stream, fwg_handle **out);

/* Zero every convolution queue (the queues start empty, i.e. all zeros,
 * Section 2.2), set t = 0 and every stream's next input to seed_input, and
 * unbind the batch size. */
int fwg_reset_queues(fwg_handle *h);

/* Generate n_steps samples for each of `batch` independent streams, continuing
 * from the current state: per sample the pop phase, the layer computations and
 * the push phase of Section 2.2 (Fig. 5, Fig. 6), then the sample drawn from the
 * output distribution becomes the next input (Section 1).  uniforms: DEVICE float32 [batch][n_steps];
 * samples: DEVICE int32 [batch][n_steps], samples[b][s] drawn for time t0+s.
 * The first call after a reset binds the batch size; later calls with another
 * batch return FWG_ESTATE.  n_steps == 0 is a no-op. */
int fwg_generate(fwg_handle *h, int32_t batch, int32_t n_steps, const float *uniforms, int32_t *samples);

/* fwg_generate for callers that cannot allocate device memory, e.g. code under
 * HIP graph capture, tight serving loops, or harnesses that forbid hipMalloc.
 * Same arguments, state, results and errors as fwg_generate.  The kernel
 * families whose blocks cooperate within a launch (fwg_regime
 * "mfma_split_bf16_r64_s512", "wide_f32_c512" and "chain_pair_f32_r32") keep
 * the words they exchange in a static device array of 4 MiB (one per device,
 * set up by fwg_create and held until the process ends) instead of the
 * workspace; a batch whose words do not fit (split family: more than 4 MiB /
 * (8 x (512 L + 8544)) groups of 16 streams, about 21 groups at L = 30; wide
 * family: 256 + 8 x (16,384 L + 17,664) bytes whatever the batch, so L <= 30;
 * gated chain pair family: 256 + 8 x (736 + 32 L) bytes per stream, 381
 * streams at L = 20) returns FWG_ENOSPACE before anything is enqueued.  The
 * other kernel families use no per-launch scratch and run exactly as
 * fwg_generate.  The array is cleared by a fill kernel at the start of every
 * launch, but every call on a device shares it: calls of this entry point that
 * overlap on one device (other streams, other handles, other threads) race and
 * must be serialised by the caller.  Allocates nothing and calls no allocating
 * routine. */
int fwg_generate_noalloc(fwg_handle *h, int32_t batch, int32_t n_steps, const float *uniforms, int32_t *samples);

/* Teacher-forced evaluation from zero queues: logits[b][t][:] is the output
 * after consuming inputs[b][0..t], i.e. the cached step of Section 2.2 with
 * each step's input given instead of sampled; it equals the dilated causal
 * convolution evaluated over the whole sequence (the training-time view of
 * Section 1).  inputs: DEVICE int32 [batch][seq_len];
 * logits: DEVICE float32 [batch][seq_len][n_classes].  Runs the generation
 * step kernels in forced mode (the input of each step taken from `inputs`
 * instead of the previous sample), so the logits check the hot path itself;
 * uses queues of its own and leaves the generation state untouched.
 * 1 <= batch <= max_batch; seq_len == 0 is a no-op. */
int fwg_teacher_forced(fwg_handle *h, int32_t batch, int32_t seq_len, const int32_t *inputs, float *logits);

/* Online prediction (the use the paper names beside generation, end of Section 1
 * and Section 4): the same cached step continues from the current queue state,
 * but the sample that follows each step is observed instead of drawn.  Step s
 * (time t0 + s) consumes the stream's pending input -- for s = 0 the input
 * fwg_generate would have consumed next (seed_input after a reset, else the last
 * sample generated or observed), for s > 0 inputs[b][s-1] -- and writes
 * logits[b][s][:], the distribution the model predicts for the next sample; then
 * inputs[b][s] becomes the pending input.  Queues and t advance exactly as in
 * fwg_generate, so generation and online prediction may alternate freely.
 * inputs: DEVICE int32 [batch][n_steps], each in [0, n_classes);
 * logits: DEVICE float32 [batch][n_steps][n_classes], or NULL when only the
 * state should advance.  Runs the generation step kernels.  Batch binding and
 * the FWG_ESTATE rule as in fwg_generate; n_steps == 0 is a no-op. */
int fwg_step_forced(fwg_handle *h, int32_t batch, int32_t n_steps, const int32_t *inputs, float *logits);

/* Time-parallel evaluation (the training-time view of the network, Section 1):
 * with every input known, each layer is one width-w dilated convolution over
 * the whole sequence, computed as matrix-core GEMMs over (stream, time) rows in
 * chunks of steps, the states before a chunk read from the layer's queue.
 * fwg_teacher_forced_parallel has the contract and results of
 * fwg_teacher_forced (queues of its own, from zero; generation state untouched);
 * only the order of the float32 sums differs.  Models whose products do not
 * fill whole 128-byte k-tiles (K of 16 float32 or 32 bf16 values) have no
 * time-parallel kernels: for them this call runs fwg_teacher_forced itself. */
int fwg_teacher_forced_parallel(fwg_handle *h, int32_t batch, int32_t seq_len, const int32_t *inputs, float *logits);

/* Priming from a prefix, time-parallel: the contract of fwg_step_forced
 * (online prediction continuing from the generation state; logits may be NULL),
 * evaluated like fwg_teacher_forced_parallel.  After each layer of a chunk the
 * chunk's newest (w-1) d_l states replace the queue's contents, so the queues
 * end in the state the step-by-step loop would leave and generation continues
 * from the prefix.  Where fwg_teacher_forced_parallel runs the step kernels,
 * so does this call (fwg_step_forced itself). */
int fwg_prime(fwg_handle *h, int32_t batch, int32_t n_steps, const int32_t *inputs, float *logits);

/* Naive generation, the baseline the paper measures against (Section 1, Fig. 1;
 * Section 3): every sample recomputes, from the last receptive-field inputs, each
 * distinct node of the tree of layer states the output depends on (a node that
 * several branches reach is computed once per sample), and nothing is cached
 * between samples.  Same model, sampling rule and contract as fwg_generate
 * (uniforms DEVICE float32 [batch][n_steps], samples DEVICE int32
 * [batch][n_steps]), but with its own state: the per-stream input history and
 * its own time and batch binding, reset by fwg_reset_queues (the history then
 * starts with seed_input).  One kernel sequence per sample; for comparison and
 * testing, not for throughput.  Returns FWG_EUNSUPPORTED where the model has
 * no time-parallel kernels or its chunk buffers cannot hold max_batch x (the
 * tree's input nodes) rows. */
int fwg_generate_naive(fwg_handle *h, int32_t batch, int32_t n_steps, const float *uniforms, int32_t *samples);

/* Layer-node evaluations per sample of fwg_generate_naive: the number of
 * distinct nodes of the tree over layers 1..L (Section 3.1; the cached method
 * evaluates L).  Pure host computation. */
int fwg_naive_nodes(const fwg_desc *desc, int64_t *nodes);

/* Free the host-side handle (the workspace stays the caller's). NULL is a no-op. */
int fwg_destroy(fwg_handle *h);

/* Message for the last non-OK status returned on this thread ("" if none). */
const char *fwg_last_error(void);

/* Short name of the kernel family a handle uses (for logs and profiles). */
const char *fwg_regime(const fwg_handle *h);

/* Wait for every call enqueued on the handle's stream, then report whether a
 * launch since the last create/reset ended without valid results: FWG_EDEVICE
 * when a bounded wait between the cooperating blocks of a split-family launch
 * ran out (its blocks were not all resident on the device at once; that launch
 * then completes quickly with invalid outputs instead of hanging), FWG_EHIP on
 * a HIP error, else FWG_OK.  Kernel families without cross-block waits always
 * return FWG_OK after the synchronisation.  The mark is cleared by
 * fwg_reset_queues. */
int fwg_device_status(fwg_handle *h);

#ifdef __cplusplus
}
#endif
#endif /* FWG_H */
