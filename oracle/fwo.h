/*
 * Fast Wavenet CPU oracle: plain, slow, double-precision reference.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may include, link or
 * call this code; only the tests, the smoke check and the CPU-baseline timing
 * of the benchmark use it.  It shares no code with the GPU library.
 *
 * What it computes (paper, Section 2): a stack of width-2 dilated causal
 * convolutions evaluated one output sample at a time.  The generation model is
 * one step of a multi-layer RNN (Section 2.1/2.2, Fig. 2 and Fig. 4): it takes
 * the current input h^0_e and, for every layer, the recurrent state popped from
 * that layer's convolution queue, and returns the output plus the new states.
 * Queues are FIFOs whose depth equals the dilation of the layer that consumes
 * them (Section 2.1, Fig. 3), start filled with zeros (Section 2.2), and each
 * step is a pop phase, the computation, then a push phase (Section 2.2,
 * Fig. 5 and Fig. 6).  Every prediction is fed back as the next input
 * (Section 1).
 *
 * Evaluation forms:
 *   fwo_generate / fwo_teacher_forced  -- the cached queue form (Section 2.2)
 *   fwo_step_forced                    -- the cached form fed observed samples
 *                                          (online prediction, Sections 1 and 4)
 *   fwo_parallel                       -- each layer over the whole sequence at
 *                                          once (the training-time view, Section 1)
 *   fwo_naive                          -- recursive recomputation of the tree of
 *                                          Fig. 1, no caching (Section 1, 3.1)
 *
 * Layer definitions (the paper leaves the layer type open; these are the three
 * kinds the workloads use):
 *   relu:           x^l_t = relu(W_r x^{l-1}_{t-d} + W_e x^{l-1}_t + b)
 *   relu_residual:  x^l_t = x^{l-1}_t + relu(W_r x^{l-1}_{t-d} + W_e x^{l-1}_t + b)
 *   gated:          a = W_r x^{l-1}_{t-d} + W_e x^{l-1}_t + b      (2R outputs)
 *                   z = tanh(a[0:R]) * sigmoid(a[R:2R])
 *                   x^l_t = x^{l-1}_t + W_res z + b_res
 *                   s_t  += W_skip z + b_skip          (s_t starts at 0)
 *   output:  relu kinds  logits = W_o x^L_t + b_o
 *            gated       logits = W_o relu(W_h relu(s_t) + b_h) + b_o
 *   sampling: inverse CDF of softmax(logits) with one uniform u per step:
 *            the first k with u * Z < S_k (S_k = prefix sum of exp(l_j - max)),
 *            else the last class.  The decision is taken in float32.
 *
 * bf16 mode rounds every operand of a weight product (the popped state, the
 * current layer input, z, relu(s), the head hidden vector and the output
 * layer's input) to bf16 with round-to-nearest-even; every accumulation,
 * bias, nonlinearity, residual stream and skip sum stays in double.
 *
 * Filter width w > 2 (Section 3.1): the dilated product takes w taps,
 * x^{l-1}_{t-(w-1)d}, ..., x^{l-1}_{t-d} (the recurrent states) and x^{l-1}_t, and
 * each queue holds (w - 1) d_l states.
 *
 * Weight layouts (row-major, PyTorch conventions):
 *   embed [C][Q], conv[l] [Cout][C][w] (tap k multiplies x_{t-(w-1-k)d}; w = 2: tap 0 =
 *   recurrent x_{t-d}, tap 1 = x_t),
 *   res[l] [R][R], skip[l] [S][R], head [H][S], out [Q][C or H].
 *   A NULL bias means zeros.
 */
#ifndef FWO_H
#define FWO_H
#ifdef __cplusplus
extern "C" {
#endif

enum { FWO_RELU = 0, FWO_RELU_RESIDUAL = 1, FWO_GATED = 2 };

typedef struct {
  int kind;
  int bf16;
  int Q, C, S, H, L;
  const int *dil;
  const double *embed, *embed_b;
  const double *const *conv, *const *conv_b;
  const double *const *res, *const *res_b;
  const double *const *skip, *const *skip_b;
  const double *head, *head_b;
  const double *out, *out_b;
  long long *products; /* optional: counts applications of W_r and W_e (one per tap) */
  int w;               /* filter width (Section 3.1); 0 means 2 */
} fwo_model;

typedef struct fwo_state fwo_state;

fwo_state *fwo_state_new(const fwo_model *m, int batch, int seed_input);
void fwo_state_free(fwo_state *st);
void fwo_state_reset(fwo_state *st);
long long fwo_state_t(const fwo_state *st);

/* Generate n_steps samples per stream, continuing from the state.
 * u: [batch][n_steps] uniforms; samples: [batch][n_steps];
 * logits: optional [batch][n_steps][Q] (the distribution each sample was drawn from). */
int fwo_generate(const fwo_model *m, fwo_state *st, int n_steps, const float *u, int *samples,
                 double *logits);

/* Online prediction, continuing from the state: step i consumes the pending
 * input, writes logits[b][i] (the distribution of the next sample) and then
 * takes inputs[b][i] as that sample (the new pending input).  inputs and
 * logits as in fwo_teacher_forced, with n_steps for T. */
int fwo_step_forced(const fwo_model *m, fwo_state *st, int n_steps, const int *inputs, double *logits);

/* Cached form from zero queues; inputs [batch][T]; logits [batch][T][Q]. */
int fwo_teacher_forced(const fwo_model *m, int batch, int T, const int *inputs, double *logits);

/* Layer-by-layer evaluation over the whole sequence (zero left padding of every
 * layer input); same contract as fwo_teacher_forced. */
int fwo_parallel(const fwo_model *m, int batch, int T, const int *inputs, double *logits);

/* Naive recursive tree: logits at time t of one stream with inputs[0..t]. */
int fwo_naive(const fwo_model *m, const int *inputs, int t, double *logits);

/* Inverse-CDF sample of one row of logits, decided in float32. */
int fwo_sample(const float *logits, int Q, float u);

/* Normalised cumulative distribution in double: cdf[k] = S_k / Z. */
void fwo_cdf(const double *logits, int Q, double *cdf);

double fwo_bf16_round(double x);
int fwo_max_threads(void);

#ifdef __cplusplus
}
#endif
#endif
