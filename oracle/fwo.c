/*
 * Fast Wavenet CPU oracle -- TEST INFRASTRUCTURE ONLY (see fwo.h).
 * Plain loops in double precision; no blocking, no fusion, no reordering
 * beyond what the definitions state.
 */
#include "fwo.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* bf16 rounding of a double: keep 8 significant bits, nearest, ties to even. */
double fwo_bf16_round(double x) {
  if (x == 0.0 || !isfinite(x)) return x;
  int e;
  double m = frexp(x, &e);       /* x = m * 2^e, 0.5 <= |m| < 1 */
  double r = rint(m * 256.0);    /* 8 significant bits; rint rounds half to even */
  return ldexp(r, e - 8);
}

static inline double opnd(const fwo_model *m, double v) { return m->bf16 ? fwo_bf16_round(v) : v; }
static inline double relu(double v) { return v > 0.0 ? v : 0.0; }
static inline double sigmoid(double v) { return 1.0 / (1.0 + exp(-v)); }
static inline double bias_at(const double *b, int i) { return b ? b[i] : 0.0; }

int fwo_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Building blocks shared by the three forms: one layer given (recurrent input,
 * current input) and the output head.  These are the definitions in fwo.h.  */

static int conv_out(const fwo_model *m) { return m->kind == FWO_GATED ? 2 * m->C : m->C; }
/* filter width w (Section 3.1); the paper's algorithm section uses w = 2 */
static int width(const fwo_model *m) { return m->w > 2 ? m->w : 2; }

/* Layer l: r = the w - 1 recurrent states x^{l-1}_{t-(w-1)d}, ..., x^{l-1}_{t-d}
 * (oldest first, C each), x = x^{l-1}_t  ->  x_next = x^l_t; for gated also adds
 * this layer's skip contribution into s (length S).  Tap k of the [Cout][C][w]
 * kernel multiplies x^{l-1}_{t-(w-1-k)d}, so tap w-1 multiplies x_t. */
static void layer_apply(const fwo_model *m, int l, const double *r, const double *x, double *x_next,
                        double *s, double *work) {
  const int C = m->C, Co = conv_out(m), w = width(m);
  const double *W = m->conv[l];
  double *a = work;
  double *ro = work + Co, *xo = work + Co + (size_t)(w - 1) * C;
  for (int i = 0; i < (w - 1) * C; ++i) ro[i] = opnd(m, r[i]);
  for (int c = 0; c < C; ++c) xo[c] = opnd(m, x[c]);
  if (m->products) *m->products += w; /* one application per tap: w - 1 recurrent (W_r), one current (W_e) */
  for (int o = 0; o < Co; ++o) {
    double acc = bias_at(m->conv_b[l], o);
    for (int c = 0; c < C; ++c) {
      for (int k = 0; k < w - 1; ++k) acc += W[(o * C + c) * w + k] * ro[k * C + c];
      acc += W[(o * C + c) * w + (w - 1)] * xo[c];
    }
    a[o] = acc;
  }
  if (m->kind == FWO_RELU) {
    for (int c = 0; c < C; ++c) x_next[c] = relu(a[c]);
  } else if (m->kind == FWO_RELU_RESIDUAL) {
    for (int c = 0; c < C; ++c) x_next[c] = x[c] + relu(a[c]);
  } else {
    const int R = C, S = m->S;
    double *z = work + Co; /* reuse: ro no longer needed */
    for (int c = 0; c < R; ++c) z[c] = opnd(m, tanh(a[c]) * sigmoid(a[R + c]));
    const double *Wr = m->res[l], *Ws = m->skip[l];
    for (int c = 0; c < R; ++c) {
      double acc = bias_at(m->res_b[l], c);
      for (int j = 0; j < R; ++j) acc += Wr[c * R + j] * z[j];
      x_next[c] = x[c] + acc;
    }
    for (int k = 0; k < S; ++k) {
      double acc = bias_at(m->skip_b[l], k);
      for (int j = 0; j < R; ++j) acc += Ws[k * R + j] * z[j];
      s[k] += acc;
    }
  }
}

/* Output node: logits from the top state (relu kinds) or the skip sum (gated).
 * work: >= max(S, H, C) + H doubles. */
static void head_apply(const fwo_model *m, const double *top, const double *s, double *logits,
                       double *work) {
  const int Q = m->Q;
  if (m->kind != FWO_GATED) {
    const int C = m->C;
    double *xo = work;
    for (int c = 0; c < C; ++c) xo[c] = opnd(m, top[c]);
    for (int q = 0; q < Q; ++q) {
      double acc = bias_at(m->out_b, q);
      for (int c = 0; c < C; ++c) acc += m->out[q * C + c] * xo[c];
      logits[q] = acc;
    }
    return;
  }
  const int S = m->S, H = m->H;
  double *rs = work, *h = work + S;
  for (int k = 0; k < S; ++k) rs[k] = opnd(m, relu(s[k]));
  for (int i = 0; i < H; ++i) {
    double acc = bias_at(m->head_b, i);
    for (int k = 0; k < S; ++k) acc += m->head[i * S + k] * rs[k];
    h[i] = opnd(m, relu(acc));
  }
  for (int q = 0; q < Q; ++q) {
    double acc = bias_at(m->out_b, q);
    for (int i = 0; i < H; ++i) acc += m->out[q * H + i] * h[i];
    logits[q] = acc;
  }
}

static void embed_apply(const fwo_model *m, int in, double *x0) {
  for (int c = 0; c < m->C; ++c) x0[c] = m->embed[c * m->Q + in] + bias_at(m->embed_b, c);
}

static size_t work_doubles(const fwo_model *m) {
  size_t w = 3 * (size_t)conv_out(m) + ((size_t)width(m) + 1) * m->C + (size_t)m->S + (size_t)m->H + 16;
  return w;
}

/* ------------------------------------------------------------------------ */
/* Convolution queues (Section 2.1, Fig. 3): one FIFO of depth d_l per layer,
 * each element a C-vector, initially d_l zero vectors (Section 2.2).  With
 * filter width w the queue holds the (w - 1) d_l newest states (Section 3.1). */
typedef struct {
  double *buf;
  int depth, head, count, C;
} fifo;

static void fifo_init(fifo *q, int depth, int C) {
  q->buf = (double *)calloc((size_t)depth * C, sizeof(double));
  q->depth = depth;
  q->C = C;
  q->head = 0;
  q->count = depth; /* full of zeros */
}
static void fifo_zero(fifo *q) {
  memset(q->buf, 0, sizeof(double) * (size_t)q->depth * q->C);
  q->head = 0;
  q->count = q->depth;
}
/* Pop the first (oldest) element into out. */
static void fifo_pop(fifo *q, double *out) {
  memcpy(out, q->buf + (size_t)q->head * q->C, sizeof(double) * q->C);
  q->head = (q->head + 1) % q->depth;
  q->count -= 1;
}
/* Copy the element at position p from the front (0 = oldest) into out. */
static void fifo_peek(const fifo *q, int p, double *out) {
  memcpy(out, q->buf + (size_t)((q->head + p) % q->depth) * q->C, sizeof(double) * q->C);
}
/* Push to the back. */
static void fifo_push(fifo *q, const double *x) {
  int tail = (q->head + q->count) % q->depth;
  memcpy(q->buf + (size_t)tail * q->C, x, sizeof(double) * q->C);
  q->count += 1;
}

struct fwo_state {
  const fwo_model *m;
  int batch, seed_input;
  long long t;
  int *last;    /* next input per stream */
  fifo *queues; /* [batch][L] */
};

fwo_state *fwo_state_new(const fwo_model *m, int batch, int seed_input) {
  if (!m || batch <= 0) return NULL;
  fwo_state *st = (fwo_state *)calloc(1, sizeof(fwo_state));
  st->m = m;
  st->batch = batch;
  st->seed_input = seed_input;
  st->last = (int *)malloc(sizeof(int) * batch);
  st->queues = (fifo *)malloc(sizeof(fifo) * (size_t)batch * m->L);
  for (int b = 0; b < batch; ++b)
    for (int l = 0; l < m->L; ++l)
      fifo_init(&st->queues[(size_t)b * m->L + l], (width(m) - 1) * m->dil[l], m->C);
  fwo_state_reset(st);
  return st;
}

void fwo_state_reset(fwo_state *st) {
  st->t = 0;
  for (int b = 0; b < st->batch; ++b) {
    st->last[b] = st->seed_input;
    for (int l = 0; l < st->m->L; ++l) fifo_zero(&st->queues[(size_t)b * st->m->L + l]);
  }
}

void fwo_state_free(fwo_state *st) {
  if (!st) return;
  for (size_t i = 0; i < (size_t)st->batch * st->m->L; ++i) free(st->queues[i].buf);
  free(st->queues);
  free(st->last);
  free(st);
}

long long fwo_state_t(const fwo_state *st) { return st->t; }

/* One step of the generation model for one stream (Section 2.2):
 * pop phase, computation of the output and the new recurrent states, push phase.
 * popped: [L][(w-1) C]; states: [L+1][C] (states[l] = x^l_t); s: [S]. */
static void model_step(const fwo_model *m, fifo *q, int in, double *logits, double *popped,
                       double *states, double *s, double *work) {
  const int L = m->L, C = m->C, w = width(m);
  /* pop phase: the oldest cached state of every queue (x^{l-1}_{t-(w-1)d}); with w > 2
   * also the states d, 2d, ... behind it (x^{l-1}_{t-(w-2)d}, ..., x^{l-1}_{t-d}) */
  for (int l = 0; l < L; ++l) {
    double *r = popped + (size_t)l * (w - 1) * C;
    for (int k = 1; k < w - 1; ++k) fifo_peek(&q[l], k * m->dil[l], r + (size_t)k * C);
    fifo_pop(&q[l], r);
  }
  /* current input h^0_e and the new recurrent states */
  embed_apply(m, in, states);
  if (m->kind == FWO_GATED) memset(s, 0, sizeof(double) * m->S);
  for (int l = 0; l < L; ++l)
    layer_apply(m, l, popped + (size_t)l * (w - 1) * C, states + (size_t)l * C, states + (size_t)(l + 1) * C, s,
                work);
  head_apply(m, states + (size_t)L * C, s, logits, work);
  /* push phase: the queue feeding layer l receives x^{l-1}_t */
  for (int l = 0; l < L; ++l) fifo_push(&q[l], states + (size_t)l * C);
}

int fwo_sample(const float *lg, int Q, float u) {
  float mx = lg[0];
  for (int k = 1; k < Q; ++k) mx = lg[k] > mx ? lg[k] : mx;
  float Z = 0.0f;
  for (int k = 0; k < Q; ++k) Z += expf(lg[k] - mx);
  const float target = u * Z;
  float S = 0.0f;
  for (int k = 0; k < Q; ++k) {
    S += expf(lg[k] - mx);
    if (target < S) return k;
  }
  return Q - 1;
}

void fwo_cdf(const double *lg, int Q, double *cdf) {
  double mx = lg[0];
  for (int k = 1; k < Q; ++k) mx = lg[k] > mx ? lg[k] : mx;
  double S = 0.0;
  for (int k = 0; k < Q; ++k) { S += exp(lg[k] - mx); cdf[k] = S; }
  for (int k = 0; k < Q; ++k) cdf[k] /= S;
}

typedef struct {
  double *popped, *states, *s, *work, *logits;
  float *lf;
} scratch;

static void scratch_init(const fwo_model *m, scratch *w) {
  w->popped = (double *)malloc(sizeof(double) * (size_t)m->L * (width(m) - 1) * m->C + 8);
  w->states = (double *)malloc(sizeof(double) * (size_t)(m->L + 1) * m->C + 8);
  w->s = (double *)malloc(sizeof(double) * ((size_t)m->S + 1));
  w->work = (double *)malloc(sizeof(double) * work_doubles(m));
  w->logits = (double *)malloc(sizeof(double) * m->Q);
  w->lf = (float *)malloc(sizeof(float) * m->Q);
}
static void scratch_free(scratch *w) {
  free(w->popped); free(w->states); free(w->s); free(w->work); free(w->logits); free(w->lf);
}

int fwo_generate(const fwo_model *m, fwo_state *st, int n_steps, const float *u, int *samples,
                 double *logits) {
  if (!m || !st || n_steps < 0 || (n_steps > 0 && (!u || !samples))) return -1;
  const int B = st->batch, L = m->L, Q = m->Q;
#pragma omp parallel for schedule(dynamic, 1) if (!m->products && B > 1)
  for (int b = 0; b < B; ++b) {
    scratch w;
    scratch_init(m, &w);
    fifo *q = &st->queues[(size_t)b * L];
    int in = st->last[b];
    for (int i = 0; i < n_steps; ++i) {
      model_step(m, q, in, w.logits, w.popped, w.states, w.s, w.work);
      if (logits) memcpy(logits + ((size_t)b * n_steps + i) * Q, w.logits, sizeof(double) * Q);
      for (int k = 0; k < Q; ++k) w.lf[k] = (float)w.logits[k];
      in = fwo_sample(w.lf, Q, u[(size_t)b * n_steps + i]);
      samples[(size_t)b * n_steps + i] = in; /* fed back as the next input (Section 1) */
    }
    st->last[b] = in;
    scratch_free(&w);
  }
  st->t += n_steps;
  return 0;
}

/* Online prediction (the use named at the end of Section 1 and in Section 4): the
 * cached step of Section 2.2 continues from the state, but the sample that
 * follows each step is observed, not drawn.  Step i consumes the pending input,
 * reports the distribution predicted for the next sample, and then takes
 * inputs[b][i] as that sample, which becomes the pending input. */
int fwo_step_forced(const fwo_model *m, fwo_state *st, int n_steps, const int *inputs, double *logits) {
  if (!m || !st || n_steps < 0 || (n_steps > 0 && (!inputs || !logits))) return -1;
  const int B = st->batch, L = m->L, Q = m->Q;
#pragma omp parallel for schedule(dynamic, 1) if (!m->products && B > 1)
  for (int b = 0; b < B; ++b) {
    scratch w;
    scratch_init(m, &w);
    fifo *q = &st->queues[(size_t)b * L];
    int in = st->last[b];
    for (int i = 0; i < n_steps; ++i) {
      model_step(m, q, in, w.logits, w.popped, w.states, w.s, w.work);
      memcpy(logits + ((size_t)b * n_steps + i) * Q, w.logits, sizeof(double) * Q);
      in = inputs[(size_t)b * n_steps + i];
    }
    st->last[b] = in;
    scratch_free(&w);
  }
  st->t += n_steps;
  return 0;
}

int fwo_teacher_forced(const fwo_model *m, int B, int T, const int *inputs, double *logits) {
  if (!m || B <= 0 || T < 0 || (T > 0 && (!inputs || !logits))) return -1;
  const int L = m->L, Q = m->Q;
#pragma omp parallel for schedule(dynamic, 1) if (!m->products && B > 1)
  for (int b = 0; b < B; ++b) {
    scratch w;
    scratch_init(m, &w);
    fifo *q = (fifo *)malloc(sizeof(fifo) * L);
    for (int l = 0; l < L; ++l) fifo_init(&q[l], (width(m) - 1) * m->dil[l], m->C);
    for (int t = 0; t < T; ++t)
      model_step(m, q, inputs[(size_t)b * T + t], logits + ((size_t)b * T + t) * Q, w.popped, w.states,
                 w.s, w.work);
    for (int l = 0; l < L; ++l) free(q[l].buf);
    free(q);
    scratch_free(&w);
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Parallel form: layer l evaluated for all t from layer l-1's full sequence,
 * with x^{l-1}_{t-kd} = 0 for t < kd.                                       */
int fwo_parallel(const fwo_model *m, int B, int T, const int *inputs, double *logits) {
  if (!m || B <= 0 || T < 0 || (T > 0 && (!inputs || !logits))) return -1;
  const int L = m->L, C = m->C, Q = m->Q, S = m->S, w = width(m);
#pragma omp parallel for schedule(dynamic, 1) if (!m->products && B > 1)
  for (int b = 0; b < B; ++b) {
    double *rtaps = (double *)malloc(sizeof(double) * (size_t)(w - 1) * C + 8);
    double *prev = (double *)malloc(sizeof(double) * (size_t)T * C + 8);
    double *next = (double *)malloc(sizeof(double) * (size_t)T * C + 8);
    double *ssum = (double *)calloc((size_t)T * (S > 0 ? S : 1), sizeof(double));
    double *zero = (double *)calloc(C, sizeof(double));
    double *work = (double *)malloc(sizeof(double) * work_doubles(m));
    for (int t = 0; t < T; ++t) embed_apply(m, inputs[(size_t)b * T + t], prev + (size_t)t * C);
    for (int l = 0; l < L; ++l) {
      const int d = m->dil[l];
      for (int t = 0; t < T; ++t) {
        for (int k = 0; k < w - 1; ++k) {
          const int tau = t - (w - 1 - k) * d;
          memcpy(rtaps + (size_t)k * C, tau >= 0 ? prev + (size_t)tau * C : zero, sizeof(double) * C);
        }
        layer_apply(m, l, rtaps, prev + (size_t)t * C, next + (size_t)t * C, ssum + (size_t)t * S, work);
      }
      double *tmp = prev; prev = next; next = tmp;
    }
    for (int t = 0; t < T; ++t)
      head_apply(m, prev + (size_t)t * C, ssum + (size_t)t * S, logits + ((size_t)b * T + t) * Q, work);
    free(rtaps); free(prev); free(next); free(ssum); free(zero); free(work);
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Naive form (Fig. 1): every node recomputed from its two children, no cache. */
static void naive_node(const fwo_model *m, const int *inputs, int l, int tau, double *out) {
  const int C = m->C;
  if (tau < 0) { memset(out, 0, sizeof(double) * C); return; } /* zero queues = zero padding */
  if (l == 0) { embed_apply(m, inputs[tau], out); return; }
  const int w = width(m);
  double *r = (double *)malloc(sizeof(double) * (size_t)(w - 1) * C);
  double *x = (double *)malloc(sizeof(double) * C);
  double *s = (double *)calloc(m->S > 0 ? m->S : 1, sizeof(double));
  double *work = (double *)malloc(sizeof(double) * work_doubles(m));
  for (int k = 0; k < w - 1; ++k) naive_node(m, inputs, l - 1, tau - (w - 1 - k) * m->dil[l - 1], r + (size_t)k * C);
  naive_node(m, inputs, l - 1, tau, x);
  layer_apply(m, l - 1, r, x, out, s, work); /* skip output of interior nodes is discarded */
  free(r); free(x); free(s); free(work);
}

int fwo_naive(const fwo_model *m, const int *inputs, int t, double *logits) {
  if (!m || !inputs || !logits || t < 0) return -1;
  const int C = m->C, S = m->S;
  double *work = (double *)malloc(sizeof(double) * work_doubles(m));
  double *top = (double *)malloc(sizeof(double) * C);
  double *s = (double *)calloc(S > 0 ? S : 1, sizeof(double));
  if (m->kind != FWO_GATED) {
    naive_node(m, inputs, m->L, t, top);
  } else {
    /* the skip sum needs z^l_t of every layer: walk the spine h^0_t .. h^L_t,
     * each recurrent operand recomputed from scratch by the tree */
    const int w = width(m);
    double *x = (double *)malloc(sizeof(double) * C);
    double *r = (double *)malloc(sizeof(double) * (size_t)(w - 1) * C);
    naive_node(m, inputs, 0, t, x);
    for (int l = 0; l < m->L; ++l) {
      for (int k = 0; k < w - 1; ++k) naive_node(m, inputs, l, t - (w - 1 - k) * m->dil[l], r + (size_t)k * C);
      layer_apply(m, l, r, x, top, s, work);
      memcpy(x, top, sizeof(double) * C);
    }
    free(x); free(r);
  }
  head_apply(m, top, s, logits, work);
  free(work); free(top); free(s);
  return 0;
}
