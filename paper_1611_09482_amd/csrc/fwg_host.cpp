// Host side of libfwg.so: descriptor validation, workspace planning, weight
// repacking, queue management and step-kernel launches.  Every check runs
// before anything is enqueued; the library never allocates device memory.
#include <hip/hip_runtime.h>

#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <new>
#include <vector>

#include "fwg.h"
#include "fwg_internal.h"

using namespace fwg;

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return code;
}

#define HIP_TRY(expr)                                                                      \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess) return fail(FWG_EHIP, "%s: %s", #expr, hipGetErrorString(e_));   \
  } while (0)

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

struct Plan {
  int kind, dtype, Q, C, S, H, L, bmax, seed_input, Co, es, rpw;
  int regime;
  int brows;              // queue rows per slot (max_batch, padded to whole blocks for the MFMA family)
  size_t off_frags, off_embT, off_bias, off_ptrtab;
  long long queue_elems;  // sum(d_l) * bmax * C
  size_t off_layers, off_embed, off_embed_b, off_head, off_head_b, off_out, off_out_b;
  std::vector<size_t> off_conv, off_conv_b, off_res, off_res_b, off_skip, off_skip_b;
  std::vector<long long> ring_off;
  size_t off_ring_gen, off_ring_tf, off_last, total;
  size_t lds_bytes;
};

bool kblock_ok(int K, int N, int kb_elems) {
  if (K % kb_elems) return false;
  const int nkb = K / kb_elems;
  if (N >= kThreads) return true;
  if (kThreads % N) return false;
  return nkb % (kThreads / N) == 0;
}

// Validate a descriptor and compute the workspace layout.
int make_plan(const fwg_desc *d, Plan *p) {
  if (!d) return fail(FWG_EINVAL, "desc is NULL");
  if (d->kind < FWG_RELU || d->kind > FWG_GATED) return fail(FWG_EINVAL, "unknown kind %d", d->kind);
  if (d->dtype != FWG_F32 && d->dtype != FWG_BF16) return fail(FWG_EINVAL, "unknown dtype %d", d->dtype);
  if (d->n_layers <= 0) return fail(FWG_EINVAL, "n_layers must be >= 1 (got %d)", d->n_layers);
  if (d->n_layers > kMaxLayers) return fail(FWG_EUNSUPPORTED, "n_layers > %d", kMaxLayers);
  if (!d->dilations) return fail(FWG_EINVAL, "dilations is NULL");
  if (d->channels <= 0) return fail(FWG_EINVAL, "channels must be >= 1");
  if (d->max_batch <= 0) return fail(FWG_EINVAL, "max_batch must be >= 1");
  if (d->n_classes <= 0) return fail(FWG_EINVAL, "n_classes must be >= 1");
  if (d->seed_input < 0 || d->seed_input >= d->n_classes) return fail(FWG_EINVAL, "seed_input out of range");
  if (d->kind == FWG_GATED && (d->skip_channels <= 0 || d->head_channels <= 0))
    return fail(FWG_EINVAL, "gated model needs skip_channels and head_channels >= 1");
  long long dsum = 0;
  for (int l = 0; l < d->n_layers; ++l) {
    if (d->dilations[l] < 1) return fail(FWG_EINVAL, "dilation[%d] = %d < 1", l, d->dilations[l]);
    dsum += d->dilations[l];
  }
  if (d->n_classes != 256) return fail(FWG_EUNSUPPORTED, "n_classes must be 256 (got %d)", d->n_classes);

  p->kind = d->kind;
  p->dtype = d->dtype;
  p->Q = d->n_classes;
  p->C = d->channels;
  p->S = d->kind == FWG_GATED ? d->skip_channels : 0;
  p->H = d->kind == FWG_GATED ? d->head_channels : 0;
  p->L = d->n_layers;
  p->bmax = d->max_batch;
  p->seed_input = d->seed_input;
  p->Co = d->kind == FWG_GATED ? 2 * p->C : p->C;
  p->es = d->dtype == FWG_BF16 ? 2 : 4;

  // shapes the K-blocked products support
  const int kb = valu_kb_elems(p->dtype);
  bool ok = kblock_ok(2 * p->C, p->Co, kb) && kblock_ok(p->kind == FWG_GATED ? p->H : p->C, p->Q, kb);
  if (p->kind == FWG_GATED)
    ok = ok && kblock_ok(p->C, p->C, kb) && kblock_ok(p->C, p->S, kb) && kblock_ok(p->S, p->H, kb);
  if (!ok)
    return fail(FWG_EUNSUPPORTED,
                "unsupported shape: every product needs K a multiple of %d, and an output width that "
                "divides 256 (with K/%d divisible by 256/N) or is at least 256",
                kb, kb);

  // rows per block: as many streams per block as LDS allows, at most 8, fewer for tiny batches
  int rpw = 8;
  while (rpw > 1 && rpw > p->bmax) rpw >>= 1;
  for (;; rpw >>= 1) {
    const ValuLds lay = valu_lds_layout(p->kind, p->C, p->S, p->H, p->Q, p->L, rpw);
    p->lds_bytes = (size_t)lay.total_floats * 4;
    if (p->lds_bytes <= 160 * 1024 || rpw == 1) break;
  }
  if (p->lds_bytes > 160 * 1024) return fail(FWG_EUNSUPPORTED, "model too wide for one block's LDS");
  p->rpw = rpw;

  // kernel family: the MFMA kernel covers gated bf16 stacks with R=64, S=H=512
  p->regime = REGIME_VALU;
  const char *force = getenv("FWG_REGIME");
  const bool mfma_shape = p->kind == FWG_GATED && p->dtype == FWG_BF16 && p->C == kMfR && p->S == kMfS &&
                          p->H == kMfH && p->Q == 256 && p->L <= kMfMaxLayers &&
                          mfma_lds_bytes(p->L) <= 160 * 1024;
  if (mfma_shape && !(force && strcmp(force, "valu") == 0)) p->regime = REGIME_MFMA;
  p->brows = p->regime == REGIME_MFMA ? (p->bmax + kMfRows - 1) / kMfRows * kMfRows : p->bmax;

  // workspace layout
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t at = off; off = align_up(off + bytes); return at; };
  p->off_layers = take(sizeof(LayerDev) * p->L);
  p->off_frags = p->off_embT = p->off_bias = p->off_ptrtab = 0;
  if (p->regime == REGIME_MFMA) {
    p->off_frags = take(mfma_frag_bytes(p->L));
    p->off_embT = take((size_t)p->Q * p->C * 2);
    p->off_bias = take(sizeof(float) * mfma_bias_floats(p->L));
    p->off_ptrtab = take(sizeof(void *) * 3 * p->L);
  }
  p->off_embed = take((size_t)p->Q * p->C * p->es);
  p->off_embed_b = take(sizeof(float) * p->C);
  p->off_conv.resize(p->L); p->off_conv_b.resize(p->L);
  p->off_res.assign(p->L, 0); p->off_res_b.assign(p->L, 0); p->off_skip.assign(p->L, 0); p->off_skip_b.assign(p->L, 0);
  for (int l = 0; l < p->L; ++l) {
    p->off_conv[l] = take((size_t)p->Co * 2 * p->C * p->es);
    p->off_conv_b[l] = take(sizeof(float) * p->Co);
    if (p->kind == FWG_GATED) {
      p->off_res[l] = take((size_t)p->C * p->C * p->es);
      p->off_res_b[l] = take(sizeof(float) * p->C);
      p->off_skip[l] = take((size_t)p->S * p->C * p->es);
      p->off_skip_b[l] = take(sizeof(float) * p->S);
    }
  }
  p->off_head = p->kind == FWG_GATED ? take((size_t)p->H * p->S * p->es) : 0;
  p->off_head_b = p->kind == FWG_GATED ? take(sizeof(float) * p->H) : 0;
  const int Kout = p->kind == FWG_GATED ? p->H : p->C;
  p->off_out = take((size_t)p->Q * Kout * p->es);
  p->off_out_b = take(sizeof(float) * p->Q);
  p->ring_off.resize(p->L);
  long long acc = 0;
  for (int l = 0; l < p->L; ++l) {
    p->ring_off[l] = acc;
    acc += (long long)d->dilations[l] * p->brows * p->C;
  }
  p->queue_elems = acc;
  (void)dsum;
  p->off_ring_gen = take((size_t)acc * p->es);
  p->off_ring_tf = take((size_t)acc * p->es);
  p->off_last = take(sizeof(int32_t) * p->bmax);
  p->total = off;
  return FWG_OK;
}

}  // namespace

struct fwg_handle {
  Plan plan;
  std::vector<int32_t> dil;
  char *ws;
  hipStream_t stream;
  long long t;
  int bound_batch;  // -1: not bound since the last reset
};

namespace {

int enqueue_reset(fwg_handle *h) {
  const Plan &p = h->plan;
  HIP_TRY(launch_fill_zero(h->ws + p.off_ring_gen, (size_t)p.queue_elems * p.es, h->stream));
  HIP_TRY(launch_fill_i32((int32_t *)(h->ws + p.off_last), p.seed_input, p.bmax, h->stream));
  h->t = 0;
  h->bound_batch = -1;
  return FWG_OK;
}

StepArgs base_args(const fwg_handle *h) {
  const Plan &p = h->plan;
  StepArgs a;
  memset(&a, 0, sizeof(a));
  a.layers = (const LayerDev *)(h->ws + p.off_layers);
  a.embed = h->ws + p.off_embed;
  a.embed_b = (const float *)(h->ws + p.off_embed_b);
  a.head = p.kind == FWG_GATED ? h->ws + p.off_head : nullptr;
  a.head_b = p.kind == FWG_GATED ? (const float *)(h->ws + p.off_head_b) : nullptr;
  a.out = h->ws + p.off_out;
  a.out_b = (const float *)(h->ws + p.off_out_b);
  a.last = (int32_t *)(h->ws + p.off_last);
  a.bmax = p.brows;
  if (p.regime == REGIME_MFMA) {
    a.mf_frags = h->ws + p.off_frags;
    a.mf_embT = h->ws + p.off_embT;
    a.mf_bias = (const float *)(h->ws + p.off_bias);
  }
  a.kind = p.kind;
  a.dtype = p.dtype;
  a.C = p.C;
  a.S = p.S;
  a.H = p.H;
  a.Q = p.Q;
  a.L = p.L;
  return a;
}

}  // namespace

extern "C" {

const char *fwg_last_error(void) { return g_err; }

int fwg_workspace_size(const fwg_desc *desc, size_t *bytes) {
  if (!bytes) return fail(FWG_EINVAL, "bytes is NULL");
  Plan p;
  int rc = make_plan(desc, &p);
  if (rc != FWG_OK) return rc;
  *bytes = p.total;
  return FWG_OK;
}

int fwg_create(const fwg_desc *desc, const fwg_weights *w, void *workspace, size_t ws_bytes, void *hip_stream,
               fwg_handle **out) {
  if (!out) return fail(FWG_EINVAL, "out is NULL");
  *out = nullptr;
  Plan p;
  int rc = make_plan(desc, &p);
  if (rc != FWG_OK) return rc;
  if (!w) return fail(FWG_EINVAL, "weights is NULL");
  if (!workspace) return fail(FWG_EINVAL, "workspace is NULL");
  if (((uintptr_t)workspace) % kAlign) return fail(FWG_ENOSPACE, "workspace must be %zu-byte aligned", kAlign);
  if (ws_bytes < p.total) return fail(FWG_ENOSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, p.total);
  if (!w->embed || !w->conv || !w->out) return fail(FWG_EINVAL, "embed, conv and out weights are required");
  for (int l = 0; l < p.L; ++l)
    if (!w->conv[l]) return fail(FWG_EINVAL, "conv[%d] is NULL", l);
  if (p.kind == FWG_GATED) {
    if (!w->res || !w->skip || !w->head) return fail(FWG_EINVAL, "gated model needs res, skip and head weights");
    for (int l = 0; l < p.L; ++l)
      if (!w->res[l] || !w->skip[l]) return fail(FWG_EINVAL, "res/skip[%d] is NULL", l);
  }

  fwg_handle *h = new (std::nothrow) fwg_handle();
  if (!h) return fail(FWG_EINVAL, "out of host memory");
  h->plan = p;
  h->dil.assign(desc->dilations, desc->dilations + p.L);
  h->ws = (char *)workspace;
  h->stream = (hipStream_t)hip_stream;
  h->t = 0;
  h->bound_batch = -1;

  auto cleanup_fail = [&](int code) { delete h; return code; };
#define TRY_OR_FREE(expr)                                                                   \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess) return cleanup_fail(fail(FWG_EHIP, "%s: %s", #expr, hipGetErrorString(e_))); \
  } while (0)

  char *ws = h->ws;
  hipStream_t s = h->stream;
  const int dt = p.dtype, C = p.C;
  TRY_OR_FREE(launch_repack(w->embed, ws + p.off_embed, REPACK_EMBED, dt, p.Q, C, C, s));
  TRY_OR_FREE(launch_copy_bias(w->embed_b, (float *)(ws + p.off_embed_b), C, s));
  std::vector<LayerDev> table(p.L);
  for (int l = 0; l < p.L; ++l) {
    TRY_OR_FREE(launch_repack(w->conv[l], ws + p.off_conv[l], REPACK_CONV, dt, 2 * C, p.Co, C, s));
    TRY_OR_FREE(launch_copy_bias(w->conv_b ? w->conv_b[l] : nullptr, (float *)(ws + p.off_conv_b[l]), p.Co, s));
    LayerDev &ld = table[l];
    memset(&ld, 0, sizeof(ld));
    ld.conv = ws + p.off_conv[l];
    ld.conv_b = (const float *)(ws + p.off_conv_b[l]);
    if (p.kind == FWG_GATED) {
      TRY_OR_FREE(launch_repack(w->res[l], ws + p.off_res[l], REPACK_LINEAR, dt, C, C, C, s));
      TRY_OR_FREE(launch_copy_bias(w->res_b ? w->res_b[l] : nullptr, (float *)(ws + p.off_res_b[l]), C, s));
      TRY_OR_FREE(launch_repack(w->skip[l], ws + p.off_skip[l], REPACK_LINEAR, dt, C, p.S, C, s));
      TRY_OR_FREE(launch_copy_bias(w->skip_b ? w->skip_b[l] : nullptr, (float *)(ws + p.off_skip_b[l]), p.S, s));
      ld.res = ws + p.off_res[l];
      ld.res_b = (const float *)(ws + p.off_res_b[l]);
      ld.skip = ws + p.off_skip[l];
      ld.skip_b = (const float *)(ws + p.off_skip_b[l]);
    }
    ld.ring_off = p.ring_off[l];
    ld.dil = h->dil[l];
  }
  if (p.kind == FWG_GATED) {
    TRY_OR_FREE(launch_repack(w->head, ws + p.off_head, REPACK_LINEAR, dt, p.S, p.H, C, s));
    TRY_OR_FREE(launch_copy_bias(w->head_b, (float *)(ws + p.off_head_b), p.H, s));
  }
  const int Kout = p.kind == FWG_GATED ? p.H : C;
  TRY_OR_FREE(launch_repack(w->out, ws + p.off_out, REPACK_LINEAR, dt, Kout, p.Q, C, s));
  TRY_OR_FREE(launch_copy_bias(w->out_b, (float *)(ws + p.off_out_b), p.Q, s));
  TRY_OR_FREE(hipMemcpyAsync(ws + p.off_layers, table.data(), sizeof(LayerDev) * p.L, hipMemcpyHostToDevice, s));
  std::vector<const void *> ptrs;
  if (p.regime == REGIME_MFMA) {
    char *frags = ws + p.off_frags;
    // layers first: a layer also writes fragments into the previous stage and the last head stage
    for (int l = 0; l < p.L; ++l)
      TRY_OR_FREE(launch_mfma_repack_layer(w->conv[l], w->res[l], w->skip[l], l, p.L, frags, s));
    TRY_OR_FREE(launch_mfma_repack_head(w->head, w->out, p.L, frags, s));
    TRY_OR_FREE(launch_mfma_embed_table(w->embed, ws + p.off_embT, s));
    ptrs.resize(3 * p.L, nullptr);
    for (int l = 0; l < p.L; ++l) {
      ptrs[l] = w->conv_b ? w->conv_b[l] : nullptr;
      ptrs[p.L + l] = w->res_b ? w->res_b[l] : nullptr;
      ptrs[2 * p.L + l] = w->skip_b ? w->skip_b[l] : nullptr;
    }
    TRY_OR_FREE(hipMemcpyAsync(ws + p.off_ptrtab, ptrs.data(), sizeof(void *) * 3 * p.L, hipMemcpyHostToDevice, s));
    const float *const *pt = (const float *const *)(ws + p.off_ptrtab);
    TRY_OR_FREE(launch_mfma_bias_block(pt, pt + p.L, pt + 2 * p.L, w->head_b, w->out_b, w->embed_b, p.L,
                                       (float *)(ws + p.off_bias), s));
    TRY_OR_FREE(set_mfma_lds_limit(mfma_lds_bytes(p.L)));
  }
  if (p.lds_bytes > 64 * 1024) TRY_OR_FREE(set_valu_lds_limit(p.lds_bytes));
  int rr = enqueue_reset(h);
  if (rr != FWG_OK) return cleanup_fail(rr);
  // the layer table is copied from host memory owned by this call
  TRY_OR_FREE(hipStreamSynchronize(s));
#undef TRY_OR_FREE
  *out = h;
  return FWG_OK;
}

int fwg_reset_queues(fwg_handle *h) {
  if (!h) return fail(FWG_EINVAL, "handle is NULL");
  return enqueue_reset(h);
}

int fwg_generate(fwg_handle *h, int32_t batch, int32_t n_steps, const float *uniforms, int32_t *samples) {
  if (!h) return fail(FWG_EINVAL, "handle is NULL");
  const Plan &p = h->plan;
  if (batch < 1 || batch > p.bmax) return fail(FWG_EINVAL, "batch %d outside [1, %d]", batch, p.bmax);
  if (n_steps < 0) return fail(FWG_EINVAL, "n_steps < 0");
  if (h->bound_batch >= 0 && h->bound_batch != batch)
    return fail(FWG_ESTATE, "batch %d differs from %d used since the last reset", batch, h->bound_batch);
  if (n_steps == 0) return FWG_OK;
  if (!uniforms || !samples) return fail(FWG_EINVAL, "uniforms and samples are required");
  StepArgs a = base_args(h);
  a.ring = h->ws + p.off_ring_gen;
  a.uniforms = uniforms;
  a.samples = samples;
  a.t0 = h->t;
  a.n_steps = n_steps;
  a.batch = batch;
  a.mode = MODE_GENERATE;
  HIP_TRY(p.regime == REGIME_MFMA ? launch_mfma_step(a, h->stream) : launch_valu_step(a, p.rpw, p.lds_bytes, h->stream));
  h->bound_batch = batch;
  h->t += n_steps;
  return FWG_OK;
}

int fwg_teacher_forced(fwg_handle *h, int32_t batch, int32_t seq_len, const int32_t *inputs, float *logits) {
  if (!h) return fail(FWG_EINVAL, "handle is NULL");
  const Plan &p = h->plan;
  if (batch < 1 || batch > p.bmax) return fail(FWG_EINVAL, "batch %d outside [1, %d]", batch, p.bmax);
  if (seq_len < 0) return fail(FWG_EINVAL, "seq_len < 0");
  if (seq_len == 0) return FWG_OK;
  if (!inputs || !logits) return fail(FWG_EINVAL, "inputs and logits are required");
  HIP_TRY(launch_fill_zero(h->ws + p.off_ring_tf, (size_t)p.queue_elems * p.es, h->stream));
  StepArgs a = base_args(h);
  a.ring = h->ws + p.off_ring_tf;
  a.inputs = inputs;
  a.logits = logits;
  a.t0 = 0;
  a.n_steps = seq_len;
  a.batch = batch;
  a.mode = MODE_TEACHER;
  HIP_TRY(p.regime == REGIME_MFMA ? launch_mfma_step(a, h->stream) : launch_valu_step(a, p.rpw, p.lds_bytes, h->stream));
  return FWG_OK;
}

int fwg_step_forced(fwg_handle *h, int32_t batch, int32_t n_steps, const int32_t *inputs, float *logits) {
  if (!h) return fail(FWG_EINVAL, "handle is NULL");
  const Plan &p = h->plan;
  if (batch < 1 || batch > p.bmax) return fail(FWG_EINVAL, "batch %d outside [1, %d]", batch, p.bmax);
  if (n_steps < 0) return fail(FWG_EINVAL, "n_steps < 0");
  if (h->bound_batch >= 0 && h->bound_batch != batch)
    return fail(FWG_ESTATE, "batch %d differs from %d used since the last reset", batch, h->bound_batch);
  if (n_steps == 0) return FWG_OK;
  if (!inputs || !logits) return fail(FWG_EINVAL, "inputs and logits are required");
  StepArgs a = base_args(h);
  a.ring = h->ws + p.off_ring_gen;
  a.inputs = inputs;
  a.logits = logits;
  a.t0 = h->t;
  a.n_steps = n_steps;
  a.batch = batch;
  a.mode = MODE_ONLINE;
  HIP_TRY(p.regime == REGIME_MFMA ? launch_mfma_step(a, h->stream) : launch_valu_step(a, p.rpw, p.lds_bytes, h->stream));
  h->bound_batch = batch;
  h->t += n_steps;
  return FWG_OK;
}

int fwg_destroy(fwg_handle *h) {
  delete h;
  return FWG_OK;
}

const char *fwg_regime(const fwg_handle *h) {
  if (!h) return "";
  return h->plan.regime == REGIME_MFMA ? "mfma_bf16_r64_s512" : "valu";
}

}  // extern "C"
