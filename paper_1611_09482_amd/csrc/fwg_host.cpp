// Host side of libfwg.so: descriptor validation, workspace planning, weight
// repacking, queue management and step-kernel launches.  Every check runs
// before anything is enqueued; the library never allocates device memory.
#include <hip/hip_runtime.h>

#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <new>
#include <vector>

#include "fwg.h"
#include "fwg_internal.h"
#include "fwg_par.h"
#include "fwg_valu.h"
#include "fwg_wave.h"
#include "fwg_chain.h"
#include "fwg_wide.h"

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
  size_t valu_block;      // bytes of one layer's weight + bias block (general step kernels)
  int valu_wbytes;        // the block when the general step kernels stage it in LDS, else 0
  int w;                  // filter width: taps per dilated product
  int regime;
  int brows;              // queue rows per slot (max_batch, padded to whole blocks for the MFMA family)
  size_t off_frags, off_embT, off_bias, off_ptrtab;
  size_t off_comm, off_sticky;  // split MFMA family: exchange words and the sticky abort word
  long long queue_elems;  // sum(d_l) * bmax * C
  size_t off_layers, off_embed, off_embed_b, off_head, off_head_b, off_out, off_out_b;
  std::vector<size_t> off_conv, off_conv_b, off_res, off_res_b, off_skip, off_skip_b;
  std::vector<long long> ring_off;
  size_t off_ring_gen, off_ring_tf, off_last, total;
  size_t lds_bytes;
  // time-parallel path (forced sequences): operand-typed [N][K] weights and chunk buffers
  bool par_ok;
  int par_tc;             // steps per chunk; a chunk holds brows * par_tc rows at most
  std::vector<size_t> off_pconv, off_pconv_b, off_pres;
  size_t off_pskip, off_pskip_b, off_phead, off_pout;
  size_t off_px[3], off_pxb[3], off_pz, off_psb, off_phb;  // three rotating row buffers
  // naive generator: the nodes of the output's dependency tree (Fig. 1), level 0 = inputs
  bool nv_ok;
  std::vector<int> nv_n;         // [L + 1] distinct nodes per level
  std::vector<size_t> nv_tab;    // [L + 1] int offset of the level's tables (toff; then w tap-source rows for l >= 1)
  std::vector<int32_t> nv_host;  // the tables, uploaded at create
  long long nv_nodes;            // layer nodes per sample: sum of nv_n[1..L]
  int nv_hc;                     // input-history capacity per stream (power of two >= receptive field)
  size_t off_nv, off_hist, off_ztop, off_nlogits;
  // wave-per-stream family: the weight image
  WaveArgs wave;
  size_t off_wave;
  // chain family: the weight image and the launch's LDS bytes
  ChainArgs chain;
  size_t off_chain, chain_lds;
  // gated chain family: packed weights (bytes) and the launch's LDS bytes
  size_t off_cg, cg_bytes, cg_lds;
  size_t cp_lds;  // pair variant: the launch's LDS bytes
  // wide family: packed weights and tables, the launch's LDS and exchange-region bytes
  WideArgs wide;
  size_t wide_lds, wide_comm;
  size_t off_wl, off_wo, off_wembT, off_wembb, off_wconvb, off_woutb;
};

// Layout of the wave family's weight image and per-wave scratch; false when the model does not fit
// (every product at most 256 wide, K multiples of 4, pops of a step in 16 registers per lane, image
// and four waves' scratch in 160 KB of LDS).
bool wave_layout(const Plan &p, WaveArgs *g) {
  const bool gated = p.kind == FWG_GATED;
  const int C = p.C, S = p.S, H = p.H, Q = p.Q, L = p.L, w = p.w, Co = p.Co;
  const int Ktop = gated ? H : C;
  if (C % 4 || (gated && (S % 4 || H % 4)) || C > 256 || (gated && (S > 256 || H > 256)) || Q != 256) return false;
  if (L * (w - 1) > 64 || (long long)L * (w - 1) * ((C + 63) / 64) > 16) return false;
  auto r4 = [](long long n) { return (int)((n + 3) & ~3ll); };
  long long o = 0;
  auto take = [&](long long n) { const long long at = o; o += r4(n); return (int)at; };
  g->o_emb = take((long long)Q * C);
  g->o_embb = take(C);
  g->o_layer = (int)o;
  long long lo = 0;
  auto ltake = [&](long long n) { const long long at = lo; lo += r4(n); return (int)at; };
  ltake((long long)w * C * Co);
  g->o_convb = ltake(Co);
  g->o_res = gated ? ltake((long long)C * C) : 0;
  g->o_resb = gated ? ltake(C) : 0;
  g->o_skip = gated ? ltake((long long)C * S) : 0;
  g->o_skipb = gated ? ltake(S) : 0;
  g->layer_floats = (int)lo;
  o += lo * L;
  g->o_head = gated ? take((long long)S * H) : 0;
  g->o_headb = gated ? take(H) : 0;
  g->o_out = take((long long)Ktop * Q);
  g->o_outb = take(Q);
  g->image_floats = r4(o);
  g->ain_floats = r4((long long)L * w * C);  // the layer inputs of every layer (pops land once per step)
  g->c_floats = r4(C);
  g->s_floats = gated ? r4(S) : 0;
  g->h_floats = gated ? r4(H) : 0;
  g->scr_floats = g->ain_floats + 2 * g->c_floats + 2 * g->s_floats + g->h_floats + r4(Q);
  const long long bytes = 4ll * ((long long)g->image_floats + 4ll * g->scr_floats);
  return o < (1ll << 30) && bytes <= 160 * 1024;
}

// Node sets of the tree of Fig. 1 for the output at offset 0: level L holds {0}; level l - 1 holds the
// level-l offsets minus j d_l for j = 0 .. w - 1 (each distinct offset once).  Tables per level l >= 1:
// the offsets, then for every tap k the index in level l - 1 of offset - (w - 1 - k) d_l.  Fills nv_n,
// nv_tab, nv_host and nv_nodes.
void naive_tables(Plan *p, const int32_t *dil) {
  const int L = p->L, w = p->w;
  std::vector<std::vector<int>> P(L + 1);
  P[L] = {0};
  for (int l = L; l >= 1; --l) {
    std::vector<int> v = P[l];
    for (int j = 1; j < w; ++j)
      for (int o : P[l]) v.push_back(o - j * dil[l - 1]);
    std::sort(v.begin(), v.end());
    v.erase(std::unique(v.begin(), v.end()), v.end());
    P[l - 1] = v;
  }
  p->nv_n.assign(L + 1, 0);
  p->nv_tab.assign(L + 1, 0);
  p->nv_host.clear();
  p->nv_nodes = 0;
  for (int l = 0; l <= L; ++l) {
    p->nv_n[l] = (int)P[l].size();
    p->nv_tab[l] = p->nv_host.size();
    p->nv_host.insert(p->nv_host.end(), P[l].begin(), P[l].end());
    if (l == 0) continue;
    p->nv_nodes += p->nv_n[l];
    const std::vector<int> &below = P[l - 1];
    auto index_of = [&](int o) { return (int32_t)(std::lower_bound(below.begin(), below.end(), o) - below.begin()); };
    for (int k = 0; k < w; ++k)
      for (int o : P[l]) p->nv_host.push_back(index_of(o - (w - 1 - k) * dil[l - 1]));
  }
}

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
  const int w = d->filter_width == 0 ? 2 : d->filter_width;
  if (w < 2) return fail(FWG_EINVAL, "filter_width must be >= 2 (or 0 for 2), got %d", d->filter_width);
  if (w > 16) return fail(FWG_EUNSUPPORTED, "filter_width > 16");

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
  p->w = w;

  // shapes the K-blocked products support
  const int kb = valu_kb_elems(p->dtype);
  bool ok = p->C % kb == 0 && kblock_ok(w * p->C, p->Co, kb) &&
            kblock_ok(p->kind == FWG_GATED ? p->H : p->C, p->Q, kb);
  if (p->kind == FWG_GATED)
    ok = ok && kblock_ok(p->C, p->C, kb) && kblock_ok(p->C, p->S, kb) && kblock_ok(p->S, p->H, kb);
  const bool valu_ok = ok;

  // one layer's block for the general step kernels: conv | res | skip weights, then the biases
  {
    const bool g = p->kind == FWG_GATED;
    size_t b = (size_t)w * p->C * p->Co * p->es;
    if (g) b += ((size_t)p->C * p->C + (size_t)p->S * p->C) * p->es;
    b += sizeof(float) * ((size_t)p->Co + (g ? (size_t)p->C + p->S : 0));
    p->valu_block = (b + 15) & ~(size_t)15;
  }
  // rows per block and weight staging.  Staging moves a layer's weight loads off its critical path
  // but costs the copy issue; it pays from two streams per block (measured: at one stream the
  // layer is too short to hide the copy).  Take the most rows per block (at most 8, fewer for
  // tiny batches) at which two layers' blocks fit in LDS, else the most rows that fit without
  // staging.  The popped states of a layer are held in registers between layers (at most
  // kValuPrefPops per thread).
  int rmax = 8;
  while (rmax > 1 && rmax > p->bmax) rmax >>= 1;
  const char *vs = getenv("FWG_VALU_STAGE");  // "0": never stage (the variant that reads weights from L2)
  const bool can_stage = p->valu_block <= (size_t)kValuStagePieces * 16 * kThreads && !(vs && strcmp(vs, "0") == 0);
  const int wf = (int)(p->valu_block / 4);
  int rpw = 0;
  bool stage = false;
  p->lds_bytes = 0;
  for (int pass = 0; pass < 2 && rpw == 0 && valu_ok; ++pass) {
    const bool st = pass == 0;
    if (st && !can_stage) continue;
    for (int r = rmax; r >= (st ? 2 : 1); r >>= 1) {
      if (r * (w - 1) * p->C > kValuPrefPops * kThreads) continue;
      const ValuLds lay = valu_lds_layout(p->kind, p->C, p->S, p->H, p->Q, p->L, r, w, st ? wf : 0);
      if ((size_t)lay.total_floats * 4 <= 160 * 1024) {
        rpw = r;
        stage = st;
        p->lds_bytes = (size_t)lay.total_floats * 4;
        break;
      }
    }
  }
  p->rpw = rpw > 0 ? rpw : 1;
  p->valu_wbytes = stage ? (int)p->valu_block : 0;

  // kernel family: the MFMA kernel covers gated bf16 stacks with R=64, S=H=512, filter width 2 or 3
  p->regime = REGIME_VALU;
  const char *force = getenv("FWG_REGIME");
  const bool mfma_shape = (w == 2 || w == 3) && p->kind == FWG_GATED && p->dtype == FWG_BF16 && p->C == kMfR &&
                          p->S == kMfS && p->H == kMfH && p->Q == 256 && p->L <= kMfMaxLayers &&
                          mfma_lds_bytes(p->L, w) <= 160 * 1024;
  // the split family takes the MFMA family's shape at width 2 when L suits its unrolled layer loop
  // (FWG_REGIME=mfma keeps the single-block kernel); fwg_create falls back to it when the split
  // launch's blocks cannot all be resident at once
  const bool split_shape = mfma_shape && w == 2 && split_layers_ok(p->L);
  if (mfma_shape && !(force && strcmp(force, "valu") == 0))
    p->regime = split_shape && !(force && strcmp(force, "mfma") == 0) ? REGIME_SPLIT : REGIME_MFMA;
  // small float32 ReLU stacks: one block per stream with the layer chain on one wavefront (chain
  // family; FWG_REGIME=wave keeps the wave-per-stream kernel)
  const bool forced_other = force && (strcmp(force, "valu") == 0 || strcmp(force, "wave") == 0);
  if (p->regime == REGIME_VALU && !forced_other &&
      chain_layout(p->kind, p->dtype, p->C, p->Q, p->L, w, d->dilations, &p->chain, &p->chain_lds))
    p->regime = REGIME_CHAIN;
  // float32 gated stacks with R = 32, S = H = 256, width 2 or 3: one block per stream, the layer chain on one
  // wavefront, the recurrent halves, the skip sum and the head on the block's other waves
  if (p->regime == REGIME_VALU && !forced_other &&
      chain_gated_ok(p->kind, p->dtype, p->C, p->S, p->H, p->Q, p->L, w, &p->cg_bytes, &p->cg_lds)) {
    // two blocks of one XCD per stream (chain block and helper) unless FWG_REGIME=chain1 keeps one;
    // fwg_create falls back to one block when the pairs cannot all be resident at once
    p->cp_lds = chain_pair_lds_bytes(p->L);
    const bool one = force && strcmp(force, "chain1") == 0;
    p->regime = !one && p->cp_lds <= 160 * 1024 ? REGIME_CHAIN_PAIR : REGIME_CHAIN_GATED;
  }
  // float32 ReLU stacks of 512 channels: each layer spread over a group of 32 blocks per XCD
  if (p->regime == REGIME_VALU && !forced_other &&
      wide_layout(p->kind, p->dtype, p->C, p->Q, p->L, w, p->bmax, d->dilations, &p->wide, &p->wide_lds,
                  &p->wide_comm))
    p->regime = REGIME_WIDE;
  // small models whose weights all fit in LDS: one wavefront per stream
  if (p->regime == REGIME_VALU && !(force && strcmp(force, "valu") == 0) && wave_layout(*p, &p->wave))
    p->regime = REGIME_WAVE;
  if (p->regime == REGIME_VALU && !valu_ok)
    return fail(FWG_EUNSUPPORTED,
                "unsupported shape: every product needs K a multiple of %d, and an output width that "
                "divides 256 (with K/%d divisible by 256/N) or is at least 256",
                kb, kb);
  if (p->regime == REGIME_VALU && rpw == 0)
    return fail(FWG_EUNSUPPORTED, "model too wide for one block's LDS and registers");
  const bool mf_family = p->regime == REGIME_MFMA || p->regime == REGIME_SPLIT;
  p->brows = mf_family ? (p->bmax + kMfRows - 1) / kMfRows * kMfRows : p->bmax;

  // workspace layout
  size_t off = 0;
  auto take = [&](size_t bytes) { size_t at = off; off = align_up(off + bytes); return at; };
  p->off_layers = take(sizeof(LayerDev) * p->L);
  p->off_frags = p->off_embT = p->off_bias = p->off_ptrtab = p->off_comm = p->off_sticky = 0;
  if (mf_family) {
    // either family's fragment streams fit (create may fall back from the split family)
    p->off_frags = take(std::max(mfma_all_frag_bytes(p->L, w), split_shape ? split_frag_bytes(p->L) : size_t(0)));
    p->off_embT = take((size_t)p->Q * p->C * 2);
    p->off_bias = take(sizeof(float) * mfma_bias_floats(p->L));
    p->off_ptrtab = take(sizeof(void *) * 3 * p->L);
    if (split_shape) {
      p->off_comm = take(split_comm_bytes(p->L, p->brows / kMfRows));
      p->off_sticky = take(sizeof(uint32_t));
    }
  }
  p->off_wl = p->off_wo = p->off_wembT = p->off_wembb = p->off_wconvb = p->off_woutb = 0;
  if (p->regime == REGIME_WIDE) {
    p->off_wl = take(p->wide.wl_bytes);
    p->off_wo = take(p->wide.wo_bytes);
    p->off_wembT = take(sizeof(float) * (size_t)p->Q * p->C);
    p->off_wembb = take(sizeof(float) * p->C);
    p->off_wconvb = take(sizeof(float) * (size_t)p->L * p->C);
    p->off_woutb = take(sizeof(float) * p->Q);
    p->off_comm = take(p->wide_comm);
    p->off_sticky = take(sizeof(uint32_t));
  }
  p->off_embed = take((size_t)p->Q * p->C * p->es);
  p->off_embed_b = take(sizeof(float) * p->C);
  p->off_conv.resize(p->L); p->off_conv_b.resize(p->L);
  p->off_res.assign(p->L, 0); p->off_res_b.assign(p->L, 0); p->off_skip.assign(p->L, 0); p->off_skip_b.assign(p->L, 0);
  for (int l = 0; l < p->L; ++l) {
    // the layer's block (layout read by the general step kernels)
    const size_t base = take(p->valu_block);
    const size_t wconv = (size_t)p->Co * w * p->C * p->es;
    p->off_conv[l] = base;
    if (p->kind == FWG_GATED) {
      p->off_res[l] = base + wconv;
      p->off_skip[l] = p->off_res[l] + (size_t)p->C * p->C * p->es;
      p->off_conv_b[l] = p->off_skip[l] + (size_t)p->S * p->C * p->es;
      p->off_res_b[l] = p->off_conv_b[l] + sizeof(float) * p->Co;
      p->off_skip_b[l] = p->off_res_b[l] + sizeof(float) * p->C;
    } else {
      p->off_conv_b[l] = base + wconv;
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
    acc += (long long)(w - 1) * d->dilations[l] * p->brows * p->C;
  }
  p->queue_elems = acc;
  // the split family addresses a queue region with 32-bit byte offsets
  if (p->regime == REGIME_SPLIT && (unsigned long long)acc * p->es >= (1ull << 31)) p->regime = REGIME_MFMA;
  (void)dsum;
  p->off_ring_gen = take((size_t)acc * p->es);
  p->off_ring_tf = take((size_t)acc * p->es);
  p->off_last = take(sizeof(int32_t) * p->bmax);
  p->off_wave = p->regime == REGIME_WAVE ? take(sizeof(float) * (size_t)p->wave.image_floats) : 0;
  p->off_chain = p->regime == REGIME_CHAIN ? take(sizeof(float) * (size_t)p->chain.image_floats) : 0;
  const bool cg_family = p->regime == REGIME_CHAIN_GATED || p->regime == REGIME_CHAIN_PAIR;
  p->off_cg = cg_family ? take(p->cg_bytes) : 0;
  if (p->regime == REGIME_CHAIN_PAIR) {
    p->off_comm = take(chain_pair_comm_bytes(p->L, p->bmax));
    p->off_sticky = take(sizeof(uint32_t));
  }

  // time-parallel path: every product's K must fill whole 128-byte k-tiles, and the gate's column
  // pairs come in groups of 16 channels
  const int kt = kParKTileBytes / p->es;
  p->par_ok = p->C % kt == 0 && (p->kind != FWG_GATED ||
                                 (p->C % 16 == 0 && ((long long)p->L * p->C) % kt == 0 && p->S % kt == 0 &&
                                  p->H % kt == 0));
  p->par_tc = 0;
  if (p->par_ok) {
    const bool gated = p->kind == FWG_GATED;
    const bool fp32_stream = p->kind != FWG_RELU;                  // residual stream kept in float32
    const bool opnd_copy = p->kind == FWG_RELU || p->dtype == FWG_BF16;  // separate operand rows
    size_t row_bytes = 0;
    if (fp32_stream) row_bytes += 2 * (size_t)p->C * 4;
    if (opnd_copy) row_bytes += 2 * (size_t)p->C * p->es;
    if (gated) row_bytes += ((size_t)p->L * p->C + p->S + p->H) * p->es;
    // chunk rows: about 64K rows, at most 512 MB of chunk buffers, at least one step
    long long rows = 65536;
    const char *pr = getenv("FWG_PAR_ROWS");
    if (pr && atoll(pr) > 0) rows = atoll(pr);
    const long long cap = (512ll << 20) / (long long)row_bytes;
    if (rows > cap) rows = cap;
    p->par_tc = (int)(rows / p->brows > 0 ? rows / p->brows : 1);
    const size_t R = (size_t)p->par_tc * p->brows;
    p->off_pconv.assign(p->L, 0); p->off_pconv_b.assign(p->L, 0); p->off_pres.assign(p->L, 0);
    for (int l = 0; l < p->L; ++l) {
      p->off_pconv[l] = take((size_t)p->Co * w * p->C * p->es);
      p->off_pconv_b[l] = take(sizeof(float) * p->Co);
      if (gated) p->off_pres[l] = take((size_t)p->C * p->C * p->es);
    }
    p->off_pskip = gated ? take((size_t)p->S * p->L * p->C * p->es) : 0;
    p->off_pskip_b = gated ? take(sizeof(float) * p->S) : 0;
    p->off_phead = gated ? take((size_t)p->H * p->S * p->es) : 0;
    p->off_pout = take((size_t)p->Q * Kout * p->es);
    for (int i = 0; i < 3; ++i) {
      p->off_px[i] = fp32_stream ? take(R * p->C * 4) : 0;
      p->off_pxb[i] = opnd_copy ? take(R * p->C * p->es) : p->off_px[i];
    }
    p->off_pz = gated ? take(R * p->L * p->C * p->es) : 0;
    p->off_psb = gated ? take(R * p->S * p->es) : 0;
    p->off_phb = gated ? take(R * p->H * p->es) : 0;
  }
  // naive generator: needs the time-parallel kernels and chunk buffers holding max_batch x (level-0 nodes)
  p->nv_ok = false;
  p->off_nv = p->off_hist = p->off_ztop = p->off_nlogits = 0;
  if (p->par_ok) {
    naive_tables(p, d->dilations);
    if ((long long)p->bmax * p->nv_n[0] <= (long long)p->par_tc * p->brows) {
      p->nv_ok = true;
      p->nv_hc = 1;
      while (p->nv_hc < (long long)(w - 1) * dsum + 1) p->nv_hc <<= 1;
      p->off_nv = take(sizeof(int32_t) * p->nv_host.size());
      p->off_hist = take(sizeof(int32_t) * (size_t)p->bmax * p->nv_hc);
      p->off_ztop = p->kind == FWG_GATED ? take((size_t)p->bmax * p->L * p->C * p->es) : 0;
      p->off_nlogits = take(sizeof(float) * (size_t)p->bmax * p->Q);
    }
  }
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
  long long nv_t;   // naive generator: its own time and batch binding (its state is the input history)
  int nv_bound_batch;
  void *static_scratch;  // split family: this device's static exchange-word array (fwg_generate_noalloc)
  // split family, the workspace's exchange words: the next launch's tag base (every tag written since
  // the region was last zeroed is at most this), and whether the region has been zeroed since create
  uint32_t sp_tag = 0;
  bool sp_comm_zeroed = false;
};

namespace {

int enqueue_reset(fwg_handle *h) {
  const Plan &p = h->plan;
  HIP_TRY(launch_fill_zero(h->ws + p.off_ring_gen, (size_t)p.queue_elems * p.es, h->stream));
  HIP_TRY(launch_fill_i32((int32_t *)(h->ws + p.off_last), p.seed_input, p.bmax, h->stream));
  if (p.regime == REGIME_SPLIT || p.regime == REGIME_WIDE || p.regime == REGIME_CHAIN_PAIR)
    HIP_TRY(launch_fill_zero(h->ws + p.off_sticky, sizeof(uint32_t), h->stream));
  if (p.nv_ok)  // every history entry the seed: the entry of time 0 is the first input
    HIP_TRY(launch_fill_i32((int32_t *)(h->ws + p.off_hist), p.seed_input, p.bmax * p.nv_hc, h->stream));
  h->t = 0;
  h->bound_batch = -1;
  h->nv_t = 0;
  h->nv_bound_batch = -1;
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
  a.valu_wbytes = p.valu_wbytes;
  if (p.regime == REGIME_MFMA || p.regime == REGIME_SPLIT) {
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
  a.w = p.w;
  return a;
}

// One naive generation step at time t for every stream: evaluate the distinct nodes of the
// output's dependency tree (Fig. 1) level by level from the input history, the head, and the
// sample, which is appended to the history.  Nothing but the inputs is kept between samples.
int naive_step(fwg_handle *h, int batch, long long t, int n_steps, int s, const float *uniforms, int32_t *samples) {
  const Plan &p = h->plan;
  hipStream_t st = h->stream;
  char *ws = h->ws;
  const int C = p.C, L = p.L, es = p.es;
  const bool gated = p.kind == FWG_GATED;
  const bool f32s = p.kind != FWG_RELU;
  const bool opnd_copy = p.kind == FWG_RELU || p.dtype == FWG_BF16;
  const int32_t *tab = (const int32_t *)(ws + p.off_nv);
  float *px[2] = {(float *)(ws + p.off_px[0]), (float *)(ws + p.off_px[1])};
  char *pxb[2] = {ws + p.off_pxb[0], ws + p.off_pxb[1]};
  ParEmbed e;
  memset(&e, 0, sizeof(e));
  e.M = batch * p.nv_n[0]; e.C = C; e.Tcur = p.nv_n[0];
  e.embed = ws + p.off_embed;
  e.embed_b = (const float *)(ws + p.off_embed_b);
  e.xout = f32s ? px[0] : nullptr;
  e.oout = pxb[0];
  e.toff = tab + p.nv_tab[0]; e.tnow = t;
  e.hist = (const int32_t *)(ws + p.off_hist); e.hmask = p.nv_hc - 1;
  HIP_TRY(launch_par_embed(e, p.dtype, st));
  int cur = 0;
  for (int l = 0; l < L; ++l) {
    const int nxt = cur ^ 1, n = p.nv_n[l + 1], nprev = p.nv_n[l];
    const int32_t *lt = tab + p.nv_tab[l + 1];
    ParGemm g;
    memset(&g, 0, sizeof(g));
    g.M = batch * n; g.N = p.Co; g.K = p.w * C; g.Tcur = n; g.C = C; g.dil = h->dil[l]; g.w = p.w;
    g.A = pxb[cur]; g.lda = C;
    g.toff = lt; g.tsrc = lt + n; g.nprev = nprev; g.tnow = t;
    if (p.kind == FWG_RELU_RESIDUAL) g.tsrc1 = lt + (size_t)p.w * n;  // x_in: the same-time node (tap w - 1)
    g.W = ws + p.off_pconv[l];
    g.bias = (const float *)(ws + p.off_pconv_b[l]);
    int em;
    if (gated) {
      em = PAR_E_GATE; g.oout = ws + p.off_pz; g.ldo = (long long)L * C; g.zoff = l * C; g.ztop = ws + p.off_ztop;
    } else if (p.kind == FWG_RELU) {
      em = PAR_E_RELU; g.oout = pxb[nxt]; g.ldo = C;
    } else {
      em = PAR_E_RELU_RES; g.xres = px[cur]; g.xout = px[nxt]; g.oout = opnd_copy ? pxb[nxt] : nullptr; g.ldo = C;
    }
    HIP_TRY(launch_par_gemm(g, p.dtype, PAR_A_TREE, em, st));
    if (gated && l + 1 < L) {
      ParGemm r;
      memset(&r, 0, sizeof(r));
      r.M = batch * n; r.N = C; r.K = C; r.Tcur = n;
      r.A = ws + p.off_pz + (size_t)l * C * es; r.lda = (long long)L * C;
      r.W = ws + p.off_pres[l];
      r.bias = (const float *)(ws + p.off_res_b[l]);
      r.xres = px[cur]; r.xout = px[nxt]; r.oout = opnd_copy ? pxb[nxt] : nullptr; r.ldo = C;
      r.tsrc1 = lt + (size_t)p.w * n; r.nprev = nprev;
      HIP_TRY(launch_par_gemm(r, p.dtype, PAR_A_PLAIN, PAR_E_RES_ADD, st));
    }
    cur = nxt;
  }
  float *lg = (float *)(ws + p.off_nlogits);
  ParGemm o;
  memset(&o, 0, sizeof(o));
  o.M = batch; o.N = p.Q; o.Tcur = 1; o.logits = lg; o.n_steps = 1; o.s0 = 0;
  o.W = ws + p.off_pout;
  o.bias = (const float *)(ws + p.off_out_b);
  if (gated) {
    ParGemm k;
    memset(&k, 0, sizeof(k));
    k.M = batch; k.N = p.S; k.K = L * C; k.Tcur = 1;
    k.A = ws + p.off_ztop; k.lda = (long long)L * C;
    k.W = ws + p.off_pskip;
    k.bias = (const float *)(ws + p.off_pskip_b);
    k.oout = ws + p.off_psb; k.ldo = p.S;
    HIP_TRY(launch_par_gemm(k, p.dtype, PAR_A_PLAIN, PAR_E_RELU, st));
    ParGemm hd;
    memset(&hd, 0, sizeof(hd));
    hd.M = batch; hd.N = p.H; hd.K = p.S; hd.Tcur = 1;
    hd.A = ws + p.off_psb; hd.lda = p.S;
    hd.W = ws + p.off_phead;
    hd.bias = (const float *)(ws + p.off_head_b);
    hd.oout = ws + p.off_phb; hd.ldo = p.H;
    HIP_TRY(launch_par_gemm(hd, p.dtype, PAR_A_PLAIN, PAR_E_RELU, st));
    o.A = ws + p.off_phb; o.lda = p.H; o.K = p.H;
  } else {
    o.A = pxb[cur]; o.lda = C; o.K = C;  // the last level holds the single node at offset 0
  }
  HIP_TRY(launch_par_gemm(o, p.dtype, PAR_A_PLAIN, PAR_E_LOGITS, st));
  HIP_TRY(launch_par_sample(lg, uniforms, samples, (int32_t *)(ws + p.off_hist), p.nv_hc - 1, t + 1, batch, n_steps,
                            s, st));
  return FWG_OK;
}

// One step-kernel launch of the handle's kernel family.  comm: where the split family's exchange
// words go (NULL: the workspace's region).
hipError_t launch_step(fwg_handle *h, const StepArgs &a, void *comm = nullptr) {
  const Plan &p = h->plan;
  switch (p.regime) {
    case REGIME_MFMA: return launch_mfma_step(a, h->stream);
    case REGIME_SPLIT: {
      StepArgs b = a;
      b.sp_nb = (a.batch + kMfRows - 1) / kMfRows;
      b.sp_comm = comm ? comm : h->ws + p.off_comm;
      b.sp_sticky = (uint32_t *)(h->ws + p.off_sticky);
      // Tags are never reused between two zero fills of the exchange words (a fill kernel, no memset
      // node).  The static array of fwg_generate_noalloc is shared by every handle on the device: it
      // is zeroed before every launch (this launch's groups), whose tags then start at 1.  The
      // workspace's region belongs to this handle: zeroed whole (every group the handle's largest
      // batch uses, since a later call may use more groups than this one) before its first launch
      // and when the tags would wrap; every launch takes the tags above the previous launch's
      // (handshake base + 1, step s base + 2 + s).
      const uint32_t need = (uint32_t)a.n_steps + 2u;
      if (comm || !h->sp_comm_zeroed || h->sp_tag > 0xFFFFFFFFu - need) {
        const size_t bytes = split_comm_bytes(p.L, comm ? b.sp_nb : p.brows / kMfRows);
        hipError_t e = launch_fill_zero(b.sp_comm, bytes, h->stream);
        if (e != hipSuccess) return e;
        if (!comm) {
          h->sp_comm_zeroed = true;
          h->sp_tag = 0;
        }
      }
      b.sp_tag0 = comm ? 0u : h->sp_tag;
      if (!comm) h->sp_tag += need - 1u;
      return launch_split_step(b, h->stream);
    }
    case REGIME_WIDE: {
      StepArgs b = a;
      b.sp_nb = (a.batch + kWideStreams - 1) / kWideStreams;
      b.sp_comm = comm ? comm : h->ws + p.off_comm;
      b.sp_sticky = (uint32_t *)(h->ws + p.off_sticky);
      // tags restart at 1 every launch: clear the exchange words first (a fill kernel, no memset node)
      hipError_t e = launch_fill_zero(b.sp_comm, p.wide_comm, h->stream);
      if (e != hipSuccess) return e;
      WideArgs g = p.wide;
      g.wl = h->ws + p.off_wl;
      g.wo = h->ws + p.off_wo;
      g.embT = (float *)(h->ws + p.off_wembT);
      g.embb = (float *)(h->ws + p.off_wembb);
      g.convb = (float *)(h->ws + p.off_wconvb);
      g.outb = (float *)(h->ws + p.off_woutb);
      return launch_wide_step(b, g, p.wide_lds, h->stream);
    }
    case REGIME_CHAIN: {
      ChainArgs g = p.chain;
      g.image = (const float *)(h->ws + p.off_chain);
      return launch_chain_step(a, g, p.chain_lds, h->stream);
    }
    case REGIME_CHAIN_GATED:
      return launch_chain_gated_step(a, chain_gated_arrays(h->ws + p.off_cg, p.L, p.w), p.cg_lds, h->stream);
    case REGIME_CHAIN_PAIR: {
      StepArgs b = a;
      b.sp_comm = comm ? comm : h->ws + p.off_comm;
      b.sp_sticky = (uint32_t *)(h->ws + p.off_sticky);
      // tags restart at 1 every launch: clear the exchange words first (a fill kernel, no memset node)
      hipError_t e = launch_fill_zero(b.sp_comm, chain_pair_comm_bytes(p.L, a.batch), h->stream);
      if (e != hipSuccess) return e;
      return launch_chain_pair_step(b, chain_gated_arrays(h->ws + p.off_cg, p.L, p.w), p.cp_lds, h->stream);
    }
    case REGIME_WAVE: {
      WaveArgs g = p.wave;
      g.image = (const float *)(h->ws + p.off_wave);
      return launch_wave_step(a, g, h->stream);
    }
    default: return launch_valu_step(a, p.rpw, p.lds_bytes, h->stream);
  }
}

// Time-parallel evaluation of a forced sequence, chunk by chunk (MODE_TEACHER or MODE_ONLINE):
// every layer is a GEMM over the chunk's rows whose popped operand comes from the chunk or from
// the layer's queue in `ring`; a layer's queue is refreshed once its product has read it (by the
// next layer's fused kernel when there is one, which is why the row buffers rotate over three).
// logits may be NULL (online mode only): then the skip sum and the head are skipped.
int par_forward(fwg_handle *h, int mode, int batch, int n, const int32_t *inputs, float *logits, char *ring,
                long long tbase) {
  const Plan &p = h->plan;
  hipStream_t s = h->stream;
  char *ws = h->ws;
  const int C = p.C, L = p.L, es = p.es;
  const bool gated = p.kind == FWG_GATED;
  const bool f32s = p.kind != FWG_RELU;
  const bool opnd_copy = p.kind == FWG_RELU || p.dtype == FWG_BF16;
  float *px[3] = {(float *)(ws + p.off_px[0]), (float *)(ws + p.off_px[1]), (float *)(ws + p.off_px[2])};
  char *pxb[3] = {ws + p.off_pxb[0], ws + p.off_pxb[1], ws + p.off_pxb[2]};
  const bool fused = gated && par_gated_layer_ok(C, p.dtype);
  for (long long s0 = 0; s0 < n; s0 += p.par_tc) {
    const int Tcur = (int)(n - s0 < p.par_tc ? n - s0 : p.par_tc);
    const int M = batch * Tcur;
    const long long t0 = tbase + s0;
    ParEmbed e;
    memset(&e, 0, sizeof(e));
    e.M = M; e.C = C; e.Tcur = Tcur; e.mode = mode; e.s0 = s0; e.n_steps = n;
    e.inputs = inputs;
    e.last = (const int32_t *)(ws + p.off_last);
    e.embed = ws + p.off_embed;
    e.embed_b = (const float *)(ws + p.off_embed_b);
    e.xout = f32s ? px[0] : nullptr;
    e.oout = pxb[0];
    HIP_TRY(launch_par_embed(e, p.dtype, s));
    int cur = 0, prev = 0;
    auto refresh = [&](int l, const char *src) {
      ParRing q;
      memset(&q, 0, sizeof(q));
      q.ring = ring + (size_t)p.ring_off[l] * es; q.src = src;
      q.t0 = t0; q.Tcur = Tcur; q.depth = (p.w - 1) * h->dil[l]; q.brows = p.brows; q.batch = batch;
      q.row_bytes = C * es;
      return launch_par_ring(q, s);
    };
    for (int l = 0; l < L; ++l) {
      const int nxt = (cur + 1) % 3;
      ParGemm g;
      memset(&g, 0, sizeof(g));
      g.M = M; g.N = p.Co; g.K = p.w * C;
      g.A = pxb[cur]; g.lda = C;
      g.ring = ring + (size_t)p.ring_off[l] * es;
      g.t0 = t0; g.dil = h->dil[l]; g.brows = p.brows; g.Tcur = Tcur; g.C = C;
      g.w = p.w; g.depth = (p.w - 1) * h->dil[l];
      g.W = ws + p.off_pconv[l];
      g.bias = (const float *)(ws + p.off_pconv_b[l]);
      int em = PAR_E_GATE;
      if (fused) {
        // dilated product, gate, z rows and residual 1x1 in one kernel, with the previous layer's
        // queue refresh
        if (l > 0) {
          g.qring = ring + (size_t)p.ring_off[l - 1] * es; g.qsrc = pxb[prev]; g.qdepth = (p.w - 1) * h->dil[l - 1];
        }
        g.zout = ws + p.off_pz; g.ldz = (long long)L * C; g.zoff = l * C;
        g.W2 = ws + p.off_pres[l];
        g.bias2 = (const float *)(ws + p.off_res_b[l]);
        g.xres = px[cur]; g.xout = px[nxt]; g.oout = opnd_copy ? pxb[nxt] : nullptr; g.ldo = C;
        HIP_TRY(launch_par_gated_layer(g, p.dtype, s));
      } else if (gated) {
        em = PAR_E_GATE; g.oout = ws + p.off_pz; g.ldo = (long long)L * C; g.zoff = l * C;
      } else if (p.kind == FWG_RELU) {
        em = PAR_E_RELU; g.oout = pxb[nxt]; g.ldo = C;
      } else {
        em = PAR_E_RELU_RES; g.xres = px[cur]; g.xout = px[nxt]; g.oout = opnd_copy ? pxb[nxt] : nullptr; g.ldo = C;
      }
      if (!fused) HIP_TRY(launch_par_gemm(g, p.dtype, PAR_A_CONV, em, s));
      if (gated && !fused && l + 1 < L) {  // the last layer's residual output feeds nothing
        ParGemm r;
        memset(&r, 0, sizeof(r));
        r.M = M; r.N = C; r.K = C; r.Tcur = Tcur;
        r.A = ws + p.off_pz + (size_t)l * C * es; r.lda = (long long)L * C;
        r.W = ws + p.off_pres[l];
        r.bias = (const float *)(ws + p.off_res_b[l]);
        r.xres = px[cur]; r.xout = px[nxt]; r.oout = opnd_copy ? pxb[nxt] : nullptr; r.ldo = C;
        HIP_TRY(launch_par_gemm(r, p.dtype, PAR_A_PLAIN, PAR_E_RES_ADD, s));
      }
      if (!fused || l + 1 == L) HIP_TRY(refresh(l, pxb[cur]));
      prev = cur;
      cur = nxt;
    }
    if (!logits) continue;
    ParGemm o;
    memset(&o, 0, sizeof(o));
    o.M = M; o.N = p.Q; o.Tcur = Tcur; o.logits = logits; o.n_steps = n; o.s0 = s0;
    o.W = ws + p.off_pout;
    o.bias = (const float *)(ws + p.off_out_b);
    if (gated) {
      ParGemm k;
      memset(&k, 0, sizeof(k));
      k.M = M; k.N = p.S; k.K = L * C; k.Tcur = Tcur;
      k.A = ws + p.off_pz; k.lda = (long long)L * C;
      k.W = ws + p.off_pskip;
      k.bias = (const float *)(ws + p.off_pskip_b);
      k.oout = ws + p.off_psb; k.ldo = p.S;
      HIP_TRY(launch_par_gemm(k, p.dtype, PAR_A_PLAIN, PAR_E_RELU, s));
      ParGemm hd;
      memset(&hd, 0, sizeof(hd));
      hd.M = M; hd.N = p.H; hd.K = p.S; hd.Tcur = Tcur;
      hd.A = ws + p.off_psb; hd.lda = p.S;
      hd.W = ws + p.off_phead;
      hd.bias = (const float *)(ws + p.off_head_b);
      hd.oout = ws + p.off_phb; hd.ldo = p.H;
      HIP_TRY(launch_par_gemm(hd, p.dtype, PAR_A_PLAIN, PAR_E_RELU, s));
      o.A = ws + p.off_phb; o.lda = p.H; o.K = p.H;
    } else {
      o.A = pxb[cur]; o.lda = C; o.K = C;
    }
    HIP_TRY(launch_par_gemm(o, p.dtype, PAR_A_PLAIN, PAR_E_LOGITS, s));
  }
  if (mode == MODE_ONLINE) HIP_TRY(launch_par_set_last(inputs, (int32_t *)(ws + p.off_last), batch, n, s));
  return FWG_OK;
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
    TRY_OR_FREE(launch_repack(w->conv[l], ws + p.off_conv[l], REPACK_CONV, dt, p.w * C, p.Co, C, s));
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
    ld.depth = (p.w - 1) * h->dil[l];
  }
  if (p.kind == FWG_GATED) {
    TRY_OR_FREE(launch_repack(w->head, ws + p.off_head, REPACK_LINEAR, dt, p.S, p.H, C, s));
    TRY_OR_FREE(launch_copy_bias(w->head_b, (float *)(ws + p.off_head_b), p.H, s));
  }
  const int Kout = p.kind == FWG_GATED ? p.H : C;
  TRY_OR_FREE(launch_repack(w->out, ws + p.off_out, REPACK_LINEAR, dt, Kout, p.Q, C, s));
  TRY_OR_FREE(launch_copy_bias(w->out_b, (float *)(ws + p.off_out_b), p.Q, s));
  TRY_OR_FREE(hipMemcpyAsync(ws + p.off_layers, table.data(), sizeof(LayerDev) * p.L, hipMemcpyHostToDevice, s));
  if (p.regime == REGIME_CHAIN) {
    TRY_OR_FREE(launch_chain_image(w->embed, w->embed_b, w->conv, w->conv_b, w->out, w->out_b, p.L, p.chain,
                                   (float *)(ws + p.off_chain), s));
    TRY_OR_FREE(set_chain_lds_limit(p.chain_lds));
  }
  if (p.regime == REGIME_CHAIN_PAIR) {
    int coresident = 0;
    TRY_OR_FREE(chain_pair_setup(p.cp_lds, p.bmax, &coresident));
    if (!coresident) h->plan.regime = REGIME_CHAIN_GATED;  // same workspace; the one-block layout below
    // set-up of fwg_generate_noalloc: this device's static exchange-word array, looked up once
    else TRY_OR_FREE(split_static_scratch(&h->static_scratch));
  }
  if (h->plan.regime == REGIME_CHAIN_GATED || h->plan.regime == REGIME_CHAIN_PAIR) {
    TRY_OR_FREE(launch_chain_gated_pack(w->embed, w->embed_b, w->conv, w->conv_b, w->res, w->res_b, w->skip,
                                        w->skip_b, w->head, w->head_b, w->out, w->out_b, p.L, p.w,
                                        h->plan.regime == REGIME_CHAIN_PAIR, chain_gated_arrays(ws + p.off_cg, p.L, p.w),
                                        s));
    TRY_OR_FREE(set_chain_gated_lds_limit(p.cg_lds));
  }
  if (p.regime == REGIME_WAVE) {
    const WaveArgs &g = p.wave;
    float *img = (float *)(ws + p.off_wave);
    const int Ktop = p.kind == FWG_GATED ? p.H : C;
    TRY_OR_FREE(launch_fill_zero(img, sizeof(float) * (size_t)g.image_floats, s));
    TRY_OR_FREE(launch_wave_image(w->embed, img + g.o_emb, dt, C, p.Q, C, 0, s));
    TRY_OR_FREE(launch_wave_vec(w->embed_b, img + g.o_embb, C, s));
    for (int l = 0; l < p.L; ++l) {
      float *blk = img + g.o_layer + (size_t)l * g.layer_floats;
      TRY_OR_FREE(launch_wave_image(w->conv[l], blk, dt, p.Co, p.w * C, C, 1, s));
      TRY_OR_FREE(launch_wave_vec(w->conv_b ? w->conv_b[l] : nullptr, blk + g.o_convb, p.Co, s));
      if (p.kind == FWG_GATED) {
        TRY_OR_FREE(launch_wave_image(w->res[l], blk + g.o_res, dt, C, C, C, 0, s));
        TRY_OR_FREE(launch_wave_vec(w->res_b ? w->res_b[l] : nullptr, blk + g.o_resb, C, s));
        TRY_OR_FREE(launch_wave_image(w->skip[l], blk + g.o_skip, dt, p.S, C, C, 0, s));
        TRY_OR_FREE(launch_wave_vec(w->skip_b ? w->skip_b[l] : nullptr, blk + g.o_skipb, p.S, s));
      }
    }
    if (p.kind == FWG_GATED) {
      TRY_OR_FREE(launch_wave_image(w->head, img + g.o_head, dt, p.H, p.S, C, 0, s));
      TRY_OR_FREE(launch_wave_vec(w->head_b, img + g.o_headb, p.H, s));
    }
    TRY_OR_FREE(launch_wave_image(w->out, img + g.o_out, dt, p.Q, Ktop, C, 0, s));
    TRY_OR_FREE(launch_wave_vec(w->out_b, img + g.o_outb, p.Q, s));
    TRY_OR_FREE(set_wave_lds_limit(sizeof(float) * ((size_t)g.image_floats + 4 * (size_t)g.scr_floats)));
  }
  if (p.nv_ok)
    TRY_OR_FREE(hipMemcpyAsync(ws + p.off_nv, p.nv_host.data(), sizeof(int32_t) * p.nv_host.size(),
                               hipMemcpyHostToDevice, s));
  if (p.par_ok) {
    const int il = p.kind == FWG_GATED;  // gated conv rows interleave tanh and sigmoid channel groups
    for (int l = 0; l < p.L; ++l) {
      TRY_OR_FREE(launch_par_repack(w->conv[l], ws + p.off_pconv[l], PAR_REPACK_CONV, dt, p.Co, p.w * C, C, il, 0, 0,
                                    s));
      TRY_OR_FREE(launch_par_bias(w->conv_b ? w->conv_b[l] : nullptr, (float *)(ws + p.off_pconv_b[l]), p.Co, il, 0, s));
      if (p.kind == FWG_GATED) {
        TRY_OR_FREE(launch_par_repack(w->res[l], ws + p.off_pres[l], PAR_REPACK_COPY, dt, C, C, C, 0, C, 0, s));
        TRY_OR_FREE(launch_par_repack(w->skip[l], ws + p.off_pskip, PAR_REPACK_COPY, dt, p.S, C, C, 0,
                                      (long long)p.L * C, (long long)l * C, s));
        TRY_OR_FREE(launch_par_bias((const float *)(ws + p.off_skip_b[l]), (float *)(ws + p.off_pskip_b), p.S, 0,
                                    l > 0, s));
      }
    }
    if (p.kind == FWG_GATED)
      TRY_OR_FREE(launch_par_repack(w->head, ws + p.off_phead, PAR_REPACK_COPY, dt, p.H, p.S, C, 0, p.S, 0, s));
    TRY_OR_FREE(launch_par_repack(w->out, ws + p.off_pout, PAR_REPACK_COPY, dt, p.Q, Kout, C, 0, Kout, 0, s));
  }
  std::vector<const void *> ptrs;
  if (p.regime == REGIME_WIDE) {
    int coresident = 0;
    TRY_OR_FREE(wide_setup(p.wide_lds, &coresident));
    if (!coresident) {
      h->plan.regime = REGIME_VALU;  // the general kernels' weights are in the workspace as well
    } else {
      WideArgs g = p.wide;
      g.wl = ws + p.off_wl;
      g.wo = ws + p.off_wo;
      g.embT = (float *)(ws + p.off_wembT);
      g.embb = (float *)(ws + p.off_wembb);
      g.convb = (float *)(ws + p.off_wconvb);
      g.outb = (float *)(ws + p.off_woutb);
      TRY_OR_FREE(launch_wide_pack(w->embed, w->embed_b, w->conv, w->conv_b, w->out, w->out_b, p.L, g, s));
      // set-up of fwg_generate_noalloc: this device's static exchange-word array, looked up once
      TRY_OR_FREE(split_static_scratch(&h->static_scratch));
    }
  }
  if (p.regime == REGIME_SPLIT) {
    int coresident = 0;
    TRY_OR_FREE(split_setup(p.L, p.brows / kMfRows, &coresident));
    if (!coresident) h->plan.regime = REGIME_MFMA;  // same workspace layout
  }
  if (h->plan.regime == REGIME_SPLIT) {
    // set-up of fwg_generate_noalloc: this device's static exchange-word array, looked up once
    TRY_OR_FREE(split_static_scratch(&h->static_scratch));
    // test hook: the workspace's exchange words zeroed now and the tag base started at the given
    // value (e.g. just below the 32-bit wrap, so that later launches cross it)
    if (const char *tb = getenv("FWG_SPLIT_TAG_BASE")) {
      TRY_OR_FREE(launch_fill_zero(ws + p.off_comm, split_comm_bytes(p.L, p.brows / kMfRows), s));
      h->sp_comm_zeroed = true;
      h->sp_tag = (uint32_t)strtoul(tb, nullptr, 0);
    }
    char *frags = ws + p.off_frags;
    for (int l = 0; l < p.L; ++l)
      TRY_OR_FREE(launch_split_repack_layer(w->conv[l], w->res[l], w->skip[l], l, p.L, frags, s));
    TRY_OR_FREE(launch_split_repack_head(w->head, w->out, p.L, frags, s));
  } else if (h->plan.regime == REGIME_MFMA) {
    char *frags = ws + p.off_frags;
    // layers first: a layer also writes fragments into the previous stage and the last head stage
    for (int l = 0; l < p.L; ++l)
      TRY_OR_FREE(launch_mfma_repack_layer(w->conv[l], w->res[l], w->skip[l], l, p.L, p.w, frags, s));
    TRY_OR_FREE(launch_mfma_repack_head(w->head, w->out, p.L, frags, s));
  }
  if (h->plan.regime == REGIME_MFMA || h->plan.regime == REGIME_SPLIT) {
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
    TRY_OR_FREE(set_mfma_lds_limit(mfma_lds_bytes(p.L, p.w)));
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

namespace {
int generate_impl(fwg_handle *h, int32_t batch, int32_t n_steps, const float *uniforms, int32_t *samples,
                  bool noalloc) {
  if (!h) return fail(FWG_EINVAL, "handle is NULL");
  const Plan &p = h->plan;
  if (batch < 1 || batch > p.bmax) return fail(FWG_EINVAL, "batch %d outside [1, %d]", batch, p.bmax);
  if (n_steps < 0) return fail(FWG_EINVAL, "n_steps < 0");
  if (h->bound_batch >= 0 && h->bound_batch != batch)
    return fail(FWG_ESTATE, "batch %d differs from %d used since the last reset", batch, h->bound_batch);
  void *comm = nullptr;
  if (noalloc && (p.regime == REGIME_SPLIT || p.regime == REGIME_WIDE || p.regime == REGIME_CHAIN_PAIR)) {
    const size_t need = p.regime == REGIME_SPLIT ? split_comm_bytes(p.L, (batch + kMfRows - 1) / kMfRows)
                        : p.regime == REGIME_WIDE ? p.wide_comm
                                                  : chain_pair_comm_bytes(p.L, batch);
    if (need > kStaticScratchBytes)
      return fail(FWG_ENOSPACE, "the exchange words of %d streams x %d layers need %zu bytes; the static scratch "
                  "array holds %zu", batch, p.L, need, kStaticScratchBytes);
    if (!h->static_scratch) return fail(FWG_ESTATE, "no static scratch address was set up for this handle");
    comm = h->static_scratch;
  }
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
  HIP_TRY(launch_step(h, a, comm));
  h->bound_batch = batch;
  h->t += n_steps;
  return FWG_OK;
}
}  // namespace

int fwg_generate(fwg_handle *h, int32_t batch, int32_t n_steps, const float *uniforms, int32_t *samples) {
  return generate_impl(h, batch, n_steps, uniforms, samples, false);
}

int fwg_generate_noalloc(fwg_handle *h, int32_t batch, int32_t n_steps, const float *uniforms, int32_t *samples) {
  return generate_impl(h, batch, n_steps, uniforms, samples, true);
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
  HIP_TRY(launch_step(h, a));
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
  if (!inputs) return fail(FWG_EINVAL, "inputs are required");
  StepArgs a = base_args(h);
  a.ring = h->ws + p.off_ring_gen;
  a.inputs = inputs;
  a.logits = logits;
  a.t0 = h->t;
  a.n_steps = n_steps;
  a.batch = batch;
  a.mode = MODE_ONLINE;
  HIP_TRY(launch_step(h, a));
  h->bound_batch = batch;
  h->t += n_steps;
  return FWG_OK;
}

int fwg_teacher_forced_parallel(fwg_handle *h, int32_t batch, int32_t seq_len, const int32_t *inputs, float *logits) {
  if (!h) return fail(FWG_EINVAL, "handle is NULL");
  const Plan &p = h->plan;
  // products narrower than one 128-byte k-tile: the step kernels evaluate the sequence instead
  if (!p.par_ok) return fwg_teacher_forced(h, batch, seq_len, inputs, logits);
  if (batch < 1 || batch > p.bmax) return fail(FWG_EINVAL, "batch %d outside [1, %d]", batch, p.bmax);
  if (seq_len < 0) return fail(FWG_EINVAL, "seq_len < 0");
  if (seq_len == 0) return FWG_OK;
  if (!inputs || !logits) return fail(FWG_EINVAL, "inputs and logits are required");
  HIP_TRY(launch_fill_zero(h->ws + p.off_ring_tf, (size_t)p.queue_elems * p.es, h->stream));
  return par_forward(h, MODE_TEACHER, batch, seq_len, inputs, logits, h->ws + p.off_ring_tf, 0);
}

int fwg_prime(fwg_handle *h, int32_t batch, int32_t n_steps, const int32_t *inputs, float *logits) {
  if (!h) return fail(FWG_EINVAL, "handle is NULL");
  const Plan &p = h->plan;
  // products narrower than one 128-byte k-tile: the step kernels run the prefix instead
  if (!p.par_ok) return fwg_step_forced(h, batch, n_steps, inputs, logits);
  if (batch < 1 || batch > p.bmax) return fail(FWG_EINVAL, "batch %d outside [1, %d]", batch, p.bmax);
  if (n_steps < 0) return fail(FWG_EINVAL, "n_steps < 0");
  if (h->bound_batch >= 0 && h->bound_batch != batch)
    return fail(FWG_ESTATE, "batch %d differs from %d used since the last reset", batch, h->bound_batch);
  if (n_steps == 0) return FWG_OK;
  if (!inputs) return fail(FWG_EINVAL, "inputs are required");
  const int rc = par_forward(h, MODE_ONLINE, batch, n_steps, inputs, logits, h->ws + p.off_ring_gen, h->t);
  if (rc != FWG_OK) return rc;
  h->bound_batch = batch;
  h->t += n_steps;
  return FWG_OK;
}

int fwg_generate_naive(fwg_handle *h, int32_t batch, int32_t n_steps, const float *uniforms, int32_t *samples) {
  if (!h) return fail(FWG_EINVAL, "handle is NULL");
  const Plan &p = h->plan;
  if (!p.nv_ok)
    return fail(FWG_EUNSUPPORTED, "no naive generator for this model: it needs the time-parallel kernels and "
                                  "max_batch x receptive field rows of chunk buffers");
  if (batch < 1 || batch > p.bmax) return fail(FWG_EINVAL, "batch %d outside [1, %d]", batch, p.bmax);
  if (n_steps < 0) return fail(FWG_EINVAL, "n_steps < 0");
  if (h->nv_bound_batch >= 0 && h->nv_bound_batch != batch)
    return fail(FWG_ESTATE, "batch %d differs from %d used since the last reset", batch, h->nv_bound_batch);
  if (n_steps == 0) return FWG_OK;
  if (!uniforms || !samples) return fail(FWG_EINVAL, "uniforms and samples are required");
  for (int s = 0; s < n_steps; ++s) {
    const int rc = naive_step(h, batch, h->nv_t + s, n_steps, s, uniforms, samples);
    if (rc != FWG_OK) return rc;
  }
  h->nv_bound_batch = batch;
  h->nv_t += n_steps;
  return FWG_OK;
}

int fwg_naive_nodes(const fwg_desc *desc, int64_t *nodes) {
  if (!nodes) return fail(FWG_EINVAL, "nodes is NULL");
  Plan p;
  int rc = make_plan(desc, &p);
  if (rc != FWG_OK) return rc;
  if (p.nv_host.empty()) naive_tables(&p, desc->dilations);
  *nodes = p.nv_nodes;
  return FWG_OK;
}

int fwg_destroy(fwg_handle *h) {
  delete h;
  return FWG_OK;
}

int fwg_device_status(fwg_handle *h) {
  if (!h) return fail(FWG_EINVAL, "handle is NULL");
  HIP_TRY(hipStreamSynchronize(h->stream));
  if (h->plan.regime == REGIME_SPLIT || h->plan.regime == REGIME_WIDE || h->plan.regime == REGIME_CHAIN_PAIR) {
    uint32_t v = 0;
    HIP_TRY(hipMemcpy(&v, h->ws + h->plan.off_sticky, sizeof(v), hipMemcpyDeviceToHost));
    if (v)
      return fail(FWG_EDEVICE, "a wait between the cooperating blocks of a launch ran out (the blocks were not all "
                               "resident at once); that launch's outputs are invalid");
  }
  return FWG_OK;
}

const char *fwg_regime(const fwg_handle *h) {
  if (!h) return "";
  switch (h->plan.regime) {
    case REGIME_MFMA: return "mfma_bf16_r64_s512";
    case REGIME_SPLIT: return "mfma_split_bf16_r64_s512";
    case REGIME_WAVE: return "wave";
    case REGIME_CHAIN: return "chain_f32_c32";
    case REGIME_CHAIN_GATED: return "chain_gated_f32_r32";
    case REGIME_CHAIN_PAIR: return "chain_pair_f32_r32";
    case REGIME_WIDE: return "wide_f32_c512";
    default: return "valu";
  }
}

}  // extern "C"
