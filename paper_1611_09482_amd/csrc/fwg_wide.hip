// Wide step kernel for float32 ReLU stacks with C = 512 channels (filter width 2): every layer is
// spread over the 32 blocks of a group, one group per XCD and up to four streams per group.
//
// One sample is a chain of L dependent layers, each a 512 x 1024 product (Section 1: the edges of
// the graph are matrix products), then the output 1x1 and the sample fed back (Section 1).  A single
// block would stream 2 MB of weights per layer; here block j of a group owns output channels
// 16j..16j+15 of every layer:
//  - per layer it reads its 64 KB of weights (W_e and W_r rows, packed per thread, prefetched into
//    registers one layer ahead; the whole model stays resident in the 256 MB last-level cache) and
//    computes both products of its 16 channels for the group's 4 streams over the whole layer
//    input: thread (oc, kp) covers channel oc over K part kp (32 channels), and the 16 K parts meet
//    in LDS;
//  - the queue (Section 2.2) keeps, per block, the product W_r x of its own channels instead of the
//    state x: a = W_e x_t + (W_r x_{t-d}) + b pops the product pushed d steps earlier, so no block
//    reads another block's queue.  The states of its own channels are kept beside them and written
//    back to the workspace queues at the end of the launch (the generation state every kernel
//    family shares); at launch the products are recomputed from those states;
//  - the layer output goes to the group's other blocks as tagged words (fwg_xchg.h); with the whole
//    group on one XCD they stay in that XCD's L2;
//  - the output 1x1 is spread the same way (8 classes per block); block s < 4 of the group gathers
//    stream s's 256 logits, draws its sample and returns it to every block of the group as a word
//    (forced modes: writes nothing and returns a step-done mark; the logits are written by their
//    blocks).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fwg_internal.h"
#include "fwg_sample.h"
#include "fwg_wide.h"
#include "fwg_xchg.h"

namespace fwg {
namespace wd {

using namespace xg;

constexpr int C = kWideC, NBG = kWideBlocks, OC = C / NBG, SG = kWideStreams, NG = kWideGroups;
constexpr int NT = 256, KP = NT / OC, KW = C / KP, Q = 256, QB = Q / NBG;
constexpr int XP = KW + 4;    // floats per (stream, K part) row of the gathered layer input (padding spreads banks)
constexpr int KCH = 64;       // steps per chunk of staged uniforms / forced inputs
constexpr int NCH = 16;       // packed weight chunks (float4) per thread and layer: 8 of W_e, 8 of W_r
constexpr int NCO = 4;        // packed output-1x1 chunks per thread
static_assert(OC == 16 && KP == 16 && KW == 32 && QB == 8, "block geometry");

// Exchange words of a group (u64): handshake slots, the layer outputs, the logits, the samples.
constexpr int HSLOT = 32;                          // words per handshake slot (a 256-byte line)
__host__ __device__ inline size_t xw_layer(int L) { (void)L; return (size_t)NBG * OC * SG; }  // 2048 words
__host__ __device__ inline size_t group_words(int L) {
  return (size_t)(NBG + 1) * HSLOT + (size_t)L * xw_layer(L) + (size_t)NBG * QB * SG + (size_t)SG * HSLOT;
}
__host__ __device__ inline u64 *grp(void *comm, int L, int g) { return (u64 *)((char *)comm + 256) + g * group_words(L); }
__host__ __device__ inline u64 *g_hs(void *comm, int L, int g) { return grp(comm, L, g); }
__host__ __device__ inline u64 *g_x(void *comm, int L, int g, int l) {
  return grp(comm, L, g) + (NBG + 1) * HSLOT + (size_t)l * xw_layer(L);
}
__host__ __device__ inline u64 *g_lg(void *comm, int L, int g) { return g_x(comm, L, g, L); }
__host__ __device__ inline u64 *g_smp(void *comm, int L, int g) { return g_lg(comm, L, g) + NBG * QB * SG; }

// LDS of a block.
struct Lds {
  float xg[2][SG][KP][XP];  // layer input (all 512 channels) by layer parity: stream s, channel 32 kp + i
  float red[KP][OC][2 * SG];  // K-part partial sums: [kp][oc][e: s | r: 4 + s]
  float u[2][KCH];          // staged uniforms (sampler blocks)
  int fin[2][KCH][SG];      // staged forced next inputs
  int in[SG];               // the step's inputs
  int mode;                 // handshake result: the group shares one XCD
  // followed by the per-layer tables dil[L], qoff[L], slot[L] and the queues:
  // P[entries][OC][SG] (products W_r x) and X[entries][OC][SG] (states), entries = sum of dilations
};
__host__ __device__ inline size_t lds_tables(int L) { return (sizeof(Lds) + 15) & ~(size_t)15; }
__host__ __device__ inline size_t lds_queues(int L) { return lds_tables(L) + (((size_t)3 * L * 4 + 15) & ~(size_t)15); }

// ---- packed weights (per block j, same for every group): layer l at
// wl + ((size_t)l * NBG + j) * NCH * NT float4 (chunk i of thread t at [i][t]); the output 1x1 at
// wo + (size_t)j * NCO * NT float4.

// Weight registers are native 4-vectors: arrays of the HIP float4 struct live across the step loop
// were copied member-wise and kept in scratch memory.
typedef float wv4 __attribute__((ext_vector_type(4)));

// Products of the block's 16 channels for the 4 streams over its thread's K part, both taps, from the
// gathered layer input xs (x[s][kp][i]); partial sums into red.
__device__ __forceinline__ void layer_products(const wv4 (&w)[NCH], const float (*xs)[KP][XP], int oc, int kp,
                                               float (*red)[OC][2 * SG]) {
  float e[SG], r[SG];
#pragma unroll
  for (int s = 0; s < SG; ++s) e[s] = r[s] = 0.f;
#pragma unroll
  for (int i = 0; i < KW / 4; ++i) {
    const wv4 we = w[i], wr = w[8 + i];
#pragma unroll
    for (int s = 0; s < SG; ++s) {
      const float4 x = *(const float4 *)&xs[s][kp][4 * i];
      e[s] = fmaf(we.x, x.x, e[s]);
      e[s] = fmaf(we.y, x.y, e[s]);
      e[s] = fmaf(we.z, x.z, e[s]);
      e[s] = fmaf(we.w, x.w, e[s]);
      r[s] = fmaf(wr.x, x.x, r[s]);
      r[s] = fmaf(wr.y, x.y, r[s]);
      r[s] = fmaf(wr.z, x.z, r[s]);
      r[s] = fmaf(wr.w, x.w, r[s]);
    }
  }
#pragma unroll
  for (int s = 0; s < SG; ++s) {
    red[kp][oc][s] = e[s];
    red[kp][oc][SG + s] = r[s];
  }
}

__device__ __forceinline__ void load_layer_weights(wv4 (&w)[NCH], const float4 *wl, int l, int j, int tid) {
  const wv4 *src = (const wv4 *)(wl + ((size_t)l * NBG + j) * NCH * NT + tid);
#pragma unroll
  for (int i = 0; i < NCH; ++i) w[i] = src[i * NT];
}

// The weights of index t of the per-step sequence (layer t for t < L, the output 1x1's NCO chunks
// for t == L, nothing beyond).
__device__ __forceinline__ void load_seq_weights(wv4 (&w)[NCH], const float4 *wl, const float4 *wo4, int t, int L,
                                                 int j, int tid) {
  if (t < L) {
    load_layer_weights(w, wl, t, j, tid);
  } else if (t == L) {
    const wv4 *src = (const wv4 *)(wo4 + (size_t)j * NCO * NT + tid);
#pragma unroll
    for (int i = 0; i < NCO; ++i) w[i] = src[i * NT];
    // the rest of the buffer is written too (a buffer written in part on one path stayed in scratch)
#pragma unroll
    for (int i = NCO; i < NCH; ++i) w[i] = wv4{0.f, 0.f, 0.f, 0.f};
  }
}

// (plain values and pointers only: a reference to a by-value kernel argument would move the argument
// to scratch memory)
struct WideLayerCtx {
  void *comm;
  const float *convb;
  Lds *sp;
  const int *qoff, *slot;
  float *Pq, *Xq;
  const float4 *wl, *wo4;
  uint32_t *abort_word, *sticky;
  int L, g, j, tid, wave, oc, kp;
  bool local, residual;
};

// One layer: products from the weights in wc (the next-but-one index of the sequence fetched into
// wp first), the epilogue of the block's channels, the gather of the layer output.
__device__ __forceinline__ void wide_layer(const WideLayerCtx &c, int l, const wv4 (&wc)[NCH], wv4 (&wp)[NCH],
                                           uint32_t tag) {
  Lds &s = *c.sp;
  const int cur = l & 1, L = c.L, tid = c.tid, j = c.j, g = c.g;
  load_seq_weights(wp, c.wl, c.wo4, l + 2, L, j, tid);
  layer_products(wc, s.xg[cur], c.oc, c.kp, s.red);
  __syncthreads();
  // epilogue of the block's channels (wave 0, lane = (s, oc)): pop the product pushed d steps ago,
  // push this step's
  if (c.wave == 0) {
    const int o2 = tid & (OC - 1), st = tid >> 4, ch = 16 * j + o2;
    float e = 0.f, r = 0.f;
#pragma unroll
    for (int p = 0; p < KP; ++p) {
      e += s.red[p][o2][st];
      r += s.red[p][o2][SG + st];
    }
    const size_t ent = ((size_t)(c.qoff[l] + c.slot[l]) * OC + o2) * SG + st;
    const float xin = s.xg[cur][st][ch / KW][ch % KW];
    const float act = fmaxf(e + c.Pq[ent] + c.convb[l * C + ch], 0.f);
    const float xo = c.residual ? xin + act : act;
    c.Pq[ent] = r;
    c.Xq[ent] = xin;
    // the layer output to the group: word (s, oc) of this block's slice, two per store
    const float xo1 = __shfl_down(xo, 1, 64);
    if (o2 % 2 == 0)
      put_words2(g_x(c.comm, L, g, l) + j * OC * SG + st * OC + o2, __float_as_uint(xo), __float_as_uint(xo1),
                 tag, c.local);
  }
  // gather the whole layer output into the other buffer (this block's own slice included)
  {
    uint32_t v[8];
    wait_words<8, NT>(g_x(c.comm, L, g, l) + tid, tag, v, c.abort_word, c.sticky);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int wi = e * NT + tid, jb = wi / (OC * SG), rr = wi % (OC * SG), st = rr / OC, ch = 16 * jb + rr % OC;
      s.xg[cur ^ 1][st][ch / KW][ch % KW] = __uint_as_float(v[e]);
    }
  }
  __syncthreads();
}

__global__ void __launch_bounds__(NT) wide_step_kernel(StepArgs a, WideArgs w) {
  extern __shared__ float4 lds_raw[];
  Lds &s = *(Lds *)lds_raw;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = blockIdx.x % NG, j = blockIdx.x / NG, G = a.sp_nb, L = a.L;
  if (g >= G) return;  // this group has no streams (all of its threads leave before any barrier)
  const int b0 = g * SG;                       // the group's first stream
  const int nval = min(SG, a.batch - b0);      // its valid streams
  int *dil = (int *)((char *)lds_raw + lds_tables(L));
  int *qoff = dil + L, *slot = qoff + L;
  float *Pq = (float *)((char *)lds_raw + lds_queues(L));  // [entries][OC][SG]
  float *Xq = Pq + (size_t)w.entries * OC * SG;
  uint32_t *abort_word = (uint32_t *)a.sp_comm, *sticky = a.sp_sticky;
  const float4 *wl = (const float4 *)w.wl, *wo4 = (const float4 *)w.wo;
  const int oc = tid & (OC - 1), kp = tid >> 4;
  const bool residual = a.kind == 1;  // relu + residual (FWG_RELU_RESIDUAL)

  // ---- per-layer tables
  for (int l = tid; l < L; l += NT) {
    int off = 0;
    for (int i = 0; i < l; ++i) off += a.layers[i].dil;
    dil[l] = a.layers[l].dil;
    qoff[l] = off;
    slot[l] = (int)(a.t0 % (long long)a.layers[l].dil);
  }
  // ---- launch handshake: every block reports its XCD; block 0 tells the group whether all share one
  u64 *hs = g_hs(a.sp_comm, L, g);
  if (tid == 0) {
    put_word(hs + HSLOT * j, xcd_id(), 1, false);
    uint32_t v[1];
    if (j == 0) {
      bool local = true;
      const uint32_t mine = xcd_id();
      for (int jb = 0; jb < NBG; ++jb) {
        wait_words<1>(hs + HSLOT * jb, 1, v, abort_word, sticky);
        local = local && v[0] == mine;
      }
      put_word(hs + HSLOT * NBG, local ? 1u : 0u, 1, false);
      s.mode = local ? 1 : 0;
    } else {
      wait_words<1>(hs + HSLOT * NBG, 1, v, abort_word, sticky);
      s.mode = (int)v[0];
    }
  }
  // first inputs, first chunk of staged per-step inputs
  if (tid < SG) {
    const int bb = b0 + tid;
    int v = 0;
    if (tid < nval) v = a.mode == MODE_TEACHER ? a.inputs[(long long)bb * a.n_steps] : a.last[bb];
    s.in[tid] = v;
  }
  for (int e = tid; e < KCH * SG; e += NT) {
    const int jj = e / SG, st = e % SG, bb = b0 + st;
    const long long nx = jj + forced_shift(a.mode);
    s.fin[0][jj][st] = (a.mode != MODE_GENERATE && st < nval && nx < a.n_steps) ? a.inputs[(long long)bb * a.n_steps + nx] : 0;
  }
  if (j < SG && tid < KCH) {
    const int bb = b0 + j;
    s.u[0][tid] = (a.mode == MODE_GENERATE && j < nval && tid < a.n_steps) ? a.uniforms[(long long)bb * a.n_steps + tid] : 0.f;
  }
  __syncthreads();
  const bool local = s.mode != 0;

  // ---- the launch's state: the states of this block's channels from the workspace queues, and the
  // products W_r x of every queued state (a pass over each layer's slots with the layer's weights)
  {
    wv4 wv[NCH];
    for (int l = 0; l < L; ++l) {
      load_layer_weights(wv, wl, l, j, tid);
      const float *src = (const float *)a.ring + a.layers[l].ring_off;
      for (int sl = 0; sl < dil[l]; ++sl) {
        // the whole queued state (all 512 channels, 4 streams) into xg[0]
        for (int e = tid; e < SG * C; e += NT) {
          const int st = e / C, c = e % C;
          s.xg[0][st][c / KW][c % KW] = st < nval ? src[((long long)sl * a.bmax + b0 + st) * C + c] : 0.f;
        }
        __syncthreads();
        layer_products(wv, s.xg[0], oc, kp, s.red);
        __syncthreads();
        if (tid < OC * SG) {
          const int o2 = tid & (OC - 1), st = tid >> 4;
          float r = 0.f;
#pragma unroll
          for (int p = 0; p < KP; ++p) r += s.red[p][o2][SG + st];
          const size_t ent = ((size_t)(qoff[l] + sl) * OC + o2) * SG + st;
          Pq[ent] = r;
          Xq[ent] = s.xg[0][st][(16 * j + o2) / KW][(16 * j + o2) % KW];
        }
        __syncthreads();
      }
    }
  }

  const float *embT = w.embT, *embb = w.embb, *convb = w.convb, *outb = w.outb;
  // weights stream through three register buffers, two layers ahead (index t of the step's
  // sequence in buffer t mod 3: layers 0..L-1, then the output 1x1): with one layer in flight the
  // group's loads did not cover the latency of the last-level cache
  wv4 W0[NCH], W1[NCH], W2[NCH];
  load_seq_weights(W0, wl, wo4, 0, L, j, tid);
  load_seq_weights(W1, wl, wo4, 1, L, j, tid);

  for (int step = 0; step < a.n_steps; ++step) {
    const uint32_t tag = (uint32_t)(step + 1);
    // ---- layer input x^0 (the embedding of the step's inputs), all 512 channels
    for (int e = tid; e < SG * C; e += NT) {
      const int st = e / C, c = e % C;
      s.xg[0][st][c / KW][c % KW] = embT[(size_t)s.in[st] * C + c] + embb[c];
    }
    __syncthreads();
    const WideLayerCtx cx{a.sp_comm, w.convb, &s, qoff, slot, Pq, Xq, wl, wo4, abort_word, sticky,
                          L, g, j, tid, wave, oc, kp, local, residual};
    for (int l = 0; l < L; l += 3) {
      wide_layer(cx, l, W0, W2, tag);
      if (l + 1 < L) wide_layer(cx, l + 1, W1, W0, tag);
      if (l + 2 < L) wide_layer(cx, l + 2, W2, W1, tag);
    }
    // ---- output 1x1: classes 8j..8j+7; thread (c8, kq) covers K part kq (16 channels)
    {
      const int lastp = L & 1;
      const int c8 = tid & (QB - 1), kq = tid >> 3;
      float acc[SG];
#pragma unroll
      for (int st = 0; st < SG; ++st) acc[st] = 0.f;
      const int ob = L % 3;  // the output 1x1's weights: index L of the sequence
#pragma unroll
      for (int i = 0; i < NCO; ++i) {
        const wv4 wv = ob == 0 ? W0[i] : ob == 1 ? W1[i] : W2[i];
        const int k = 16 * kq + 4 * i;
#pragma unroll
        for (int st = 0; st < SG; ++st) {
          const float4 x = *(const float4 *)&s.xg[lastp][st][k / KW][k % KW];
          acc[st] = fmaf(wv.x, x.x, acc[st]);
          acc[st] = fmaf(wv.y, x.y, acc[st]);
          acc[st] = fmaf(wv.z, x.z, acc[st]);
          acc[st] = fmaf(wv.w, x.w, acc[st]);
        }
      }
      // 32 K parts x 8 classes x 4 streams of partial sums (the layer scratch viewed flat)
      float *r2 = &s.red[0][0][0];
#pragma unroll
      for (int st = 0; st < SG; ++st) r2[(kq * QB + c8) * SG + st] = acc[st];
      // the next step's first two indices, read while the logits are summed and sampled
      load_seq_weights(W0, wl, wo4, 0, L, j, tid);
      load_seq_weights(W1, wl, wo4, 1, L, j, tid);
      __syncthreads();
      if (wave == 0) {
        // lanes 0..31: (s, class); lanes 32..63 repeat them and store nothing
        const int cc = tid & (QB - 1), st = (tid >> 3) & (SG - 1), cls = QB * j + cc;
        float lg = outb[cls];
        for (int p = 0; p < NT / QB; ++p) lg += r2[(p * QB + cc) * SG + st];
        const float lg1 = __shfl_down(lg, 1, 64);
        if (tid < QB * SG) {
          if (a.mode != MODE_GENERATE && a.logits && st < nval)
            a.logits[((long long)(b0 + st) * a.n_steps + step) * Q + cls] = lg;
          if (cc % 2 == 0)
            put_words2(g_lg(a.sp_comm, L, g) + j * QB * SG + st * QB + cc, __float_as_uint(lg), __float_as_uint(lg1),
                       tag, local);
        }
      }
    }
    // ---- sampler blocks: block s < 4 takes stream s of the group (wave 0): lane l gathers classes
    // 4l..4l+3 (block l / 2's words, classes 4 (l % 2) .. + 3)
    if (j < SG && wave == 0) {
      uint32_t v[4];
      const u64 *src = g_lg(a.sp_comm, L, g) + (lane >> 1) * QB * SG + j * QB + 4 * (lane & 1);
      wait_words<4>(src, tag, v, abort_word, sticky);
      uint32_t res = 0u;
      if (a.mode == MODE_GENERATE) {
        const float4 lg4 = make_float4(__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]),
                                       __uint_as_float(v[3]));
        const int k = sample_row4(lg4, s.u[(step / KCH) & 1][step % KCH]);
        if (lane == 0 && j < nval) a.samples[(long long)(b0 + j) * a.n_steps + step] = k;
        res = (uint32_t)k;
      }
      if (lane == 0) put_word(g_smp(a.sp_comm, L, g) + HSLOT * j, res, tag, local);
    }
    // ---- the step's samples (step-done marks in forced modes) from the group's sampler blocks
    if (tid < SG) {
      uint32_t v[1];
      wait_words<1>(g_smp(a.sp_comm, L, g) + HSLOT * tid, tag, v, abort_word, sticky);
      s.in[tid] = a.mode == MODE_GENERATE ? (int)v[0] : s.fin[(step / KCH) & 1][step % KCH][tid];
    }
    // slot advance, then staging of the next chunk (every forced input before it is used)
    for (int l = tid; l < L; l += NT) slot[l] = slot[l] + 1 == dil[l] ? 0 : slot[l] + 1;
    if ((step + 1) % KCH == 0) {
      const int base = step + 1, buf = ((step + 1) / KCH) & 1;
      for (int e = tid; e < KCH * SG; e += NT) {
        const int jj = e / SG, st = e % SG, bb = b0 + st;
        const long long nx = base + jj + forced_shift(a.mode);
        s.fin[buf][jj][st] = (a.mode != MODE_GENERATE && st < nval && nx < a.n_steps) ? a.inputs[(long long)bb * a.n_steps + nx] : 0;
      }
      if (j < SG && tid < KCH) {
        const int bb = b0 + j;
        s.u[buf][tid] = (a.mode == MODE_GENERATE && j < nval && base + tid < a.n_steps)
                            ? a.uniforms[(long long)bb * a.n_steps + base + tid] : 0.f;
      }
    }
    __syncthreads();
  }

  // ---- launch end: the states of this block's channels back to the workspace queues; the pending
  // inputs (block 0 of the group)
  for (int l = 0; l < L; ++l) {
    float *dst = (float *)a.ring + a.layers[l].ring_off;
    for (int e = tid; e < dil[l] * OC * SG; e += NT) {
      const int sl = e / (OC * SG), rr = e % (OC * SG), o2 = rr / SG, st = rr % SG;
      if (st < nval) dst[((long long)sl * a.bmax + b0 + st) * C + 16 * j + o2] = Xq[(size_t)(qoff[l] + sl) * OC * SG + rr];
    }
  }
  if (j == 0 && tid < nval && a.mode != MODE_TEACHER) a.last[b0 + tid] = s.in[tid];
}

// ---- repacking (once per fwg_create)
__global__ void wide_pack_layer_kernel(const float *conv, int l, float4 *wl) {
  // chunk i of thread t of block j: oc = t % 16, kp = t / 16; i < 8: W_e[16j + oc][32 kp + 4i ..],
  // i >= 8: W_r[16j + oc][32 kp + 4(i - 8) ..]; conv is [C][C][2] (tap 0 = W_r, tap 1 = W_e)
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= NBG * NCH * NT) return;
  const int t = e % NT, i = (e / NT) % NCH, jb = e / (NT * NCH);
  const int o = 16 * jb + (t & (OC - 1)), k0 = KW * (t >> 4) + 4 * (i & 7), tap = i < 8 ? 1 : 0;
  float v[4];
  for (int q = 0; q < 4; ++q) v[q] = conv[((size_t)o * C + k0 + q) * 2 + tap];
  wl[((size_t)l * NBG + jb) * NCH * NT + (size_t)i * NT + t] = make_float4(v[0], v[1], v[2], v[3]);
}
__global__ void wide_pack_out_kernel(const float *out, float4 *wo) {
  // chunk i of thread t of block j: class 8j + t % 8, channels 16 (t / 8) + 4i ..
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= NBG * NCO * NT) return;
  const int t = e % NT, i = (e / NT) % NCO, jb = e / (NT * NCO);
  const int cls = QB * jb + (t & (QB - 1)), k0 = 16 * (t >> 3) + 4 * i;
  float v[4];
  for (int q = 0; q < 4; ++q) v[q] = out[(size_t)cls * C + k0 + q];
  wo[((size_t)jb * NCO + i) * NT + t] = make_float4(v[0], v[1], v[2], v[3]);
}
__global__ void wide_transpose_kernel(const float *src, float *dst, int rows, int cols) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= rows * cols) return;
  dst[(size_t)(e % cols) * rows + e / cols] = src[e];  // dst[c][r] = src[r][c]
}
__global__ void wide_vec_kernel(const float *src, float *dst, int n) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e < n) dst[e] = src ? src[e] : 0.f;
}

}  // namespace wd

bool wide_layout(int kind, int dtype, int C, int Q, int L, int w, int bmax, const int32_t *dil, WideArgs *g,
                 size_t *lds, size_t *comm_bytes) {
  if ((kind != 0 && kind != 1) || dtype != 0 || C != kWideC || Q != 256 || w != 2 || L < 1 || L > 256 ||
      bmax > kWideStreams * kWideGroups)
    return false;
  long long ent = 0;
  for (int l = 0; l < L; ++l) ent += dil[l];
  g->entries = (int)ent;
  g->wl_bytes = (size_t)L * wd::NBG * wd::NCH * wd::NT * 16;
  g->wo_bytes = (size_t)wd::NBG * wd::NCO * wd::NT * 16;
  *lds = wd::lds_queues(L) + (size_t)2 * ent * wd::OC * wd::SG * 4;
  *comm_bytes = 256 + (size_t)wd::NG * wd::group_words(L) * 8;
  return ent < (1 << 20) && *lds <= 160 * 1024;
}

size_t wide_comm_bytes(int L) { return 256 + (size_t)wd::NG * wd::group_words(L) * 8; }

hipError_t wide_setup(size_t lds, int *coresident_ok) {
  hipError_t e = hipFuncSetAttribute((const void *)wd::wide_step_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds);
  if (e != hipSuccess) return e;
  int per_cu = 0, dev = 0, cus = 0;
  if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, wd::wide_step_kernel, wd::NT, lds)) != hipSuccess)
    return e;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  *coresident_ok = (long long)per_cu * cus >= (long long)wd::NG * wd::NBG;
  return hipSuccess;
}

hipError_t launch_wide_step(const StepArgs &a, const WideArgs &g, size_t lds, hipStream_t s) {
  hipLaunchKernelGGL(wd::wide_step_kernel, dim3(wd::NG * wd::NBG), dim3(wd::NT), lds, s, a, g);
  return hipGetLastError();
}

hipError_t launch_wide_pack(const void *embed, const float *embed_b, const void *const *conv,
                            const float *const *conv_b, const void *out, const float *out_b, int L, const WideArgs &g,
                            hipStream_t s) {
  const int C = kWideC, Q = 256;
  for (int l = 0; l < L; ++l) {
    hipLaunchKernelGGL(wd::wide_pack_layer_kernel, dim3((wd::NBG * wd::NCH * wd::NT + 255) / 256), dim3(256), 0, s,
                       (const float *)conv[l], l, (float4 *)g.wl);
    hipLaunchKernelGGL(wd::wide_vec_kernel, dim3((C + 255) / 256), dim3(256), 0, s, conv_b ? conv_b[l] : nullptr,
                       (float *)g.convb + (size_t)l * C, C);
  }
  hipLaunchKernelGGL(wd::wide_pack_out_kernel, dim3((wd::NBG * wd::NCO * wd::NT + 255) / 256), dim3(256), 0, s,
                     (const float *)out, (float4 *)g.wo);
  hipLaunchKernelGGL(wd::wide_transpose_kernel, dim3((C * Q + 255) / 256), dim3(256), 0, s, (const float *)embed,
                     (float *)g.embT, C, Q);
  hipLaunchKernelGGL(wd::wide_vec_kernel, dim3((C + 255) / 256), dim3(256), 0, s, embed_b, (float *)g.embb, C);
  hipLaunchKernelGGL(wd::wide_vec_kernel, dim3(1), dim3(256), 0, s, out_b, (float *)g.outb, Q);
  return hipGetLastError();
}

}  // namespace fwg
