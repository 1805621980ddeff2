// Wide step kernel for float32 ReLU stacks with C = 512 channels (filter width 2): every layer is
// spread over the 32 blocks of a group, one group per XCD and up to four streams per group.
//
// One sample is a chain of L dependent layers, each a 512 x 1024 product (Section 1: the edges of
// the graph are matrix products), then the output 1x1 and the sample fed back (Section 1).  A single
// block would stream 2 MB of weights per layer; here block j of a group owns output channels
// 16j..16j+15 of every layer:
//  - per layer it reads its 64 KB of weights (W_e and W_r rows; the whole model stays resident in
//    the 256 MB last-level cache) and computes both products of its 16 channels for the group's 4
//    streams over the whole layer input: thread (oc, kp) of the four compute waves covers channel oc
//    over K part kp (32 channels), and the 16 K parts meet in LDS;
//  - a fifth wave only streams weights: it copies the step's sequence of 16 KB chunks (each layer's
//    weights as four chunks, then the output 1x1's) into a ring of LDS slots, one chunk in flight,
//    and the compute waves take each chunk from its slot.  The weight stream of an XCD is bound by
//    what the XCD can fetch beyond its L2, and a wave that issues a layer's loads itself stalls at
//    the issue until the compute unit's memory queue drains; with the loads on their own wave the
//    products, the exchange and the polls run while the next weights arrive.  The compute waves
//    synchronise through LDS counters, not block barriers, so the streaming wave never waits for
//    them except for a free slot;
//  - the queue (Section 2.2) keeps, per block, the product W_r x of its own channels instead of the
//    state x: a = W_e x_t + (W_r x_{t-d}) + b pops the product pushed d steps earlier, so no block
//    reads another block's queue.  The states of its own channels are pushed to the workspace queues
//    (the generation state every kernel family shares); at launch the products are recomputed from
//    them;
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
constexpr int NTL = 64;       // the streaming wave
constexpr int XP = KW + 4;    // floats per (stream, K part) row of the gathered layer input (padding spreads banks)
constexpr int KCH = 64;       // steps per chunk of staged uniforms / forced inputs
constexpr int CPL = 4;        // weight chunks per layer
constexpr int CF4 = 4;        // float4 per compute thread and chunk
constexpr int CHUNK = CF4 * NT;  // float4 per chunk (16 KB)
constexpr int NCO = 4;        // float4 per compute thread of the output 1x1 (one chunk)
constexpr int MAXSLOT = 8;    // ring slots at most
static_assert(OC == 16 && KP == 16 && KW == 32 && QB == 8, "block geometry");
static_assert(NCO == CF4 && (KW / 4) == 2 * CPL, "a layer is four chunks, the output 1x1 one");

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

typedef __attribute__((address_space(3))) volatile int lds_flag;

// LDS of a block.
struct Lds {
  float xg[2][SG][KP][XP];  // layer input (all 512 channels) by layer parity: stream s, channel 32 kp + i
  float red[KP][OC][2 * SG];  // K-part partial sums: [kp][oc][e: s | r: 4 + s]
  float u[2][KCH];          // staged uniforms (sampler blocks)
  int fin[2][KCH][SG];      // staged forced next inputs
  int in[SG];               // the step's inputs
  int mode;                 // handshake result: the group shares one XCD
  int ready[MAXSLOT];       // ring slot s holds chunk k of the launch once ready[s] == k + 1
  int cons[4];              // chunks each compute wave has finished reading
  int cbar;                 // compute-wave barrier counter (each wave adds 1 per barrier)
  int abort_;               // an LDS wait ran out: later LDS waits return at once
  // followed by the per-layer tables dil[L], qoff[L], slot[L], the conv biases of the block's
  // channels [L][OC], the ring of weight slots and the queue P[entries][OC][SG] (products W_r x),
  // entries = sum of dilations
};
__host__ __device__ inline size_t lds_tables() { return (sizeof(Lds) + 15) & ~(size_t)15; }
__host__ __device__ inline size_t lds_ring(int L) {
  return lds_tables() + (((size_t)(3 + OC) * L * 4 + 15) & ~(size_t)15);
}
__host__ __device__ inline size_t lds_queue(int L, int ns) { return lds_ring(L) + (size_t)ns * CHUNK * 16; }

// ---- packed weights (per block j, same for every group): chunk c of layer l at
// wl + ((size_t)(CPL l + c) * NBG + j) * CHUNK float4, float4 i of compute thread t at [i][t]:
// i = 0, 1: W_e row chunks 2c, 2c + 1 of the thread's K part, i = 2, 3: W_r likewise; the output
// 1x1 at wo + (size_t)j * CHUNK float4 (thread (c8, kq): class 8j + c8, channels 16 kq + 4i ..).

__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

// Waits until *flag >= want (every LDS wait of the launch is bounded: one that runs out marks the
// block's LDS abort word and the launch's sticky word, and every later LDS wait returns at once).
__device__ __forceinline__ void wait_ge(Lds &s, lds_flag *flag, int want, uint32_t *sticky) {
  lds_flag *ab = (lds_flag *)&s.abort_;
  for (int it = 0; *flag < want; ++it) {
    if (*ab) break;
    if (it >= kSpinMax) {
      *ab = 1;
      __hip_atomic_store(sticky, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      break;
    }
    __builtin_amdgcn_s_sleep(1);
  }
  compiler_fence();
}

// Barrier of the four compute waves (the streaming wave takes no part): each wave adds 1 and waits
// for the count of this barrier.  A wave's LDS operations run in order, so its writes before the
// add are visible to a wave that has seen the count.
__device__ __forceinline__ void cbar(Lds &s, int &ph, int lane, uint32_t *sticky) {
  ph += 4;
  compiler_fence();
  if (lane == 0) __hip_atomic_fetch_add((__attribute__((address_space(3))) int *)&s.cbar, 1, __ATOMIC_RELAXED,
                                        __HIP_MEMORY_SCOPE_WORKGROUP);
  wait_ge(s, (lds_flag *)&s.cbar, ph, sticky);
}

// Compute wave: chunk k of the launch is in its slot; afterwards the slot may be refilled.
__device__ __forceinline__ const float4 *take_chunk(Lds &s, const float4 *ring, long long k, int ns, uint32_t *sticky) {
  const int slot = (int)(k % ns);
  lds_flag *f = (lds_flag *)&s.ready[slot];
  lds_flag *ab = (lds_flag *)&s.abort_;
  for (int it = 0; *f != (int)(k + 1); ++it) {
    if (*ab) break;
    if (it >= kSpinMax) {
      *ab = 1;
      __hip_atomic_store(sticky, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      break;
    }
    __builtin_amdgcn_s_sleep(1);
  }
  compiler_fence();
  return ring + (size_t)slot * CHUNK;
}
__device__ __forceinline__ void done_chunk(Lds &s, int wave, int lane, long long k) {
  compiler_fence();
  if (lane == 0) *(lds_flag *)&s.cons[wave] = (int)(k + 1);
}

// Products of the block's 16 channels for the 4 streams over chunk c of the thread's K part (K
// 8c .. 8c + 7), both taps, accumulated into e and r (the same order of operations as one pass
// over the eight K groups of the part).
__device__ __forceinline__ void chunk_products(const float4 *ch, const float (*xs)[KP][XP], int tid, int kp, int c,
                                               float (&e)[SG], float (&r)[SG]) {
  float4 w[CF4];
#pragma unroll
  for (int i = 0; i < CF4; ++i) w[i] = ch[i * NT + tid];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const float4 we = w[h], wr = w[2 + h];
#pragma unroll
    for (int s = 0; s < SG; ++s) {
      const float4 x = *(const float4 *)&xs[s][kp][8 * c + 4 * h];
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
}

// The streaming wave: every chunk of the launch (n_steps x (4 L + 1)) into ring slot k mod ns with
// loads that write LDS directly (no register copy), one chunk in flight (a second one made the
// compute waves' polls wait longer behind the stream's loads and the step slower); a slot is
// loaded once every compute wave has finished reading its last chunk.
struct Stream {
  const float4 *wl, *wo4;
  int L, j, ns, per_step;
};
__device__ __forceinline__ const float4 *chunk_src(const Stream &m, int q) {
  return q < CPL * m.L ? m.wl + ((size_t)q * NBG + m.j) * CHUNK : m.wo4 + (size_t)m.j * CHUNK;
}
__device__ __forceinline__ void stream_weights(Lds &s, float4 *ring, const Stream &m, long long n_steps, int lane,
                                               uint32_t *sticky) {
  const long long total = n_steps * m.per_step;
  int q = 0, slot = 0;  // chunk of the step and ring slot of chunk k
  for (long long k = 0; k < total; ++k) {
    if (k >= m.ns) {
      // the slot's previous chunk (k - ns) read by all four compute waves
      const int want = (int)(k - m.ns + 1);
#pragma unroll
      for (int w = 0; w < 4; ++w) wait_ge(s, (lds_flag *)&s.cons[w], want, sticky);
    }
    const float4 *src = chunk_src(m, q) + lane;
    float4 *dst = ring + (size_t)slot * CHUNK;
    // lane i's 16 bytes of each load land at dst + 16 i (64 lanes: 1 KB per load)
#pragma unroll
    for (int u = 0; u < CHUNK / NTL; ++u)
      __builtin_amdgcn_global_load_lds((const void *)(src + u * NTL), (__attribute__((address_space(3))) void *)(dst + u * NTL),
                                       16, 0, 0);
    // vmcnt(0): the chunk is in LDS (the count drops once a load's data is written there)
    __builtin_amdgcn_s_waitcnt(0x0F70);
    compiler_fence();
    if (lane == 0) *(lds_flag *)&s.ready[slot] = (int)(k + 1);
    q = q + 1 == m.per_step ? 0 : q + 1;
    slot = slot + 1 == m.ns ? 0 : slot + 1;
  }
}

__global__ void __launch_bounds__(NT + NTL) wide_step_kernel(StepArgs a, WideArgs w) {
  extern __shared__ float4 lds_raw[];
  Lds &s = *(Lds *)lds_raw;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = blockIdx.x % NG, j = blockIdx.x / NG, G = a.sp_nb, L = a.L;
  if (g >= G) return;  // this group has no streams (all of its threads leave before any barrier)
  const int b0 = g * SG;                       // the group's first stream
  const int nval = min(SG, a.batch - b0);      // its valid streams
  const int ns = w.nslots;
  int *dil = (int *)((char *)lds_raw + lds_tables());
  int *qoff = dil + L, *slot = qoff + L;
  float *cb = (float *)(slot + L);  // [L][OC]: conv biases of the block's channels (no global load per layer)
  float4 *ring = (float4 *)((char *)lds_raw + lds_ring(L));
  float *Pq = (float *)((char *)lds_raw + lds_queue(L, ns));  // [entries][OC][SG]
  uint32_t *abort_word = (uint32_t *)a.sp_comm, *sticky = a.sp_sticky;
  const float4 *wl = (const float4 *)w.wl, *wo4 = (const float4 *)w.wo;
  const int oc = tid & (OC - 1), kp = tid >> 4;
  const bool residual = a.kind == 1;  // relu + residual (FWG_RELU_RESIDUAL)

  // ---- per-layer tables, ring flags and counters
  for (int l = tid; l < L; l += NT + NTL) {
    int off = 0;
    for (int i = 0; i < l; ++i) off += a.layers[i].dil;
    dil[l] = a.layers[l].dil;
    qoff[l] = off;
    slot[l] = (int)(a.t0 % (long long)a.layers[l].dil);
  }
  for (int i = tid; i < L * OC; i += NT + NTL) cb[i] = w.convb[(i / OC) * C + 16 * j + i % OC];
  if (tid < MAXSLOT) s.ready[tid] = 0;
  if (tid < 4) s.cons[tid] = 0;
  if (tid == 0) {
    s.cbar = 0;
    s.abort_ = 0;
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
  for (int e = tid; e < KCH * SG; e += NT + NTL) {
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

  // ---- the streaming wave: from here on it runs on its own
  if (tid >= NT) {
    const Stream m{wl, wo4, L, j, ns, CPL * L + 1};
    stream_weights(s, ring, m, a.n_steps, lane, sticky);
    return;
  }

  int ph = 0;  // compute-wave barrier count
  // ---- the launch's state: the products W_r x of every queued state of this block's channels (a
  // pass over each layer's slots with the layer's W_r rows, read straight from the packed weights)
  for (int l = 0; l < L; ++l) {
    float4 wr[2 * CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c)
#pragma unroll
      for (int h = 0; h < 2; ++h) wr[2 * c + h] = wl[((size_t)(CPL * l + c) * NBG + j) * CHUNK + (2 + h) * NT + tid];
    const float *src = (const float *)a.ring + a.layers[l].ring_off;
    for (int sl = 0; sl < dil[l]; ++sl) {
      // the whole queued state (all 512 channels, 4 streams) into xg[0]
      for (int e = tid; e < SG * C; e += NT) {
        const int st = e / C, c = e % C;
        s.xg[0][st][c / KW][c % KW] = st < nval ? src[((long long)sl * a.bmax + b0 + st) * C + c] : 0.f;
      }
      cbar(s, ph, lane, sticky);
      float r[SG];
#pragma unroll
      for (int st = 0; st < SG; ++st) r[st] = 0.f;
#pragma unroll
      for (int i = 0; i < 2 * CPL; ++i) {
#pragma unroll
        for (int st = 0; st < SG; ++st) {
          const float4 x = *(const float4 *)&s.xg[0][st][kp][4 * i];
          r[st] = fmaf(wr[i].x, x.x, r[st]);
          r[st] = fmaf(wr[i].y, x.y, r[st]);
          r[st] = fmaf(wr[i].z, x.z, r[st]);
          r[st] = fmaf(wr[i].w, x.w, r[st]);
        }
      }
#pragma unroll
      for (int st = 0; st < SG; ++st) s.red[kp][oc][SG + st] = r[st];
      cbar(s, ph, lane, sticky);
      if (tid < OC * SG) {
        const int o2 = tid & (OC - 1), st = tid >> 4;
        float rr = 0.f;
#pragma unroll
        for (int p = 0; p < KP; ++p) rr += s.red[p][o2][SG + st];
        Pq[((size_t)(qoff[l] + sl) * OC + o2) * SG + st] = rr;
      }
      cbar(s, ph, lane, sticky);
    }
  }

  const float *embT = w.embT, *embb = w.embb, *outb = w.outb;
  long long k = 0;  // chunk of the launch the compute waves take next
  for (int step = 0; step < a.n_steps; ++step) {
    const uint32_t tag = (uint32_t)(step + 1);
    // ---- layer input x^0 (the embedding of the step's inputs), all 512 channels
    for (int e = tid; e < SG * C; e += NT) {
      const int st = e / C, c = e % C;
      s.xg[0][st][c / KW][c % KW] = embT[(size_t)s.in[st] * C + c] + embb[c];
    }
    cbar(s, ph, lane, sticky);
    for (int l = 0; l < L; ++l) {
      const int cur = l & 1;
      float e[SG], r[SG];
#pragma unroll
      for (int st = 0; st < SG; ++st) e[st] = r[st] = 0.f;
      // one wait for the layer's last chunk: the stream writes chunks in order, and none of the
      // layer's slots is refilled before this wave has read it (at least four slots), so the LDS reads
      // of all four chunks can run ahead of their products
      take_chunk(s, ring, k + CPL - 1, ns, sticky);
#pragma unroll
      for (int c = 0; c < CPL; ++c)
        chunk_products(ring + (size_t)((k + c) % ns) * CHUNK, s.xg[cur], tid, kp, c, e, r);
      done_chunk(s, wave, lane, k + CPL - 1);
      k += CPL;
#pragma unroll
      for (int st = 0; st < SG; ++st) {
        s.red[kp][oc][st] = e[st];
        s.red[kp][oc][SG + st] = r[st];
      }
      cbar(s, ph, lane, sticky);
      // epilogue of the block's channels (wave 0, lane = (s, oc)): pop the product pushed d steps
      // ago, push this step's
      float xin = 0.f;
      if (wave == 0) {
        const int o2 = tid & (OC - 1), st = tid >> 4, ch = 16 * j + o2;
        float ee = 0.f, rr = 0.f;
#pragma unroll
        for (int p = 0; p < KP; ++p) {
          ee += s.red[p][o2][st];
          rr += s.red[p][o2][SG + st];
        }
        const size_t ent = ((size_t)(qoff[l] + slot[l]) * OC + o2) * SG + st;
        xin = s.xg[cur][st][ch / KW][ch % KW];
        const float act = fmaxf(ee + Pq[ent] + cb[l * OC + o2], 0.f);
        const float xo = residual ? xin + act : act;
        Pq[ent] = rr;
        // the layer output to the group: word (s, oc) of this block's slice, two per store
        const float xo1 = __shfl_down(xo, 1, 64);
        if (o2 % 2 == 0)
          put_words2(g_x(a.sp_comm, L, g, l) + j * OC * SG + st * OC + o2, __float_as_uint(xo), __float_as_uint(xo1),
                     tag, local);
      }
      // gather the whole layer output into the other buffer (this block's own slice included)
      {
        uint32_t v[8];
        wait_words<8, NT>(g_x(a.sp_comm, L, g, l) + tid, tag, v, abort_word, sticky);
#pragma unroll
        for (int ee = 0; ee < 8; ++ee) {
          const int wi = ee * NT + tid, jb = wi / (OC * SG), rr = wi % (OC * SG), st = rr / OC, ch = 16 * jb + rr % OC;
          s.xg[cur ^ 1][st][ch / KW][ch % KW] = __uint_as_float(v[ee]);
        }
      }
      // the layer input of the block's channels to the workspace queue, once every block of the
      // group has published this layer (so none is still reading the queues in its state pass)
      if (wave == 0) {
        const int o2 = tid & (OC - 1), st = tid >> 4;
        if (st < nval)
          ((float *)a.ring)[a.layers[l].ring_off + ((long long)slot[l] * a.bmax + b0 + st) * C + 16 * j + o2] = xin;
      }
      cbar(s, ph, lane, sticky);
    }
    // ---- output 1x1: classes 8j..8j+7; thread (c8, kq) covers K part kq (16 channels)
    {
      const int lastp = L & 1;
      const int c8 = tid & (QB - 1), kq = tid >> 3;
      float acc[SG];
#pragma unroll
      for (int st = 0; st < SG; ++st) acc[st] = 0.f;
      const float4 *ch = take_chunk(s, ring, k, ns, sticky);
      float4 wv[NCO];
#pragma unroll
      for (int i = 0; i < NCO; ++i) wv[i] = ch[i * NT + tid];
      done_chunk(s, wave, lane, k);
      ++k;
#pragma unroll
      for (int i = 0; i < NCO; ++i) {
        const int kk = 16 * kq + 4 * i;
#pragma unroll
        for (int st = 0; st < SG; ++st) {
          const float4 x = *(const float4 *)&s.xg[lastp][st][kk / KW][kk % KW];
          acc[st] = fmaf(wv[i].x, x.x, acc[st]);
          acc[st] = fmaf(wv[i].y, x.y, acc[st]);
          acc[st] = fmaf(wv[i].z, x.z, acc[st]);
          acc[st] = fmaf(wv[i].w, x.w, acc[st]);
        }
      }
      // 32 K parts x 8 classes x 4 streams of partial sums (the layer scratch viewed flat)
      float *r2 = &s.red[0][0][0];
#pragma unroll
      for (int st = 0; st < SG; ++st) r2[(kq * QB + c8) * SG + st] = acc[st];
      cbar(s, ph, lane, sticky);
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
        const int kc = sample_row4(lg4, s.u[(step / KCH) & 1][step % KCH]);
        if (lane == 0 && j < nval) a.samples[(long long)(b0 + j) * a.n_steps + step] = kc;
        res = (uint32_t)kc;
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
    cbar(s, ph, lane, sticky);
  }
  // the pending inputs (block 0 of the group)
  if (j == 0 && tid < nval && a.mode != MODE_TEACHER) a.last[b0 + tid] = s.in[tid];
}

// ---- repacking (once per fwg_create)
__global__ void wide_pack_layer_kernel(const float *conv, int l, float4 *wl) {
  // float4 i of compute thread t of block j in chunk c: oc = t % 16, kp = t / 16; i < 2:
  // W_e[16j + oc][32 kp + 8c + 4i ..], i >= 2: W_r[16j + oc][32 kp + 8c + 4(i - 2) ..]; conv is
  // [C][C][2] (tap 0 = W_r, tap 1 = W_e)
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= NBG * CPL * CHUNK) return;
  const int t = e % NT, i = (e / NT) % CF4, jb = (e / CHUNK) % NBG, c = e / (CHUNK * NBG);
  const int o = 16 * jb + (t & (OC - 1)), k0 = KW * (t >> 4) + 8 * c + 4 * (i & 1), tap = i < 2 ? 1 : 0;
  float v[4];
  for (int q = 0; q < 4; ++q) v[q] = conv[((size_t)o * C + k0 + q) * 2 + tap];
  wl[((size_t)(CPL * l + c) * NBG + jb) * CHUNK + (size_t)i * NT + t] = make_float4(v[0], v[1], v[2], v[3]);
}
__global__ void wide_pack_out_kernel(const float *out, float4 *wo) {
  // float4 i of thread t of block j: class 8j + t % 8, channels 16 (t / 8) + 4i ..
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= NBG * CHUNK) return;
  const int t = e % NT, i = (e / NT) % NCO, jb = e / CHUNK;
  const int cls = QB * jb + (t & (QB - 1)), k0 = 16 * (t >> 3) + 4 * i;
  float v[4];
  for (int q = 0; q < 4; ++q) v[q] = out[(size_t)cls * C + k0 + q];
  wo[(size_t)jb * CHUNK + (size_t)i * NT + t] = make_float4(v[0], v[1], v[2], v[3]);
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
  if (ent >= (1 << 20)) return false;
  g->entries = (int)ent;
  g->wl_bytes = (size_t)L * wd::CPL * wd::NBG * wd::CHUNK * 16;
  g->wo_bytes = (size_t)wd::NBG * wd::CHUNK * 16;
  // the ring takes what LDS is left after the tables and the queue, at most MAXSLOT slots; at least
  // four: a compute wave waits once per layer, for its last chunk, with the other three in their slots
  const size_t limit = 160 * 1024, fixed = wd::lds_ring(L) + (size_t)ent * wd::OC * wd::SG * 4;
  if (fixed + (size_t)wd::CPL * wd::CHUNK * 16 > limit) return false;
  const size_t ns = (limit - fixed) / ((size_t)wd::CHUNK * 16);
  g->nslots = (int)(ns < (size_t)wd::MAXSLOT ? ns : wd::MAXSLOT);
  *lds = fixed + (size_t)g->nslots * wd::CHUNK * 16;
  *comm_bytes = 256 + (size_t)wd::NG * wd::group_words(L) * 8;
  return true;
}

size_t wide_comm_bytes(int L) { return 256 + (size_t)wd::NG * wd::group_words(L) * 8; }

hipError_t wide_setup(size_t lds, int *coresident_ok) {
  hipError_t e = hipFuncSetAttribute((const void *)wd::wide_step_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds);
  if (e != hipSuccess) return e;
  int per_cu = 0, dev = 0, cus = 0;
  if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, wd::wide_step_kernel, wd::NT + wd::NTL, lds)) !=
      hipSuccess)
    return e;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  *coresident_ok = (long long)per_cu * cus >= (long long)wd::NG * wd::NBG;
  return hipSuccess;
}

hipError_t launch_wide_step(const StepArgs &a, const WideArgs &g, size_t lds, hipStream_t s) {
  hipLaunchKernelGGL(wd::wide_step_kernel, dim3(wd::NG * wd::NBG), dim3(wd::NT + wd::NTL), lds, s, a, g);
  return hipGetLastError();
}

hipError_t launch_wide_pack(const void *embed, const float *embed_b, const void *const *conv,
                            const float *const *conv_b, const void *out, const float *out_b, int L, const WideArgs &g,
                            hipStream_t s) {
  const int C = kWideC, Q = 256;
  for (int l = 0; l < L; ++l) {
    hipLaunchKernelGGL(wd::wide_pack_layer_kernel, dim3((wd::NBG * wd::CPL * wd::CHUNK + 255) / 256), dim3(256), 0, s,
                       (const float *)conv[l], l, (float4 *)g.wl);
    hipLaunchKernelGGL(wd::wide_vec_kernel, dim3((C + 255) / 256), dim3(256), 0, s, conv_b ? conv_b[l] : nullptr,
                       (float *)g.convb + (size_t)l * C, C);
  }
  hipLaunchKernelGGL(wd::wide_pack_out_kernel, dim3((wd::NBG * wd::CHUNK + 255) / 256), dim3(256), 0, s,
                     (const float *)out, (float4 *)g.wo);
  hipLaunchKernelGGL(wd::wide_transpose_kernel, dim3((C * Q + 255) / 256), dim3(256), 0, s, (const float *)embed,
                     (float *)g.embT, C, Q);
  hipLaunchKernelGGL(wd::wide_vec_kernel, dim3((C + 255) / 256), dim3(256), 0, s, embed_b, (float *)g.embb, C);
  hipLaunchKernelGGL(wd::wide_vec_kernel, dim3(1), dim3(256), 0, s, out_b, (float *)g.outb, Q);
  return hipGetLastError();
}

}  // namespace fwg
