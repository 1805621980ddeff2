// Split MFMA step kernel for gated stacks with bf16 operands, R = 64 residual channels,
// S = H = 512 skip/head channels and 256 classes (gfx950, v_mfma_f32_16x16x32_bf16, fp32
// accumulation).  Same model shape and results as the MFMA step kernel of fwg_mfma.hip.
//
// The work of one step of a block of 16 streams is split over 2 + kSpHelpers blocks of the same
// launch (a group):
//  - the chain block runs what lies on the layer-to-layer dependency chain: per layer the pop, the
//    dilated width-2 product, the gate, the residual 1x1 and the push (paper Section 2.2); the
//    sample the class block returns is the next step's input (Section 1);
//  - helper h owns 64 of the 512 channels of the skip sum and of the head's hidden layer.  Per
//    step it accumulates sum_l W_skip^l z^l + b for its skip channels from the gate outputs z^l
//    the chain block publishes, then (after gathering the whole relu(skip sum) from the group) its
//    rows of the first head 1x1.  Its head weights, and up to 32 layers its skip weights, stay in
//    its waves' registers for the launch;
//  - the class block gathers the whole hidden layer, computes all 256 logits (the output 1x1 is in
//    its waves' registers for the launch), draws the softmax / inverse-CDF sample of every stream
//    and returns the samples to the chain block (forced modes: writes the logits out and returns a
//    mark that the step's head is done).
// No later layer reads a skip product and the head follows the last layer, so the chain block
// streams only the 40 KB of conv and residual weights per layer from the L2, which then also keeps
// the exchange words that are rewritten every step; in the single-block kernel every
// block that owns streams streams all 4 MB of weights once per step, which bounds its step.
//
// Hand-offs between blocks are 8-byte words of (32-bit payload, 32-bit tag), loaded with relaxed
// device-scope atomics.  A word is fresh once its tag equals the step's tag, so no fence or flag
// has to order the payload.  Tags are never reused between two zero fills of the exchange buffers:
// the host passes each launch a tag base above every tag written since the last fill (the launch
// handshake uses base + 1, step s base + 2 + s), so a handle's exchange buffers are zeroed only
// before its first launch and when the 32-bit tags would wrap, not before every launch.  The blocks of a group compare their XCD ids at launch: when they share one,
// and so its L2, the words are stored with workgroup-scope stores, which complete in that L2;
// otherwise with device-scope stores, which write through to memory and whose slow completion holds
// up every later memory wait of the storing wave.  Each load instruction of a poll reads
// consecutive words across the polling lanes.  Every wait is bounded: a wait that runs out sets
// the launch's mark (base + 1) in the abort word, which ends every other wait of that launch and of
// no later one (the results are then invalid, and a sticky
// word lets the host report it); every wave keeps executing its straight-line program, so the grid
// always drains.
//
// Chain block: 8 waves, A = waves 0..3 and B = waves 4..7, A and B of pair p share SIMD p.
//  - wave A (p): the current-input half of the dilated product (W_e x) for tanh tile p and
//    sigmoid tile p, plus W_r v + b from LDS, the gate, the residual 1x1 for channel tile p;
//  - wave B (p): W_r v + b of the next layer (v = the popped state, known early) and the queue
//    pops of stream rows 4p..4p+3, issued five layers before they land in LDS; between the layer's
//    two barriers, while A runs the residual product, the publication of z^l to the helpers and the
//    push of the layer input.
// Every chain wave streams its own pre-packed weight fragments from L2 through a ring of registers,
// 18 fragments (three layers) for A and 24 (six layers) for B, whose loads also queue behind the
// queue reads; a slot is refilled with the fragment one ring length ahead as soon as it is
// consumed.  The layer loop is unrolled by six layers so every ring slot is a fixed register.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "fwg_internal.h"
#include "fwg_mfma_dev.h"
#include "fwg_xchg.h"

namespace fwg {
namespace sp {

using namespace mfd;
using namespace xg;

constexpr int R = kMfR, S = kMfS, H = kMfH, Q = 256, ROWS = kMfRows;
constexpr int NT = kMfThreads, NW = kMfWaves;
constexpr int NHLP = kSpHelpers;          // helpers per group
// skip and hidden slices of a helper; classes of a class-block wave (one per helper index)
constexpr int SL = S / NHLP, HL = H / NHLP, QL = Q / NHLP;
constexpr int PX = R + 8;   // 64-channel activation rows (bf16)
constexpr int PS = S + 8;   // 512-channel activation rows (bf16)
constexpr int PL = Q + 4;   // fp32 logits rows
constexpr int PP = 20;      // fp32 partial-tile rows
constexpr int PH = SL + 4;  // fp32 helper skip-partial rows
constexpr int ZST = R / 2 + 4;  // staged z^l rows of a helper wave (32-bit words)
constexpr int FA = kSpFA, FB = kSpFB, FS = kSpFS;
// fragments of a helper's first-1x1 slice and of a class-block wave's output-1x1 slice
constexpr int FW1 = (HL / 16) * (S / 32), FW2 = (QL / 16) * (H / 32);
constexpr int DA = 3 * FA, DB = 6 * FB;  // ring depths (fragments) of chain waves A and B
constexpr int KCH = 64;                  // steps per chunk of per-step inputs staged in LDS
static_assert(ZST <= PH && ZST % 4 == 0, "a wave's staged z^l rows fit its partial-sum area, 16-byte aligned");
static_assert(SL == 64 && FS == 8 && HL == 64 && QL == 32 && NHLP == NW,
              "helper slices of 4 skip and 4 hidden tiles; 2 class tiles per class-block wave");

struct ChainLds {
  uint16_t vbuf[3][ROWS * PX];     // popped queue rows, by layer index mod 3
  uint16_t xbuf[2][ROWS * PX];     // layer inputs x^l, by layer parity
  uint16_t zbuf[2][ROWS * PX];     // gate outputs z^l, by layer parity
  float pbuf[2][4][2][ROWS * PP];  // W_r v + b of a layer: [layer parity][tile][tanh / sigmoid]
  uint16_t embT[Q * R];            // embedding table, [class][channel]
  int in[ROWS][KCH];               // forced inputs (forced modes)
  int ins[ROWS + NHLP + 1];        // next inputs, then (at launch) the helpers' and the class block's XCD ids
  // followed by the per-layer tables: slot[L], dil[L], rbase[L], qoff[2][L] (32-bit), then the fp32
  // bias block
};
struct HelperLds {
  union {
    float part[NW][ROWS * PH];  // per-wave partial skip sums of the slice
    uint16_t act[ROWS * PS];    // gathered relu(skip sum), then relu(hidden)
  } u;
  float pw[4][ROWS * PP];       // k-split partial tiles of the first head product
  float bias[SL + HL];          // the slice's summed skip biases and hidden biases
  int local;                    // the group's mode from the launch handshake
};
struct ClassLds {
  uint16_t act[ROWS * PS];  // gathered relu(hidden)
  float lg[ROWS * PL];      // logits
  float u[ROWS][KCH];       // uniforms (generation)
  float bias[Q];            // output biases
  int local;                // the group's mode from the launch handshake
};

__host__ __device__ constexpr size_t chain_fixed_bytes() { return (sizeof(ChainLds) + 15) & ~size_t(15); }
__host__ __device__ inline size_t dyn_bias_offset(int L) { return ((size_t)L * 20 + 15) & ~size_t(15); }

// Fragment stream geometry (1 KB fragments): chain wave A p, chain wave B p, helper (h, wave w)
// skip stream, then the helpers' head slices.
__host__ __device__ inline int len_a(int L) { return FA * L; }
__host__ __device__ inline int len_b(int L) { return FB * L; }
__host__ __device__ inline int helper_layers(int L) { return (L + NW - 1) / NW; }
__host__ __device__ inline size_t base_a(int L, int p) { return (size_t)p * len_a(L); }
__host__ __device__ inline size_t base_b(int L, int p) { return 4 * (size_t)len_a(L) + (size_t)p * len_b(L); }
__host__ __device__ inline size_t base_h(int L, int h, int w) {
  return 4 * (size_t)len_a(L) + 4 * (size_t)len_b(L) + (size_t)(NW * h + w) * helper_layers(L) * FS;
}
__host__ __device__ inline size_t base_w1(int L, int h) { return base_h(L, NHLP, 0) + (size_t)h * FW1; }
__host__ __device__ inline size_t base_w2(int L, int h) { return base_w1(L, NHLP) + (size_t)h * FW2; }
__host__ __device__ inline size_t frag_count(int L) { return base_w2(L, NHLP); }

// Exchange buffers: abort word, then per group: z^l words [L][512]; relu(skip sum) and relu(hidden)
// words [16 streams][256] each; the step's samples (forced modes: step-done marks) [16] in a
// 256-byte line of their own; the launch handshake (slot h: XCD of helper h; slot NHLP: XCD of the
// class block; slot NHLP + 1: the group's mode).  A device-scope load is served by the reader's own L2 when that L2 holds
// the line from the reader's own store, so no block ever reads a line another block writes after
// it has written to that line itself: every helper slice of a word array spans whole 256-byte
// lines, and every handshake word has a 256-byte slot of its own.
constexpr int ZWORDS = ROWS * R / 2, XWORDS = ROWS * 256, SWORDS = 32, HSLOT = 32, HWORDS = (NHLP + 2) * HSLOT;
static_assert((SL / 2) % 32 == 0 && (HL / 2) % 32 == 0 && SWORDS == 32 && HSLOT == 32,
              "helper slices, the sample line and handshake slots span whole 256-byte lines");
__host__ __device__ inline size_t group_words(int L) { return (size_t)L * ZWORDS + 2 * (size_t)XWORDS + SWORDS + HWORDS; }
__host__ __device__ inline u64 *comm_group(void *comm, int L, int blk) {
  return (u64 *)((char *)comm + 256) + (size_t)blk * group_words(L);
}
__host__ __device__ inline u64 *comm_z(void *comm, int L, int blk) { return comm_group(comm, L, blk); }
__host__ __device__ inline u64 *comm_s(void *comm, int L, int blk) { return comm_group(comm, L, blk) + (size_t)L * ZWORDS; }
__host__ __device__ inline u64 *comm_hid(void *comm, int L, int blk) { return comm_s(comm, L, blk) + XWORDS; }
__host__ __device__ inline u64 *comm_smp(void *comm, int L, int blk) { return comm_hid(comm, L, blk) + XWORDS; }
__host__ __device__ inline u64 *comm_hs(void *comm, int L, int blk) { return comm_smp(comm, L, blk) + SWORDS; }
// Tags of a launch: the handshake words and the abort mark use base + 1, step s uses base + 2 + s.
__device__ __forceinline__ uint32_t launch_mark(const StepArgs &a) { return a.sp_tag0 + 1u; }
__device__ __forceinline__ uint32_t step_tag(const StepArgs &a, long long step) {
  return a.sp_tag0 + 2u + (uint32_t)step;
}

// ---------------------------------------------------------------------------
// Chain block

struct Ctx {
  const StepArgs *a;
  ChainLds *s;
  int *slot, *dil;
  uint32_t *rbase;  // byte offset of each layer's queue in the queue region
  uint32_t *qoff;   // [2][L]: byte offset of the rows of the current slot (0) and the next step's (1)
  char *ring;       // queue region
  uint32_t rowb;    // byte offset of this lane's 16-byte chunk of a queue row (wave B)
  const float *conv_b, *res_b, *emb_b;
  const char *fw;   // this wave's fragment stream (wave-uniform)
  const char *fend; // its end: the stream holds one step and is read cyclically
  const char *nxt;  // next fragment the ring loads
  int wvoff;        // 16 * lane
  u64 *zp;          // this group's z^0 words (layer l at + l * ZWORDS)
  const u64 *smp;   // this group's sample words
  uint32_t *abort_word, *sticky;
  uint32_t mark;    // this launch's abort mark
  bool local;       // the helpers and the class block share this XCD: workgroup-scope stores suffice
  int L, w, p, lane, n, q, b0, nrows, blk;
};

__device__ __forceinline__ u32x4 frag_at(const Ctx &c, int pos) {
  return *(const u32x4 *)(c.fw + (size_t)pos * 1024 + c.wvoff);
}
// Slot `f` of ring W has just been consumed: load the stream's next fragment into it (the ring is a
// FIFO over the cyclic stream).  The scheduling barriers keep the load after the MFMA that still
// reads the slot's old contents.
template <int D>
__device__ __forceinline__ void refill(Ctx &c, u32x4 (&W)[D], int f) {
  __builtin_amdgcn_sched_barrier(0);
  if (c.nxt == c.fend) c.nxt = c.fw;
  W[f] = *(const u32x4 *)(c.nxt + c.wvoff);
  c.nxt += 1024;
  __builtin_amdgcn_sched_barrier(0);
}

// Queue rows moved by wave B of pair p: stream rows 4p..4p+3, lane l handling row 4p + (l%32)/8
// and 16-byte chunk l%8 (lanes 32..63 mirror lanes 0..31 on loads and skip the stores).  The lane
// that pushes a row chunk is the lane that later pops it, so program order keeps every pop after
// the push it must see.
// Pop of layer l for the step `ahead` (0 or 1) steps after the one the offset table describes.
__device__ __forceinline__ u32x4 pop_issue(const Ctx &c, int l, int ahead) {
  return *(const u32x4 *)(c.ring + (c.qoff[ahead * c.L + l] + c.rowb));
}
// The same load from an offset read from the table earlier.
__device__ __forceinline__ u32x4 pop_issue_at(const Ctx &c, uint32_t off) {
  return *(const u32x4 *)(c.ring + (off + c.rowb));
}
__device__ __forceinline__ void pop_land(const Ctx &c, int buf, u32x4 v) {
  if (c.lane < 32) {
    const int r = 4 * c.p + (c.lane >> 3);
    *(u32x4 *)(c.s->vbuf[buf] + r * PX + 8 * (c.lane & 7)) = v;
  }
}
// Between the layer's barriers: z^l of stream rows 4p..4p+3 to the helpers (lane l covers row
// 4p + l/16, channels 4(l%16)..+3, as two words of two bf16 each; word index = row * 32 +
// channel / 2), and the push of layer l (its input x^l replaces the slot popped for this step).
// All LDS reads are issued before either store, so the wave waits for LDS once.
__device__ __forceinline__ void publish_and_push(const Ctx &c, int l, uint32_t tag) {
  const int rz = 4 * c.p + (c.lane >> 4), cp = 2 * (c.lane & 15);
  const int rx = 4 * c.p + ((c.lane & 31) >> 3);
  const u32x2 zv = *(const u32x2 *)(c.s->zbuf[l & 1] + rz * PX + 2 * cp);
  const u32x4 xv = *(const u32x4 *)(c.s->xbuf[l & 1] + rx * PX + 8 * (c.lane & 7));
  const uint32_t off = c.qoff[l];
  __builtin_amdgcn_sched_barrier(0);
  put_words2(c.zp + (size_t)l * ZWORDS + rz * (R / 2) + cp, zv.x, zv.y, tag, c.local);
  if (c.lane < 32) *(u32x4 *)(c.ring + (off + c.rowb)) = xv;
}

// W_r v + b of layer ln from the popped rows in vbuf[vb3] and ring slots f0..f0+3 (tanh tile p
// k-steps 0,1, sigmoid tile p k-steps 0,1), into pbuf[par].
template <int D>
__device__ __forceinline__ void recurrent_half(const Ctx &c, int ln, int vb3, int par, const u32x4 (&W)[D], int f0) {
  ChainLds &s = *c.s;
  const uint16_t *vb = s.vbuf[vb3] + c.n * PX;
  const float *cb = c.conv_b + ln * 2 * R;
  // the biases (C operands) first, so the two products interleave (the LDS reads land in order)
  f32x4 pt = ldsf4(cb + 16 * c.p + 4 * c.q), pg = ldsf4(cb + R + 16 * c.p + 4 * c.q);
  const u32x4 bv0 = lds16(vb + 8 * c.q), bv1 = lds16(vb + 32 + 8 * c.q);
  // the four LDS reads in flight together (one wait), not one round trip per product
  __builtin_amdgcn_sched_barrier(0);
  pt = mfma(W[f0 + 0], bv0, pt);
  pg = mfma(W[f0 + 2], bv0, pg);
  pt = mfma(W[f0 + 1], bv1, pt);
  pg = mfma(W[f0 + 3], bv1, pg);
  stf4(s.pbuf[par][c.p][0] + c.n * PP + 4 * c.q, pt);
  stf4(s.pbuf[par][c.p][1] + c.n * PP + 4 * c.q, pg);
}

// Forced inputs of steps [s0, s0 + KCH) into LDS (forced modes; every thread): the input that
// follows each step.
__device__ __forceinline__ void stage_inputs(const Ctx &c, long long s0) {
  const StepArgs &a = *c.a;
  ChainLds &s = *c.s;
  static_assert((ROWS * KCH) % NT == 0, "the chunk divides evenly over the threads");
#pragma unroll
  for (int e = 0; e < ROWS * KCH / NT; ++e) {
    const int idx = (int)threadIdx.x + e * NT;
    const int r = idx / KCH, j = idx % KCH;
    const long long nx = s0 + j + forced_shift(a.mode);
    int v = 0;
    if (r < c.nrows && nx < a.n_steps) v = a.inputs[(long long)(c.b0 + r) * a.n_steps + nx];
    s.in[r][j] = v;
  }
}

// Layer l on wave A, ring slots PHS..PHS+5 (x-half of tanh/sigmoid tile p, residual tile p).
template <int PHS>
__device__ __forceinline__ void a_layer(Ctx &c, int l, u32x4 (&W)[DA], f32x4 &xres) {
  ChainLds &s = *c.s;
  const int n = c.n, q = c.q, p = c.p;
  const int par = l & 1;
  // W_r v + b first: the LDS reads land in order, and with both C operands in before the layer input
  // the tanh and sigmoid products interleave instead of running as two dependent pairs
  f32x4 af = ldsf4(s.pbuf[par][p][0] + n * PP + 4 * q);
  f32x4 ag = ldsf4(s.pbuf[par][p][1] + n * PP + 4 * q);
  u32x4 bx0, bx1;
  if (l == 0) {
    // embedding (current input x^0): row gather of the transposed 1x1 convolution plus bias
    const uint16_t *e = s.embT + s.ins[n] * R;
    const u32x4 r0 = lds16(e + 8 * q), r1 = lds16(e + 32 + 8 * q);
    const float *eb = c.emb_b;
    auto cvt = [&](u32x4 raw, int k0) {
      u32x4 pk;
#pragma unroll
      for (int j = 0; j < 4; ++j) pk[j] = pack2(bf_lo(raw[j]) + eb[k0 + 2 * j], bf_hi(raw[j]) + eb[k0 + 2 * j + 1]);
      return pk;
    };
    bx0 = cvt(r0, 8 * q);
    bx1 = cvt(r1, 32 + 8 * q);
    const int ch = 16 * p + 4 * q;
    const u32x2 raw = *(const u32x2 *)(e + ch);
    xres = f32x4{bf_lo(raw.x) + eb[ch], bf_hi(raw.x) + eb[ch + 1], bf_lo(raw.y) + eb[ch + 2], bf_hi(raw.y) + eb[ch + 3]};
    lds8(s.xbuf[0] + n * PX + ch, pack4(xres));
  } else {
    const uint16_t *xb = s.xbuf[par] + n * PX;
    bx0 = lds16(xb + 8 * q);
    bx1 = lds16(xb + 32 + 8 * q);
  }
  af = mfma(W[PHS + 0], bx0, af);
  ag = mfma(W[PHS + 2], bx0, ag);
  af = mfma(W[PHS + 1], bx1, af);
  ag = mfma(W[PHS + 3], bx1, ag);
#pragma unroll
  for (int f = 0; f < 4; ++f) refill(c, W, PHS + f);
  // x^l + b_res while the gate runs, so the residual product starts as soon as z^l lands
  f32x4 xr = xres + ldsf4(c.res_b + l * R + 16 * p + 4 * q);
  f32x4 z;
#pragma unroll
  for (int i = 0; i < 4; ++i) z[i] = gate(af[i], ag[i]);
  lds8(s.zbuf[par] + n * PX + 16 * p + 4 * q, pack4(z));
  __syncthreads();
  const uint16_t *zb = s.zbuf[par] + n * PX;
  const u32x4 bz0 = lds16(zb + 8 * q), bz1 = lds16(zb + 32 + 8 * q);
  xr = mfma(W[PHS + 4], bz0, xr);
  xr = mfma(W[PHS + 5], bz1, xr);
#pragma unroll
  for (int f = 4; f < FA; ++f) refill(c, W, PHS + f);
  xres = xr;
  lds8(s.xbuf[par ^ 1] + n * PX + 16 * p + 4 * q, pack4(xr));
  __syncthreads();
}

// Layer l on wave B, ring slots PBS..PBS+3 (W_r of the next layer), pop registers rotated by
// G6 = l mod 6 (L is a multiple of 6, so this is also the global layer index mod 6): the pop of
// global layer index g sits in P[g mod 6] from its issue, five layers ahead of landing, until it
// lands in vbuf[g mod 3] before the first barrier of layer g - 3, four block barriers before its
// product.
template <int PBS, int G6>
__device__ __forceinline__ void b_layer(Ctx &c, int l, u32x4 (&W)[DB], u32x4 (&P)[6], uint32_t tag) {
  const int L = c.L;
  const int ln = l + 1 < L ? l + 1 : 0;
  // queue offset of the pop issued below, read with the product's LDS reads
  const int j = l + 8 < L ? l + 8 : l + 8 - L;
  const uint32_t joff = c.qoff[(l + 8 < L ? 0 : L) + j];
  recurrent_half(c, ln, (G6 + 1) % 3, (l + 1) & 1, W, PBS);
#pragma unroll
  for (int f = 0; f < FB; ++f) refill(c, W, PBS + f);
  // the pop of layer l + 3 into LDS (its buffer was last read before the previous layer's first
  // barrier) and the pop of layer l + 8 issued
  pop_land(c, G6 % 3, P[(G6 + 3) % 6]);
  P[(G6 + 2) % 6] = pop_issue_at(c, joff);
  __syncthreads();
  // while wave A runs the residual product: the layer's gate output to the helpers and its input
  // into its queue
  publish_and_push(c, l, tag);
  __syncthreads();
}

// End of step `step` on every chain wave: the slot advance, then the class block's word for each
// stream (the sample in generation, which becomes the next input; a step-done mark in forced modes,
// where the next input is the forced one).  Waiting for it in every mode also keeps the chain from
// rewriting the z^l words before the helpers have read this step's.  One barrier (two when forced
// inputs are staged).
__device__ __forceinline__ void finish_step(Ctx &c, long long step) {
  ChainLds &s = *c.s;
  const StepArgs &a = *c.a;
  const int tid = threadIdx.x;
  if (a.mode != MODE_GENERATE && step % KCH == 0) {
    stage_inputs(c, step);
    __syncthreads();
  }
  // no wave reads the offset table between the last layer's push and the next step's first layer
  for (int l = tid; l < c.L; l += NT) {
    const int nx = c.slot[l] + 1 == c.dil[l] ? 0 : c.slot[l] + 1;
    const int nn = nx + 1 == c.dil[l] ? 0 : nx + 1;
    c.slot[l] = nx;
    c.qoff[l] = c.qoff[c.L + l];
    c.qoff[c.L + l] = c.rbase[l] + (uint32_t)nn * (uint32_t)(a.bmax * R * 2);
  }
  if (tid < ROWS) {
    uint32_t v[1];
    wait_words<1>(c.smp + tid, step_tag(a, step), v, c.abort_word, c.sticky, c.mark);
    if (a.mode == MODE_GENERATE) {
      s.ins[tid] = (int)v[0];
    } else if (tid < c.nrows && step + forced_shift(a.mode) < a.n_steps) {
      s.ins[tid] = s.in[tid][step % KCH];
    }
  }
  __syncthreads();
}

// Launch handshake, second half (after the barrier that follows wave A's poll of the XCD ids):
// whether the whole group shares this block's XCD, which decides the scope of every word the block
// stores; thread 0 publishes it to the group.
__device__ __forceinline__ void set_mode(Ctx &c) {
  bool local = true;
  for (int h = 0; h < NHLP + 1; ++h) local = local && (uint32_t)c.s->ins[ROWS + h] == xcd_id();
  c.local = local;
  if (threadIdx.x == 0) put_word(comm_hs(c.a->sp_comm, c.L, c.blk) + HSLOT * (NHLP + 1), local ? 1u : 0u, c.mark, false);
}

__device__ __forceinline__ void a_role(Ctx &c) {
  const int L = c.L;
  c.fw = (const char *)c.a->mf_frags + base_a(L, c.p) * 1024;
  c.fend = c.fw + (size_t)len_a(L) * 1024;
  u32x4 W[DA];
#pragma unroll
  for (int f = 0; f < DA; ++f) W[f] = frag_at(c, f);
  c.nxt = c.fw + DA * 1024;
  f32x4 xres = f32x4{0.f, 0.f, 0.f, 0.f};
  // launch handshake, first half: the XCD ids of the group's other blocks (published at their start)
  const int tid = threadIdx.x;
  if (tid < NHLP + 1) {
    uint32_t v[1];
    wait_words<1>(comm_hs(c.a->sp_comm, L, c.blk) + HSLOT * tid, c.mark, v, c.abort_word, c.sticky, c.mark);
    c.s->ins[ROWS + tid] = (int)v[0];
  }
  __syncthreads();  // the popped rows of layers 0..2 and the XCD ids are in LDS
  set_mode(c);
  __syncthreads();  // W_r v + b of layer 0 is in LDS
  for (long long step = 0; step < c.a->n_steps; ++step) {
    for (int l = 0; l < L; l += 6) {
      a_layer<0>(c, l, W, xres);
      a_layer<FA>(c, l + 1, W, xres);
      a_layer<2 * FA>(c, l + 2, W, xres);
      a_layer<0>(c, l + 3, W, xres);
      a_layer<FA>(c, l + 4, W, xres);
      a_layer<2 * FA>(c, l + 5, W, xres);
    }
    finish_step(c, step);
  }
}

__device__ __forceinline__ void b_role(Ctx &c) {
  const int L = c.L;
  c.fw = (const char *)c.a->mf_frags + base_b(L, c.p) * 1024;
  c.fend = c.fw + (size_t)len_b(L) * 1024;
  u32x4 W[DB], P[6];
  // layers 0..2 of step 0 land now and layers 3..7 are issued; layer 0's W_r v + b comes from its
  // stream stage L - 1 (all of these loads in flight together)
  const u32x4 v0 = pop_issue(c, 0, 0), v1 = pop_issue(c, 1, 0), v2 = pop_issue(c, 2, 0);
#pragma unroll
  for (int g = 3; g < 8; ++g) P[g % 6] = pop_issue(c, g, 0);
#pragma unroll
  for (int f = 0; f < FB; ++f) W[f] = frag_at(c, FB * (L - 1) + f);
  pop_land(c, 0, v0);
  pop_land(c, 1, v1);
  pop_land(c, 2, v2);
  __syncthreads();  // the popped rows of layers 0..2 and the XCD ids are in LDS
  set_mode(c);
  recurrent_half(c, 0, 0, 0, W, 0);
#pragma unroll
  for (int f = 0; f < DB; ++f) W[f] = frag_at(c, f);
  c.nxt = c.fw + DB * 1024;
  __syncthreads();
  for (long long step = 0; step < c.a->n_steps; ++step) {
    const uint32_t tag = step_tag(*c.a, step);
    for (int l = 0; l < L; l += 6) {
      b_layer<0, 0>(c, l, W, P, tag);
      b_layer<FB, 1>(c, l + 1, W, P, tag);
      b_layer<2 * FB, 2>(c, l + 2, W, P, tag);
      b_layer<3 * FB, 3>(c, l + 3, W, P, tag);
      b_layer<4 * FB, 4>(c, l + 4, W, P, tag);
      b_layer<5 * FB, 5>(c, l + 5, W, P, tag);
    }
    finish_step(c, step);
  }
}

__device__ __forceinline__ void chain_block(const StepArgs &a, char *lds_raw, int blk) {
  ChainLds &s = *(ChainLds *)lds_raw;
  const int tid = threadIdx.x, L = a.L;
  char *dyn = lds_raw + chain_fixed_bytes();
  int *slot = (int *)dyn;
  int *dil = slot + L;
  uint32_t *rbase = (uint32_t *)(dil + L);
  uint32_t *qoff = rbase + L;
  float *bias = (float *)(dyn + dyn_bias_offset(L));  // conv_b [L][2R], res_b [L][R], emb_b [R]

  Ctx c;
  c.a = &a;
  c.s = &s;
  c.slot = slot;
  c.dil = dil;
  c.rbase = rbase;
  c.qoff = qoff;
  c.ring = (char *)a.ring;
  c.conv_b = bias;
  c.res_b = c.conv_b + L * 2 * R;
  c.emb_b = c.res_b + L * R;
  c.L = L;
  c.w = __builtin_amdgcn_readfirstlane(tid >> 6);
  c.p = c.w & 3;
  c.lane = tid & 63;
  c.n = c.lane & 15;
  c.q = c.lane >> 4;
  c.blk = blk;
  c.b0 = blk * ROWS;
  c.nrows = min(ROWS, a.batch - c.b0);
  c.wvoff = 16 * c.lane;
  c.rowb = (uint32_t)(((c.b0 + 4 * c.p + ((c.lane & 31) >> 3)) * R + 8 * (c.lane & 7)) * 2);
  c.zp = comm_z(a.sp_comm, L, blk);
  c.smp = comm_smp(a.sp_comm, L, blk);
  c.abort_word = (uint32_t *)a.sp_comm;
  c.sticky = a.sp_sticky;
  c.mark = launch_mark(a);

  // What the block keeps in LDS for the launch: the embedding table, the conv and residual biases,
  // the embedding bias (the last R floats of the bias block), the per-layer queue tables and the
  // first inputs.  Every thread issues all of its loads before its first LDS store, so the launch
  // waits for one memory round trip here instead of one per loop iteration (a 30-layer launch
  // spent ~5 us in these loops).
  {
    constexpr int NE = Q * R / 8 / NT;  // 16-byte pieces of the embedding table per thread
    static_assert(Q * R / 8 == NE * NT, "the embedding table splits evenly over the block");
    constexpr int NB4 = 4;              // 16-byte pieces of the bias block per thread in the first batch
    const u32x4 *esrc = (const u32x4 *)a.mf_embT;
    const u32x4 *bsrc = (const u32x4 *)a.mf_bias;  // L * 3 * R floats, a multiple of 4
    const int nb4 = L * 3 * R / 4;
    u32x4 ev[NE];
#pragma unroll
    for (int k = 0; k < NE; ++k) ev[k] = esrc[tid + k * NT];
    u32x4 bv[NB4];
#pragma unroll
    for (int k = 0; k < NB4; ++k)
      if (tid + k * NT < nb4) bv[k] = bsrc[tid + k * NT];
    const float eb = tid < R ? a.mf_bias[L * 3 * R + S + H + Q + tid] : 0.f;
    long long roff = 0;  // the layer's queue offset and dilation (first batch of layers)
    int ldil = 1;
    if (tid < L) {
      roff = a.layers[tid].ring_off;
      ldil = a.layers[tid].dil;
    }
    int in0 = 0;
    if (tid < c.nrows) in0 = a.mode == MODE_TEACHER ? a.inputs[(long long)(c.b0 + tid) * a.n_steps] : a.last[c.b0 + tid];
#pragma unroll
    for (int k = 0; k < NE; ++k) ((u32x4 *)s.embT)[tid + k * NT] = ev[k];
#pragma unroll
    for (int k = 0; k < NB4; ++k)
      if (tid + k * NT < nb4) ((u32x4 *)bias)[tid + k * NT] = bv[k];
    for (int i = tid + NB4 * NT; i < nb4; i += NT) ((u32x4 *)bias)[i] = bsrc[i];  // more than 42 layers
    if (tid < R) bias[L * 3 * R + tid] = eb;
    const uint32_t slot_bytes = (uint32_t)(a.bmax * R * 2);
    for (int l = tid; l < L; l += NT) {
      if (l >= NT) {  // more than NT layers
        roff = a.layers[l].ring_off;
        ldil = a.layers[l].dil;
      }
      const int s0 = (int)(a.t0 % (long long)ldil), s1 = s0 + 1 == ldil ? 0 : s0 + 1;
      rbase[l] = (uint32_t)(roff * 2);
      dil[l] = ldil;
      slot[l] = s0;
      qoff[l] = rbase[l] + (uint32_t)s0 * slot_bytes;
      qoff[L + l] = rbase[l] + (uint32_t)s1 * slot_bytes;
    }
    if (tid < ROWS) s.ins[tid] = in0;
  }
  __syncthreads();  // the tables are in LDS
  // The launch handshake (the helpers' and the class block's XCD ids, then the group's mode) runs
  // inside the roles' first loads: wave A polls the ids while its weight loads and wave B's first
  // pops are in flight.
  if (c.w < 4) a_role(c);
  else b_role(c);
  if (a.mode != MODE_TEACHER && tid < c.nrows) a.last[c.b0 + tid] = s.ins[tid];
}

// ---------------------------------------------------------------------------
// Helper h of group blk.  Per step:
//  1. skip: wave w takes layers w, w + 8, ...; for each it waits for z^l and accumulates the 4 tiles
//     x 2 k-steps of its 64 skip channels (weights streamed from L2, one layer ahead); the eight
//     waves' partials meet in LDS, get the summed skip biases, relu and bf16 rounding, and go out
//     as words;
//  2. hidden: gather relu(skip sum) of all 512 channels; 64 hidden rows = 4 tiles, each over two
//     waves that split the 16 k-steps; + bias, relu, bf16, out as words to the class block.

// Gather 16 x 512 bf16 activations (4096 words of two channels each) into act: word i = e NT + t
// holds stream i / 256, channels 2 (i % 256) and 2 (i % 256) + 1.
__device__ __forceinline__ void gather_act(uint16_t *act, const u64 *src, uint32_t tag, uint32_t *abort_word,
                                           uint32_t *sticky, uint32_t mark) {
  const int tid = threadIdx.x;
  uint32_t v[8];
  wait_words<8, NT>(src + tid, tag, v, abort_word, sticky, mark);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int i = e * NT + tid;
    ((uint32_t *)(act + (i >> 8) * PS))[i & 255] = v[e];
  }
}

// Values of a helper wave for its step loop (plain values and pointers).
struct HelperCtx {
  const StepArgs *a;
  HelperLds *s;
  const char *fw;  // this wave's skip fragment stream (layers w, w + 8, ...)
  const u64 *zb;
  u64 *sw, *hw;
  uint32_t *abort_word;
  uint32_t mark;  // this launch's abort mark
  int tid, w, lane, n, q, nl, wvoff, h;
  bool local;
};

// z^l (512 words) as this wave's two B operand rows: lane takes words e 64 + lane (stream
// 2e + lane / 32, channel pair lane % 32) and turns them into rows (stream n, channels 8q..8q+7 for
// k-step 0, 32 + 8q.. for k-step 1) through its wave's partial-sum area, which the wave next writes
// after its last layer of the step (LDS operations of one wave complete in order).
__device__ __forceinline__ void z_operands(const HelperCtx &c, int l, uint32_t tag, u32x4 &b0, u32x4 &b1) {
  uint32_t zv[8];
  wait_words<8, 64>(c.zb + (size_t)l * ZWORDS + c.lane, tag, zv, c.abort_word, c.a->sp_sticky, c.mark);
  uint32_t *stg = (uint32_t *)c.s->u.part[c.w];
#pragma unroll
  for (int e = 0; e < 8; ++e) stg[(2 * e + (c.lane >> 5)) * ZST + (c.lane & 31)] = zv[e];
  b0 = *(const u32x4 *)(stg + c.n * ZST + 4 * c.q);
  b1 = *(const u32x4 *)(stg + c.n * ZST + 16 + 4 * c.q);
}

// Skip fragments kept in a helper wave's registers for the whole launch when it has at most this
// many layers (L <= 32): streamed every step they filled most of the XCD's L2, and the exchange
// words, rewritten every step, were evicted to memory.
constexpr int NRES = 4;

// The helper's step loop.  RES: this wave's skip fragments (at most NRES layers) stay in registers;
// otherwise they stream from L2 through an 8-fragment ring, one layer ahead.
template <bool RES>
__device__ __forceinline__ void helper_steps(const HelperCtx &c, const u32x4 (&hw1)[8]) {
  const StepArgs &a = *c.a;
  HelperLds &s = *c.s;
  const int tid = c.tid, w = c.w, n = c.n, q = c.q, nl = c.nl, wvoff = c.wvoff, h = c.h;
  const float *skip_sum = s.bias, *head_b = s.bias + SL;
  constexpr int NW_ = RES ? NRES : 1;
  u32x4 W[NW_][FS];
  if (RES) {
#pragma unroll
    for (int i = 0; i < NW_; ++i)
#pragma unroll
      for (int f = 0; f < FS; ++f)
        W[i][f] = i < nl ? *(const u32x4 *)(c.fw + (size_t)(i * FS + f) * 1024 + wvoff) : u32x4{0u, 0u, 0u, 0u};
  } else {
#pragma unroll
    for (int f = 0; f < FS; ++f) W[0][f] = *(const u32x4 *)(c.fw + f * 1024 + wvoff);
  }
  const char *nxt = c.fw + (nl > 1 ? FS * 1024 : 0);
  for (long long step = 0; step < a.n_steps; ++step) {
    const uint32_t tag = step_tag(a, step);
    // ---- 1. skip sums of the slice
    f32x4 acc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (RES) {
#pragma unroll
      for (int i = 0; i < NW_; ++i) {
        if (i < nl) {
          u32x4 b0, b1;
          z_operands(c, w + NW * i, tag, b0, b1);
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            acc[j] = mfma(W[i][2 * j], b0, acc[j]);
            acc[j] = mfma(W[i][2 * j + 1], b1, acc[j]);
          }
        }
      }
    } else {
      for (int i = 0; i < nl; ++i) {
        u32x4 b0, b1;
        z_operands(c, w + NW * i, tag, b0, b1);
        if (i + 1 == nl) nxt = c.fw;  // the next layer of this wave is its first of the next step
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          acc[j] = mfma(W[0][2 * j], b0, acc[j]);
          __builtin_amdgcn_sched_barrier(0);
          W[0][2 * j] = *(const u32x4 *)(nxt + wvoff);
          __builtin_amdgcn_sched_barrier(0);
          acc[j] = mfma(W[0][2 * j + 1], b1, acc[j]);
          __builtin_amdgcn_sched_barrier(0);
          W[0][2 * j + 1] = *(const u32x4 *)(nxt + 1024 + wvoff);
          __builtin_amdgcn_sched_barrier(0);
          nxt += 2048;
        }
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) stf4(s.u.part[w] + n * PH + 16 * j + 4 * q, acc[j]);
    __syncthreads();
    if (tid < ROWS * SL / 4) {
      // thread t: stream t/16, slice channels 4 (t%16) .. +3
      const int r = tid >> 4, c4 = 4 * (tid & 15);
      f32x4 v = ldsf4(skip_sum + c4);
#pragma unroll
      for (int ww = 0; ww < NW; ++ww) v += ldsf4(s.u.part[ww] + r * PH + c4);
      const u32x2 pk = pack4(relu4(v));
      put_words2(c.sw + r * 256 + (h * SL + c4) / 2, pk.x, pk.y, tag, c.local);
    }
    __syncthreads();
    // ---- 2. hidden rows of the slice: tile j = w % 4, k-steps 8 (w / 4) .. +7
    gather_act(s.u.act, c.sw, tag, c.abort_word, a.sp_sticky, c.mark);
    __syncthreads();
    {
      const int k0 = 8 * (w >> 2);
      // two accumulators (even and odd k-steps): two dependent chains of four MFMAs, not one of eight
      f32x4 t = f32x4{0.f, 0.f, 0.f, 0.f}, t1 = t;
#pragma unroll
      for (int i = 0; i < 8; i += 2) {
        t = mfma(hw1[i], lds16(s.u.act + n * PS + 32 * (k0 + i) + 8 * q), t);
        t1 = mfma(hw1[i + 1], lds16(s.u.act + n * PS + 32 * (k0 + i + 1) + 8 * q), t1);
      }
      t += t1;
      if (w >= 4) stf4(s.pw[w - 4] + n * PP + 4 * q, t);
      acc[0] = t;
    }
    __syncthreads();
    if (w < 4) {
      const int ch = 16 * w + 4 * q;
      f32x4 t = acc[0] + ldsf4(s.pw[w] + n * PP + 4 * q);
#pragma unroll
      for (int i = 0; i < 4; ++i) t[i] = fmaxf(t[i] + head_b[ch + i], 0.f);
      const u32x2 pk = pack4(t);
      put_words2(c.hw + n * 256 + (h * HL + ch) / 2, pk.x, pk.y, tag, c.local);
    }
  }
}

__device__ __forceinline__ void helper_block(const StepArgs &a, char *lds_raw, int blk, int h) {
  HelperLds &s = *(HelperLds *)lds_raw;
  const int tid = threadIdx.x, L = a.L;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  uint32_t *abort_word = (uint32_t *)a.sp_comm;
  // launch handshake, first half: publish this block's XCD before loading anything, so that the
  // chain block's wait for it overlaps the loads below
  u64 *hs = comm_hs(a.sp_comm, L, blk);
  const uint32_t mark = launch_mark(a);
  if (tid == 0) put_word(hs + HSLOT * h, xcd_id(), mark, false);
  // the slice's biases into LDS for the whole launch
  {
    const float *src = a.mf_bias + L * 3 * R;  // skip sum [S], head [H], out [Q]
    for (int i = tid; i < SL; i += NT) s.bias[i] = src[h * SL + i];
    for (int i = tid; i < HL; i += NT) s.bias[SL + i] = src[S + h * HL + i];
  }
  // this wave's fragments of the first head 1x1 (tile w % 4, k-steps 8 (w / 4) .. +7), in registers
  // for the whole launch
  u32x4 hw1[8];
  {
    const u32x4 *w1 = (const u32x4 *)((const char *)a.mf_frags + base_w1(L, h) * 1024);
#pragma unroll
    for (int i = 0; i < 8; ++i) hw1[i] = w1[((w & 3) * (S / 32) + 8 * (w >> 2) + i) * 64 + lane];
  }
  // launch handshake, second half: learn whether the whole group shares one XCD
  if (tid == 0) {
    uint32_t v[1];
    wait_words<1>(hs + HSLOT * (NHLP + 1), mark, v, abort_word, a.sp_sticky, mark);
    s.local = (int)v[0];
  }
  __syncthreads();
  HelperCtx c;
  c.a = &a;
  c.s = &s;
  c.fw = (const char *)a.mf_frags + base_h(L, h, w) * 1024;
  c.zb = comm_z(a.sp_comm, L, blk);
  c.sw = comm_s(a.sp_comm, L, blk);
  c.hw = comm_hid(a.sp_comm, L, blk);
  c.abort_word = abort_word;
  c.mark = mark;
  c.tid = tid;
  c.w = w;
  c.lane = lane;
  c.n = lane & 15;
  c.q = lane >> 4;
  c.nl = (L - w + NW - 1) / NW;  // layers of this wave (L >= NW)
  c.wvoff = 16 * lane;
  c.h = h;
  c.local = s.local != 0;
  if (helper_layers(L) <= NRES) helper_steps<true>(c, hw1);
  else helper_steps<false>(c, hw1);
}

// ---------------------------------------------------------------------------
// Class block of group blk.  Per step: gather relu(hidden) of all 512 channels; wave w computes
// classes 32w .. 32w + 31 (output 1x1 tiles 2w, 2w + 1 over all 16 k-steps, its fragments in
// registers for the whole launch) + bias into LDS; then each wave takes streams w and w + 8:
// generation draws their samples (written out and returned to the chain block), forced modes write
// their logits out and return a step-done mark.

__device__ __forceinline__ void class_block(const StepArgs &a, char *lds_raw, int blk) {
  ClassLds &s = *(ClassLds *)lds_raw;
  const int tid = threadIdx.x, L = a.L;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, n = lane & 15, q = lane >> 4;
  const int b0 = blk * ROWS, nrows = min(ROWS, a.batch - b0);
  const u64 *hw = comm_hid(a.sp_comm, L, blk);
  u64 *sm = comm_smp(a.sp_comm, L, blk);
  uint32_t *abort_word = (uint32_t *)a.sp_comm;
  // launch handshake, first half: publish this block's XCD before loading anything
  u64 *hs = comm_hs(a.sp_comm, L, blk);
  const uint32_t mark = launch_mark(a);
  if (tid == 0) put_word(hs + HSLOT * NHLP, xcd_id(), mark, false);
  for (int i = tid; i < Q; i += NT) s.bias[i] = a.mf_bias[L * 3 * R + S + H + i];
  // output 1x1 fragments of classes 32w .. 32w + 31: tile j, k-step ks at j * 16 + ks of slice w
  u32x4 wo[2][H / 32];
  {
    const u32x4 *src = (const u32x4 *)((const char *)a.mf_frags + base_w2(L, w) * 1024);
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int ks = 0; ks < H / 32; ++ks) wo[j][ks] = src[(j * (H / 32) + ks) * 64 + lane];
  }
  // launch handshake, second half: learn whether the whole group shares one XCD
  if (tid == 0) {
    uint32_t v[1];
    wait_words<1>(hs + HSLOT * (NHLP + 1), mark, v, abort_word, a.sp_sticky, mark);
    s.local = (int)v[0];
  }
  __syncthreads();
  const bool local = s.local != 0;
  for (long long step = 0; step < a.n_steps; ++step) {
    const uint32_t tag = step_tag(a, step);
    // uniforms of steps [step, step + KCH): loaded before the wait for the hidden layer (their
    // latency hides behind it), stored after the barrier below, by which every wave has sampled the
    // previous chunk's last step
    constexpr int NU = ROWS * KCH / NT;
    static_assert(ROWS * KCH == NU * NT, "uniform chunk splits evenly over the block");
    const bool stage = a.mode == MODE_GENERATE && step % KCH == 0;
    float uv[NU];
#pragma unroll
    for (int e = 0; e < NU; ++e) {
      const int idx = tid + e * NT, r = idx / KCH, j = idx % KCH;
      uv[e] = 0.f;
      if (stage && r < nrows && step + j < a.n_steps) uv[e] = a.uniforms[(long long)(b0 + r) * a.n_steps + step + j];
    }
    gather_act(s.act, hw, tag, abort_word, a.sp_sticky, mark);
    __syncthreads();
    if (stage) {
#pragma unroll
      for (int e = 0; e < NU; ++e) {
        const int idx = tid + e * NT;
        s.u[idx / KCH][idx % KCH] = uv[e];
      }
    }
    // classes 32w + 16j + 4q .. +3 of stream n; two accumulators per tile (even and odd k-steps),
    // the k-step loop outermost: each activation read feeds both tiles and four independent
    // accumulation chains keep the matrix core busy
    f32x4 acc[2][2];
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[j][0] = acc[j][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < H / 32; ++ks) {
      const u32x4 b = lds16(s.act + n * PS + 32 * ks + 8 * q);
      acc[0][ks & 1] = mfma(wo[0][ks], b, acc[0][ks & 1]);
      acc[1][ks & 1] = mfma(wo[1][ks], b, acc[1][ks & 1]);
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int k = 32 * w + 16 * j + 4 * q;
      stf4(s.lg + n * PL + k, acc[j][0] + acc[j][1] + ldsf4(s.bias + k));
    }
    __syncthreads();
    const int r0 = w, r1 = w + NW;
    static_assert(ROWS == 2 * NW, "two rows per wave");
    if (a.mode == MODE_GENERATE) {
      const int2 k = sample256x2(s.lg + r0 * PL, s.lg + r1 * PL, s.u[r0][step % KCH], s.u[r1][step % KCH]);
      if (lane == 0) {
        if (r0 < nrows) a.samples[(long long)(b0 + r0) * a.n_steps + step] = k.x;
        if (r1 < nrows) a.samples[(long long)(b0 + r1) * a.n_steps + step] = k.y;
        put_word(sm + r0, (uint32_t)k.x, tag, local);
        put_word(sm + r1, (uint32_t)k.y, tag, local);
      }
    } else {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const int r = kk ? r1 : r0;
        if (r < nrows && a.logits) {
          const float4 v = *(const float4 *)(s.lg + r * PL + 4 * lane);
          *(float4 *)(a.logits + ((long long)(b0 + r) * a.n_steps + step) * Q + 4 * lane) = v;
        }
      }
      if (lane == 0) {
        put_word(sm + r0, 0u, tag, local);
        put_word(sm + r1, 0u, tag, local);
      }
    }
  }
}

__global__ void __launch_bounds__(NT) split_step_kernel(StepArgs a) {
  extern __shared__ float4 lds_raw[];
  const int nb = a.sp_nb;
  // helper h of group b sits at nb + h nb + b and its class block at (1 + NHLP) nb + b: with nb a
  // multiple of 8, all on the XCD of chain block b
  const int e = (int)blockIdx.x - nb;
  if (e < 0) {
    chain_block(a, (char *)lds_raw, blockIdx.x);
  } else if (e < NHLP * nb) {
    helper_block(a, (char *)lds_raw, e % nb, e / nb);
  } else {
    class_block(a, (char *)lds_raw, e - NHLP * nb);
  }
}

// ---------------------------------------------------------------------------
// Repacking into the fragment streams.  Fragment (tile t, k-step ks) of a matrix M[out][k] gives
// lane l the 8 values M[16t + l%16][32ks + 8(l/16) + j].

__device__ __forceinline__ uint16_t conv_elem(const uint16_t *conv, int o, int k) {
  return conv[(o * R + (k % R)) * 2 + (k >= R ? 1 : 0)];
}
__device__ __forceinline__ uint4 pack8(const uint16_t *v) {
  return make_uint4(v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16), v[6] | (v[7] << 16));
}

// Layer l: A wave p stream position 6l + f (f 0..3: x-half of tanh tile p k-steps 2,3 and sigmoid
// tile p k-steps 2,3; f 4,5: residual tile p k-steps 0,1); B wave p stream position 4 ((l-1) mod L)
// + f (v-half of tanh tile p k-steps 0,1, sigmoid tile p k-steps 0,1); helper (h, l % 8) position
// 8 (l / 8) + 2j + ks (skip tile 4h + j, k-step ks).
constexpr int LAYER_FRAGS = 4 * FA + 4 * FB + NHLP * FS;
__global__ void repack_layer_kernel(const uint16_t *conv, const uint16_t *res, const uint16_t *skip, int l, int L,
                                    uint4 *frags) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= LAYER_FRAGS * 64) return;
  const int lane = e % 64, m = lane % 16, kq = 8 * (lane / 16);
  int fi = e / 64;
  uint16_t v[8];
  size_t dst;
  if (fi < 4 * FA) {
    const int p = fi / FA, f = fi % FA;
    for (int j = 0; j < 8; ++j)
      v[j] = f < 4 ? conv_elem(conv, (f < 2 ? 0 : R) + 16 * p + m, R + 32 * (f & 1) + kq + j)
                   : res[(16 * p + m) * R + 32 * (f - 4) + kq + j];
    dst = base_a(L, p) + (size_t)FA * l + f;
  } else if ((fi -= 4 * FA) < 4 * FB) {
    const int p = fi / FB, f = fi % FB;
    for (int j = 0; j < 8; ++j) v[j] = conv_elem(conv, (f < 2 ? 0 : R) + 16 * p + m, 32 * (f & 1) + kq + j);
    dst = base_b(L, p) + (size_t)FB * ((l + L - 1) % L) + f;
  } else {
    fi -= 4 * FB;
    const int h = fi / FS, f = fi % FS, t = (SL / 16) * h + f / 2, ks = f % 2;
    for (int j = 0; j < 8; ++j) v[j] = skip[(16 * t + m) * R + 32 * ks + kq + j];
    dst = base_h(L, h, l % NW) + (size_t)FS * (l / NW) + f;
  }
  frags[dst * 64 + lane] = pack8(v);
}

// Head slices h: first 1x1 fragment (tile j, k-step ks) of rows 64h + 16j.. at j * 16 + ks (helper
// h); output 1x1 fragment (tile j, k-step ks) of classes 32h + 16j.. at j * 16 + ks (class block
// wave h).
__global__ void repack_head_kernel(const uint16_t *head, const uint16_t *out, int L, uint4 *frags) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= NHLP * (FW1 + FW2) * 64) return;
  const int lane = e % 64, m = lane % 16, kq = 8 * (lane / 16);
  const int fi = e / 64, h = fi / (FW1 + FW2), f = fi % (FW1 + FW2);
  uint16_t v[8];
  size_t dst;
  if (f < FW1) {
    const int j = f / (S / 32), ks = f % (S / 32);
    for (int i = 0; i < 8; ++i) v[i] = head[(h * HL + 16 * j + m) * S + 32 * ks + kq + i];
    dst = base_w1(L, h) + f;
  } else {
    const int g = f - FW1, j = g / (H / 32), ks = g % (H / 32);
    for (int i = 0; i < 8; ++i) v[i] = out[(h * QL + 16 * j + m) * H + 32 * ks + kq + i];
    dst = base_w2(L, h) + g;
  }
  frags[dst * 64 + lane] = pack8(v);
}

}  // namespace sp

// Exchange words of fwg_generate_noalloc (callers that cannot allocate): every launch of that entry
// point on a device uses this device's copy, so such launches that overlap on one device race.
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

hipError_t split_static_scratch(void **ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void *addr[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(mu);
  if (!addr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return hipSuccess;
}

size_t split_frag_bytes(int L) { return sp::frag_count(L) * 1024; }

size_t split_comm_bytes(int L, int nb) { return 256 + (size_t)nb * sp::group_words(L) * sizeof(unsigned long long); }

size_t split_lds_bytes(int L) {
  const size_t chain = sp::chain_fixed_bytes() + sp::dyn_bias_offset(L) + sizeof(float) * ((size_t)L * 3 * kMfR + kMfR);
  const size_t helper = sizeof(sp::HelperLds), cls = sizeof(sp::ClassLds);
  const size_t m = chain > helper ? chain : helper;
  return m > cls ? m : cls;
}

hipError_t launch_split_step(const StepArgs &a, hipStream_t s) {
  const dim3 grid(a.sp_nb * (2 + kSpHelpers)), block(kMfThreads);
  hipLaunchKernelGGL(sp::split_step_kernel, grid, block, split_lds_bytes(a.L), s, a);
  return hipGetLastError();
}

hipError_t split_setup(int L, int nb, int *coresident_ok) {
  const size_t lds = split_lds_bytes(L);
  hipError_t e = hipFuncSetAttribute((const void *)sp::split_step_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds);
  if (e != hipSuccess) return e;
  int per_cu = 0, dev = 0, cus = 0;
  if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, sp::split_step_kernel, kMfThreads, lds)) != hipSuccess)
    return e;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  *coresident_ok = (long long)per_cu * cus >= (long long)nb * (2 + kSpHelpers);
  return hipSuccess;
}

hipError_t launch_split_repack_layer(const void *conv, const void *res, const void *skip, int l, int L, void *frags,
                                     hipStream_t s) {
  const int n = sp::LAYER_FRAGS * 64;
  hipLaunchKernelGGL(sp::repack_layer_kernel, dim3((n + 255) / 256), dim3(256), 0, s, (const uint16_t *)conv,
                     (const uint16_t *)res, (const uint16_t *)skip, l, L, (uint4 *)frags);
  return hipGetLastError();
}

hipError_t launch_split_repack_head(const void *head, const void *out, int L, void *frags, hipStream_t s) {
  const int n = sp::NHLP * (sp::FW1 + sp::FW2) * 64;
  hipLaunchKernelGGL(sp::repack_head_kernel, dim3((n + 255) / 256), dim3(256), 0, s, (const uint16_t *)head,
                     (const uint16_t *)out, L, (uint4 *)frags);
  return hipGetLastError();
}

}  // namespace fwg
