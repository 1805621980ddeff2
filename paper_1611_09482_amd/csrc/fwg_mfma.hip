// MFMA step kernel for gated stacks with bf16 operands, R = 64 residual
// channels, S = H = 512 skip/head channels and 256 classes (gfx950,
// v_mfma_f32_16x16x32_bf16, fp32 accumulation).
//
// One block of 8 waves owns 16 independent streams; one launch runs n_steps
// whole generation steps.  Per step and layer (paper Section 2.2): pop the
// layer's queue (the state pushed d_l steps earlier; at filter width 3 also the
// one pushed 2 d_l steps earlier, Section 3.1), compute the dilated product
// [W_r W_e] [v; x], the gate, the residual and skip 1x1 products, then push the
// layer's input into the slot of the oldest state popped.  After the
// last layer: relu(skip sum) -> 1x1 -> relu -> 1x1 -> logits, softmax and the
// inverse-CDF sample, which becomes the next step's input (Section 1).
//
// Products are computed transposed, D[channel][stream] = W[channel][k] X[stream][k]:
// weights are the MFMA A operand (16 output channels x 32 k), activations the B
// operand (32 k x 16 streams).  Each lane then holds 4 consecutive channels of
// one stream, so activation tiles move to and from LDS as 8- and 16-byte rows.
//
// Wave roles.  Waves p and p + 4 share SIMD p and split the work of channel tile p:
//  - wave p ("A", on the layer-to-layer dependency chain): the current-input half of the
//    dilated product (W_e x) for tanh tile p and sigmoid tile p, the gate, the residual
//    1x1 for tile p, and 7 of the 16 skip fragments of skip tiles 8p..8p+7;
//  - wave p + 4 ("B"): the recurrent half (W_r v, v = the popped states, known early) of the
//    NEXT layer plus its bias, handed to A through LDS, the other 9 skip fragments, and the
//    queue pops and pushes of rows 4p..4p+3.  At width 3 the oldest tap's fragments come from a
//    stream of their own (4 per layer and wave), loaded one recurrent product ahead.
// Both halves of the head are split the same way.  Every wave streams its own pre-packed
// weight fragments from L2 (13 per stage, refilled one stage ahead as soon as consumed); a
// wave stalls while the load unit is saturated, and the second wave on the SIMD keeps the
// SIMD busy meanwhile, so the dependency chain overlaps the weight stream.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fwg_internal.h"
#include "fwg_mfma_dev.h"

namespace fwg {
namespace mf {

using namespace mfd;

// ---------------------------------------------------------------------------
// Shapes and LDS layout (elements; activations bf16 with 8-element row padding)
constexpr int R = kMfR, S = kMfS, H = kMfH, Q = 256, ROWS = kMfRows;
constexpr int NT = kMfThreads;
constexpr int PX = R + 8;   // 64-channel activation rows
constexpr int PS = S + 8;   // 512-channel activation rows (skip / head hidden)
constexpr int PL = Q + 4;   // fp32 logits rows
constexpr int PP = 20;      // fp32 partial-tile rows (16 channels + 4 padding)
constexpr int F = kMfFrags, NHEAD = kMfHeadStages;
// per-wave head fragment stream g = 13 h + f, k-step major: first 1x1 (g < GH1: 4 tiles), output
// 1x1 (GH1 <= g < GOUT: 2 tiles), then padding (wave B carries the next layer 0's W_r at GCV..)
constexpr int GH1 = 64, GOUT = 96, GCV = 100;
constexpr int KCH = 64;  // steps per chunk of per-step inputs staged in LDS

struct Lds {
  uint16_t vbuf[2][ROWS * PX];     // popped queue rows (layer input d steps ago), by stage parity
                                   // (width 3: the rows 2d steps ago follow the bias block)
  uint16_t xbuf[2][ROWS * PX];     // layer inputs x^l, by layer parity
  uint16_t zbuf[ROWS * PX];        // gate output of the current layer
  float pbuf[2][4][2][ROWS * PP];  // W_r v + b of a layer: [stage parity][tile][tanh / sigmoid]
  float ptile[4][ROWS * PP];       // partial skip tile 8p+3 of wave A, handed to wave B at the head
  uint16_t hbuf[ROWS * PS];
  union {
    uint16_t sbuf[ROWS * PS];
    float lg[ROWS * PL];
  } u;
  uint16_t embT[Q * R];  // embedding table, [class][channel]
  // per-step inputs of the block's streams for a chunk of KCH steps: uniforms (generation) or the
  // forced input that follows each step, loaded once per chunk
  union {
    float u[ROWS][KCH];
    int in[ROWS][KCH];
  } chunk;
  int ins[ROWS];
  int pad_[ROWS];
  // followed by the per-layer tables (dynamic part): roff[L] (int64), slot[L], dep[L], then fp32 biases,
  // then (width 3) the second popped-row buffer [2][ROWS * PX]
};

__host__ __device__ constexpr size_t lds_fixed_bytes() { return (sizeof(Lds) + 15) & ~size_t(15); }
// dynamic part: roff[L] (8 B), slot[L], dep[L] (4 B each; dep = queue depth (w - 1) d), then the
// bias block at a 16-byte boundary, then (width 3) the rows popped 2d steps back
__host__ __device__ inline size_t lds_dyn_bias_offset(int L) { return ((size_t)L * 16 + 15) & ~size_t(15); }
__host__ __device__ inline size_t lds_dyn_vb1_offset(int L) {
  return (lds_dyn_bias_offset(L) + sizeof(float) * mfma_bias_floats(L) + 15) & ~size_t(15);
}

struct Frags {
  u32x4 f[F];
};
// the oldest tap's recurrent fragments of one layer (width 3)
struct TapFrags {
  u32x4 f[4];
};

// Stage k of a step is layer k (k < L) or head stage k - L.
struct Ctx {
  const StepArgs *a;
  Lds *s;
  uint16_t *vb1;  // width 3: popped rows of the oldest tap, [2][ROWS * PX]
  int *slot, *dep;
  const long long *roff;
  const float *conv_b, *res_b, *skip_sum, *head_b, *out_b, *emb_b;
  const char *frags;  // fragment streams (wave-uniform base)
  const char *tapfrags;  // width 3: the oldest tap's fragments, [L][4 B waves][4] x 1 KB
  int wvoff;          // this lane's byte offset inside a fragment (16 * lane)
  int L, NS, w, p, lane, n, q, b0, nrows;
};

// Byte offset (wave-uniform) of stage k's fragment stream for this wave: stage-major, 8 waves
// per stage, F fragments of 1 KB each.
__device__ __forceinline__ int stage_off(const Ctx &c, int k) { return (k * kMfWaves + c.w) * F * 1024; }
__device__ __forceinline__ u32x4 load_frag(const Ctx &c, int off, int f) {
  return *(const u32x4 *)(c.frags + (off + f * 1024) + c.wvoff);
}
// Slot f has just been consumed: start loading the same slot of the next stage.
// The scheduling barrier keeps the compiler from hoisting the load above the MFMA that still
// reads the slot's previous contents (which would keep both copies live).
__device__ __forceinline__ void refill(const Ctx &c, Frags &W, int nx, int f) {
  __builtin_amdgcn_sched_barrier(0);
  W.f[f] = load_frag(c, nx, f);
  __builtin_amdgcn_sched_barrier(0);
}
// Load a whole stage in slot order, as the loop refills them (the compiler's load accounting at
// the loop entry then matches the loop's own).
__device__ __forceinline__ void load_stage(const Ctx &c, int k, Frags &fr) {
  const int off = stage_off(c, k);
#pragma unroll
  for (int f = 0; f < F; ++f) refill(c, fr, off, f);
}

// Queue traffic is issued by the B waves: wave B of pair p moves stream rows 4p..4p+3, lane l
// handling row 4p + (l%32)/8 and 16-byte chunk l%8 (lanes 32..63 mirror lanes 0..31 on loads and
// skip the stores); the lane that pushes a row chunk later pops it.  Vector loads return to a
// wave in issue order, so a queue read that goes out to HBM holds back the weight fragments its
// wave requests after it: wave B therefore prefetches its fragments two stages ahead.
__device__ __forceinline__ long long ring_elem(const Ctx &c, int l, int slotv) {
  const int r = 4 * c.p + ((c.lane & 31) >> 3);
  return c.roff[l] + ((long long)slotv * c.a->bmax + (c.b0 + r)) * R + 8 * (c.lane & 7);
}
// Issue the pop of stage k (a layer) for step offset `ahead` (0: the step the slot table
// describes, 1: the next one).  Head stages pop layer 0 as a harmless placeholder.  The queue of
// a layer holds its last (w - 1) d inputs; the slot of the step holds the oldest, tap j sits j d
// slots after it.  Width 2 (TP = 1): lanes 32..63 repeat the loads of lanes 0..31; width 3
// (TP = 2): lanes 0..31 load the oldest rows (2d steps back), lanes 32..63 those d steps back.
template <int TP>
__device__ __forceinline__ u32x4 pop_issue(const Ctx &c, int k, int ahead) {
  const int l = k < c.L ? k : 0;
  const int dep = c.dep[l];
  int sl = c.slot[l] + ahead;
  if (sl >= dep) sl -= dep;
  if (TP == 2 && c.lane >= 32) {
    sl += dep >> 1;
    if (sl >= dep) sl -= dep;
  }
  const uint16_t *ring = (const uint16_t *)c.a->ring;
  return __builtin_nontemporal_load((const u32x4 *)(ring + ring_elem(c, l, sl)));
}
// vbuf holds the rows d steps back; at width 3 vb1 the rows 2d steps back
template <int TP>
__device__ __forceinline__ void pop_land(const Ctx &c, int parity, u32x4 v) {
  const int r = 4 * c.p + ((c.lane & 31) >> 3);
  const int e = r * PX + 8 * (c.lane & 7);
  if (TP == 1) {
    if (c.lane < 32) *(u32x4 *)(c.s->vbuf[parity] + e) = v;
  } else {
    *(u32x4 *)((c.lane < 32 ? c.vb1 + parity * ROWS * PX : c.s->vbuf[parity]) + e) = v;
  }
}
// push phase of layer l: its input x^l replaces the slot popped for this step
__device__ __forceinline__ void push_rows(const Ctx &c, int l) {
  if (c.lane < 32) {
    const int r = 4 * c.p + (c.lane >> 3);
    const u32x4 v = *(const u32x4 *)(c.s->xbuf[l & 1] + r * PX + 8 * (c.lane & 7));
    uint16_t *ring = (uint16_t *)c.a->ring;
    __builtin_nontemporal_store(v, (u32x4 *)(ring + ring_elem(c, l, c.slot[l])));
  }
}

// Accumulators.  Wave A: xres (residual channels 16p + 4q + i of stream n), acc[0..2] skip tiles
// 8p..8p+2, acc[3] the k-step-0 half of skip tile 8p+3.  Wave B: acc[0] the k-step-1 half of skip
// tile 8p+3, acc[1..4] skip tiles 8p+4..8p+7.  In the head acc[0..3] hold the first 1x1's tiles
// and acc[0..1] the output tiles of the wave's half.
struct Acc {
  f32x4 xres;
  f32x4 acc[5];
};

// The oldest tap's fragments of layer l for this B wave (width 3).
__device__ __forceinline__ void load_tap(const Ctx &c, int l, TapFrags &X) {
#pragma unroll
  for (int f = 0; f < 4; ++f)
    X.f[f] = *(const u32x4 *)(c.tapfrags + ((size_t)(l * 4 + c.p) * 4 + f) * 1024 + c.wvoff);
}

// W_r v + b for layer `ln`, computed by wave B one stage ahead from fragments f0..f0+3 (tanh tile
// p k-steps 0,1, sigmoid tile p k-steps 0,1) and the popped rows in vbuf[par]; stored in pbuf[par].
// Width 3 (TP = 2) adds the oldest tap's product (fragments X, rows in vb1), then loads X with the
// next recurrent product's fragments (layer ln + 1, or layer 0 of the next step).
template <int TP>
__device__ __forceinline__ void recurrent_half(const Ctx &c, int ln, int par, const Frags &W, int f0, TapFrags &X) {
  Lds &s = *c.s;
  const uint16_t *vb = s.vbuf[par] + c.n * PX;
  const u32x4 bv0 = lds16(vb + 8 * c.q), bv1 = lds16(vb + 32 + 8 * c.q);
  u32x4 bo0, bo1;
  if (TP == 2) {
    const uint16_t *vo = c.vb1 + par * ROWS * PX + c.n * PX;
    bo0 = lds16(vo + 8 * c.q);
    bo1 = lds16(vo + 32 + 8 * c.q);
  }
  const float *cb = c.conv_b + ln * 2 * R;
  f32x4 pt = ldsf4(cb + 16 * c.p + 4 * c.q), pg = ldsf4(cb + R + 16 * c.p + 4 * c.q);
  pt = mfma(W.f[f0 + 0], bv0, pt);
  pg = mfma(W.f[f0 + 2], bv0, pg);
  pt = mfma(W.f[f0 + 1], bv1, pt);
  pg = mfma(W.f[f0 + 3], bv1, pg);
  if (TP == 2) {
    pt = mfma(X.f[0], bo0, pt);
    pg = mfma(X.f[2], bo0, pg);
    pt = mfma(X.f[1], bo1, pt);
    pg = mfma(X.f[3], bo1, pg);
    __builtin_amdgcn_sched_barrier(0);
    load_tap(c, ln + 1 < c.L ? ln + 1 : 0, X);
    __builtin_amdgcn_sched_barrier(0);
  }
  stf4(s.pbuf[par][c.p][0] + c.n * PP + 4 * c.q, pt);
  stf4(s.pbuf[par][c.p][1] + c.n * PP + 4 * c.q, pg);
}

// Stage position helpers.
struct Pos {
  long long step;
  int k;
};
__device__ __forceinline__ Pos advance(const Ctx &c, Pos p, int m) {
  p.k += m;
  while (p.k >= c.NS) { p.k -= c.NS; p.step += 1; }
  return p;
}

// Stage body shared by the two roles' loops; `nx` is the fragment stream that refills W.
// Stage the per-step inputs of steps [s0, s0 + KCH) in LDS: the uniform of (row r, step s) for
// generation; in the forced modes the input that follows step s (inputs[s + 1] for teacher
// forcing, the observed sample inputs[s] for online prediction).  Called by every thread of the block
// once per chunk (in the first head stage, before its barriers).
__device__ __forceinline__ void stage_chunk(const Ctx &c, long long s0) {
  const StepArgs &a = *c.a;
  Lds &s = *c.s;
  // a fixed number of entries per thread (no loop), which keeps the compiler's load accounting
  // precise in the code around it
  static_assert((ROWS * KCH) % NT == 0, "the chunk divides evenly over the threads");
#pragma unroll
  for (int e = 0; e < ROWS * KCH / NT; ++e) {
    const int idx = (int)threadIdx.x + e * NT;
    const int r = idx / KCH, j = idx % KCH;
    const long long st = s0 + j;
    if (a.mode != MODE_GENERATE) {
      const long long nx = st + forced_shift(a.mode);
      int v = 0;
      if (r < c.nrows && nx < a.n_steps) v = a.inputs[(long long)(c.b0 + r) * a.n_steps + nx];
      s.chunk.in[r][j] = v;
    } else {
      float v = 0.f;
      if (r < c.nrows && st < a.n_steps) v = a.uniforms[(long long)(c.b0 + r) * a.n_steps + st];
      s.chunk.u[r][j] = v;
    }
  }
}

// End of a step: logits to LDS, sample (or write logits), next inputs, queue slots advance.
template <bool ISA>
__device__ __forceinline__ void finish_step(const Ctx &c, long long step, Acc &A) {
  Lds &s = *c.s;
  const StepArgs &a = *c.a;
  constexpr int ooff = ISA ? 0 : 32;
#pragma unroll
  for (int j = 0; j < 2; ++j) stf4(s.u.lg + c.n * PL + 64 * c.p + ooff + 16 * j + 4 * c.q, A.acc[j]);
  __syncthreads();
  const int tid = threadIdx.x;
  // straight-line code (no loop exits), which keeps the compiler's load accounting precise
  if (a.mode != MODE_GENERATE) {
#pragma unroll
    for (int kk = 0; kk < ROWS / kMfWaves; ++kk) {
      const int r = c.w + kMfWaves * kk;
      if (r < c.nrows && a.logits) {
        const float4 v = *(const float4 *)(s.u.lg + r * PL + 4 * c.lane);
        *(float4 *)(a.logits + ((long long)(c.b0 + r) * a.n_steps + step) * Q + 4 * c.lane) = v;
      }
    }
    if (tid < c.nrows && step + forced_shift(a.mode) < a.n_steps) s.ins[tid] = s.chunk.in[tid][step % KCH];
  } else {
    // rows c.w and c.w + 8 in one pass
    static_assert(ROWS == 2 * kMfWaves, "two rows per wave");
    const int r0 = c.w, r1 = c.w + kMfWaves;
    const int2 k = sample256x2(s.u.lg + r0 * PL, s.u.lg + r1 * PL, s.chunk.u[r0][step % KCH], s.chunk.u[r1][step % KCH]);
    if (c.lane == 0) {
      if (r0 < c.nrows) {
        a.samples[(long long)(c.b0 + r0) * a.n_steps + step] = k.x;
        s.ins[r0] = k.x;
      }
      if (r1 < c.nrows) {
        a.samples[(long long)(c.b0 + r1) * a.n_steps + step] = k.y;
        s.ins[r1] = k.y;
      }
    }
  }
  // waves A cover threads 0..255, more than the layer count
  for (int l = tid; l < c.L; l += NT) {
    const int nx = c.slot[l] + 1;
    c.slot[l] = nx == c.dep[l] ? 0 : nx;
  }
  __syncthreads();
}

// Head stage C, fragments [F0, F1) of the wave's head stream g = 13C + f.  Wave A owns first-1x1
// tiles 8p..8p+3 and output tiles 4p, 4p+1; wave B tiles 8p+4..8p+7 and 4p+2, 4p+3.  One barrier
// at the first output fragment (g = GH1, in head stage 4).
static_assert(F * 4 + 12 == GH1, "the head's hidden-layer barrier sits in head stage 4");
template <int TP, int C, bool ISA, int F0, int F1>
__device__ __forceinline__ void head_frags(const Ctx &c, long long i, const Frags &W, Acc &A, TapFrags &X) {
  Lds &s = *c.s;
  const int n = c.n, q = c.q, p = c.p;
  constexpr int hoff = ISA ? 0 : 64;  // channel offset of this wave's half inside the pair's 128
  constexpr int ooff = ISA ? 0 : 32;  // class offset of this wave's half inside the pair's 64
  u32x4 b = u32x4{0, 0, 0, 0};
#pragma unroll
  for (int f = F0; f < F1; ++f) {
    const int g = F * C + f;
    if (g < GH1) {
      const int ks = g / 4, j = g % 4;
      if (j == 0 || f == F0) b = lds16(s.u.sbuf + n * PS + 32 * ks + 8 * q);
      A.acc[j] = mfma(W.f[f], b, A.acc[j]);
    } else if (g < GOUT) {
      if (g == GH1) {
        // relu(head hidden) becomes the output 1x1's input
#pragma unroll
        for (int j = 0; j < 4; ++j) lds8(s.hbuf + n * PS + 128 * p + hoff + 16 * j + 4 * q, pack4(relu4(A.acc[j])));
#pragma unroll
        for (int j = 0; j < 2; ++j) A.acc[j] = ldsf4(c.out_b + 64 * p + ooff + 16 * j + 4 * q);
        __syncthreads();
      }
      const int ks = (g - GH1) / 2, j = (g - GH1) % 2;
      if (j == 0 || f == F0) b = lds16(s.hbuf + n * PS + 32 * ks + 8 * q);
      A.acc[j] = mfma(W.f[f], b, A.acc[j]);
    } else if (g == GCV && !ISA) {
      // W_r v + b of the next step's layer 0
      recurrent_half<TP>(c, 0, (int)((i + 1) & 1), W, f, X);
    }
  }
}

// Start of head stage 0: relu(skip sum) becomes the first head 1x1's input (skip tile 8p+3 is
// split over the pair), then the head accumulators take the first 1x1's bias.  Two barriers.
template <bool ISA>
__device__ __forceinline__ void head_start(const Ctx &c, Pos p0, Acc &A) {
  Lds &s = *c.s;
  const int n = c.n, q = c.q, p = c.p;
  constexpr int hoff = ISA ? 0 : 64;
  if (p0.step % KCH == 0) stage_chunk(c, p0.step);
  if (ISA) {
#pragma unroll
    for (int j = 0; j < 3; ++j) lds8(s.u.sbuf + n * PS + 128 * p + 16 * j + 4 * q, pack4(relu4(A.acc[j])));
    stf4(s.ptile[p] + n * PP + 4 * q, A.acc[3]);
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) lds8(s.u.sbuf + n * PS + 128 * p + 64 + 16 * j + 4 * q, pack4(relu4(A.acc[1 + j])));
  }
  __syncthreads();
  if (!ISA) {
    const f32x4 t = A.acc[0] + ldsf4(s.ptile[p] + n * PP + 4 * q);
    lds8(s.u.sbuf + n * PS + 128 * p + 48 + 4 * q, pack4(relu4(t)));
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) A.acc[j] = ldsf4(c.head_b + 128 * p + hoff + 16 * j + 4 * q);
  __syncthreads();
}

template <int TP, bool ISA, int F0, int F1>
__device__ __forceinline__ void head_part(const Ctx &c, Pos p0, long long i, const Frags &W, Acc &A, TapFrags &X) {
  switch (p0.k - c.L) {
    case 0:
      if (F0 == 0) head_start<ISA>(c, p0, A);
      head_frags<TP, 0, ISA, F0, F1>(c, i, W, A, X);
      break;
    case 1: head_frags<TP, 1, ISA, F0, F1>(c, i, W, A, X); break;
    case 2: head_frags<TP, 2, ISA, F0, F1>(c, i, W, A, X); break;
    case 3: head_frags<TP, 3, ISA, F0, F1>(c, i, W, A, X); break;
    case 4: head_frags<TP, 4, ISA, F0, F1>(c, i, W, A, X); break;
    case 5: head_frags<TP, 5, ISA, F0, F1>(c, i, W, A, X); break;
    case 6: head_frags<TP, 6, ISA, F0, F1>(c, i, W, A, X); break;
    default: head_frags<TP, 7, ISA, F0, F1>(c, i, W, A, X); break;
  }
}
static_assert(NHEAD == 8, "head_part dispatches eight head stages");

// Refill fragment slots [F0, F1) from stage stream `nx`.
template <int F0, int F1>
__device__ __forceinline__ void refill_range(const Ctx &c, Frags &W, int nx) {
#pragma unroll
  for (int f = F0; f < F1; ++f) refill(c, W, nx, f);
}

// Every stage of either role runs as parts that consume fragment slots [0,4), [4,6) and [6,13)
// in that order, whatever the stage type; the slots are refilled between the parts, in code
// common to all stage types, so each fragment register has a single definition in the loop (per
// stage-type refills would make the compiler copy registers at the merge, which waits for every
// outstanding load).

// Stage of wave A (global stage index i).  Layer: x -> W_e x + (W_r v + b) -> gate -> z |
// barrier | residual 1x1 -> x^{l+1}, skip fragments.
__device__ __forceinline__ void a_stage(const Ctx &c, Pos p0, long long i, Frags &W, int nx, Acc &A) {
  Lds &s = *c.s;
  TapFrags X;  // unused: wave A computes no recurrent half
  const int n = c.n, q = c.q, p = c.p;
  const int par = (int)(i & 1);
  const int l = p0.k;
  const bool layer = l < c.L;
  f32x4 af, ag;
  // ---- slots 0..3: the current-input half of the dilated product
  if (layer) {
    u32x4 bx0, bx1;
    if (l == 0) {
      // embedding (current input x^0): row gather of the transposed 1x1 convolution plus bias
      const int in = s.ins[n];
      const uint16_t *e = s.embT + in * R;
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
      // this wave's residual tile and its bf16 copy (pushed into queue 0 by wave B)
      const int ch = 16 * p + 4 * q;
      const u32x2 raw = *(const u32x2 *)(e + ch);
      A.xres = f32x4{bf_lo(raw.x) + eb[ch], bf_hi(raw.x) + eb[ch + 1], bf_lo(raw.y) + eb[ch + 2],
                     bf_hi(raw.y) + eb[ch + 3]};
      lds8(s.xbuf[0] + n * PX + ch, pack4(A.xres));
#pragma unroll
      for (int j = 0; j < 4; ++j) A.acc[j] = ldsf4(c.skip_sum + 128 * p + 16 * j + 4 * q);
    } else {
      const uint16_t *xb = s.xbuf[l & 1] + n * PX;
      bx0 = lds16(xb + 8 * q);
      bx1 = lds16(xb + 32 + 8 * q);
    }
    af = ldsf4(s.pbuf[par][p][0] + n * PP + 4 * q);
    ag = ldsf4(s.pbuf[par][p][1] + n * PP + 4 * q);
    af = mfma(W.f[0], bx0, af);
    ag = mfma(W.f[2], bx0, ag);
    af = mfma(W.f[1], bx1, af);
    ag = mfma(W.f[3], bx1, ag);
  } else {
    head_part<1, true, 0, 4>(c, p0, i, W, A, X);
  }
  refill_range<0, 4>(c, W, nx);
  u32x4 bz0, bz1;
  if (layer) {
    f32x4 z;
#pragma unroll
    for (int i4 = 0; i4 < 4; ++i4) z[i4] = gate(af[i4], ag[i4]);
    lds8(s.zbuf + n * PX + 16 * p + 4 * q, pack4(z));
    __syncthreads();
    // ---- slots 4, 5: residual 1x1 -> x^{l+1}
    const uint16_t *zb = s.zbuf + n * PX;
    bz0 = lds16(zb + 8 * q);
    bz1 = lds16(zb + 32 + 8 * q);
    f32x4 xr = A.xres + ldsf4(c.res_b + l * R + 16 * p + 4 * q);
    xr = mfma(W.f[4], bz0, xr);
    xr = mfma(W.f[5], bz1, xr);
    A.xres = xr;
    lds8(s.xbuf[(l + 1) & 1] + n * PX + 16 * p + 4 * q, pack4(xr));
  } else {
    head_part<1, true, 4, 6>(c, p0, i, W, A, X);
  }
  refill_range<4, 6>(c, W, nx);
  // ---- slots 6..12: skip tiles 8p..8p+2 (both k-steps) and the k-step-0 half of tile 8p+3
  if (layer) {
#pragma unroll
    for (int j = 0; j < 3; ++j) A.acc[j] = mfma(W.f[6 + j], bz0, A.acc[j]);
#pragma unroll
    for (int j = 0; j < 3; ++j) A.acc[j] = mfma(W.f[9 + j], bz1, A.acc[j]);
    A.acc[3] = mfma(W.f[12], bz0, A.acc[3]);
  } else {
    head_part<1, true, 6, F>(c, p0, i, W, A, X);
  }
  refill_range<6, F>(c, W, nx);
  if (p0.k == c.NS - 1) finish_step<true>(c, p0.step, A);
}

// Stage of wave B.  Layer: W_r v + b of the next layer (its popped rows are already in LDS) |
// barrier | push of the layer input, skip fragments.  `W` is the buffer of this stage's parity
// and `nx` the fragment stream of the stage two ahead.
template <int TP>
__device__ __forceinline__ void b_stage(const Ctx &c, Pos p0, long long i, Frags &W, int nx, Acc &A, TapFrags &X) {
  Lds &s = *c.s;
  const int n = c.n, q = c.q, p = c.p;
  const int par = (int)(i & 1);
  const int l = p0.k;
  const bool layer = l < c.L;
  // ---- slots 0..3: W_r v + b of the next layer
  if (layer) {
    if (l == 0) {
      A.acc[0] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < 4; ++j) A.acc[1 + j] = ldsf4(c.skip_sum + 128 * p + 64 + 16 * j + 4 * q);
    }
    if (l + 1 < c.L) recurrent_half<TP>(c, l + 1, par ^ 1, W, 0, X);
  } else {
    head_part<TP, false, 0, 4>(c, p0, i, W, A, X);
  }
  refill_range<0, 4>(c, W, nx);
  u32x4 bz0, bz1;
  if (layer) {
    __syncthreads();
    push_rows(c, l);
    const uint16_t *zb = s.zbuf + n * PX;
    bz0 = lds16(zb + 8 * q);
    bz1 = lds16(zb + 32 + 8 * q);
    // ---- slots 4, 5: the k-step-1 half of skip tile 8p+3, skip tile 8p+4 k-step 0
    A.acc[0] = mfma(W.f[4], bz1, A.acc[0]);
    A.acc[1] = mfma(W.f[5], bz0, A.acc[1]);
  } else {
    head_part<TP, false, 4, 6>(c, p0, i, W, A, X);
  }
  refill_range<4, 6>(c, W, nx);
  // ---- slots 6..12: skip tiles 8p+5..8p+7 k-step 0, tiles 8p+4..8p+7 k-step 1
  if (layer) {
#pragma unroll
    for (int j = 1; j < 4; ++j) A.acc[1 + j] = mfma(W.f[5 + j], bz0, A.acc[1 + j]);
#pragma unroll
    for (int j = 0; j < 4; ++j) A.acc[1 + j] = mfma(W.f[9 + j], bz1, A.acc[1 + j]);
  } else {
    head_part<TP, false, 6, F>(c, p0, i, W, A, X);
  }
  refill_range<6, F>(c, W, nx);
  if (p0.k == c.NS - 1) finish_step<false>(c, p0.step, A);
}

// Main loop of wave A: one fragment buffer, each slot refilled with the next stage's.
__device__ __forceinline__ void a_role(const Ctx &c, long long total) {
  Acc A;
  Frags W;
  __syncthreads();  // queue rows of stages 0 and 1 are in LDS
  load_stage(c, 0, W);
  __syncthreads();  // W_r v + b of layer 0 is in LDS
  Pos p0{0, 0};
  for (long long i = 0; i < total; ++i) {
    const Pos p1 = advance(c, p0, 1);
    a_stage(c, p0, i, W, stage_off(c, p1.k), A);
    __syncthreads();
    p0 = p1;
  }
}

// Main loop of wave B: two fragment buffers by stage parity, each slot refilled with the stage two
// ahead; queue rows of stage i+3 are read at the start of stage i and land in LDS at the end of
// stage i+1, for the W_r v of stage i+3 computed during stage i+2.
template <int TP>
__device__ __forceinline__ void b_role(const Ctx &c, long long total) {
  Acc A;
  Frags W0, W1;
  TapFrags X;
  const Pos p0i{0, 0};
  const Pos p1i = advance(c, p0i, 1), p2i = advance(c, p0i, 2);
  pop_land<TP>(c, 0, pop_issue<TP>(c, 0, 0));
  pop_land<TP>(c, 1, pop_issue<TP>(c, p1i.k, (int)p1i.step));
  u32x4 vA, vB = pop_issue<TP>(c, p2i.k, (int)p2i.step);
  __syncthreads();
  {
    // W_r v + b of layer 0 from this wave's fragments in the last head stage
    const int off = stage_off(c, c.NS - 1);
#pragma unroll
    for (int f = 0; f < 4; ++f) W0.f[f] = load_frag(c, off, GCV - F * (NHEAD - 1) + f);
    if (TP == 2) load_tap(c, 0, X);
    recurrent_half<TP>(c, 0, 0, W0, 0, X);
  }
  load_stage(c, 0, W0);
  load_stage(c, p1i.k, W1);
  __syncthreads();
  Pos p0 = p0i;
  long long i = 0;
  for (; i + 1 < total; i += 2) {
    const Pos p1 = advance(c, p0, 1), p2 = advance(c, p0, 2), p3 = advance(c, p0, 3), p4 = advance(c, p0, 4);
    vA = pop_issue<TP>(c, p3.k, (int)(p3.step - p0.step));
    __builtin_amdgcn_sched_barrier(0);
    b_stage<TP>(c, p0, i, W0, stage_off(c, p2.k), A, X);
    if (p2.k < c.L && i + 2 < total) pop_land<TP>(c, 0, vB);
    __syncthreads();
    vB = pop_issue<TP>(c, p4.k, (int)(p4.step - p1.step));
    __builtin_amdgcn_sched_barrier(0);
    b_stage<TP>(c, p1, i + 1, W1, stage_off(c, p3.k), A, X);
    if (p3.k < c.L && i + 3 < total) pop_land<TP>(c, 1, vA);
    __syncthreads();
    p0 = p2;
  }
  if (i < total) {
    // odd stage count: the last stage (its queue rows for later stages are not needed)
    const Pos p2 = advance(c, p0, 2);
    b_stage<TP>(c, p0, i, W0, stage_off(c, p2.k), A, X);
    __syncthreads();
  }
}

// TP = recurrent taps per dilated product (filter width - 1): 1 or 2.
template <int TP>
__global__ void __launch_bounds__(NT) mfma_step_kernel(StepArgs a) {
  extern __shared__ float4 lds_raw[];
  Lds &s = *(Lds *)lds_raw;
  const int tid = threadIdx.x;
  const int L = a.L;
  char *dyn = (char *)lds_raw + lds_fixed_bytes();
  long long *roff = (long long *)dyn;
  int *slot = (int *)(roff + L);
  int *dep = slot + L;
  // conv_b [L][2R], res_b [L][R], skip_sum [S], head_b [H], out_b [Q], emb_b [R]; 16-byte aligned
  float *bias = (float *)(dyn + lds_dyn_bias_offset(L));

  Ctx c;
  c.a = &a;
  c.s = &s;
  c.slot = slot;
  c.dep = dep;
  c.vb1 = (uint16_t *)(dyn + lds_dyn_vb1_offset(L));
  c.roff = roff;
  c.conv_b = bias;
  c.res_b = c.conv_b + L * 2 * R;
  c.skip_sum = c.res_b + L * R;
  c.head_b = c.skip_sum + S;
  c.out_b = c.head_b + H;
  c.emb_b = c.out_b + Q;
  c.L = L;
  c.NS = L + NHEAD;
  c.w = __builtin_amdgcn_readfirstlane(tid >> 6);
  c.p = c.w & 3;
  c.lane = tid & 63;
  c.n = c.lane & 15;
  c.q = c.lane >> 4;
  c.b0 = blockIdx.x * ROWS;
  c.nrows = min(ROWS, a.batch - c.b0);
  c.frags = (const char *)a.mf_frags;
  c.tapfrags = c.frags + mfma_frag_bytes(L);
  c.wvoff = 16 * c.lane;

  // tables: embedding [Q][R], biases, queue offsets, dilations and slots
  const u32x4 *embsrc = (const u32x4 *)a.mf_embT;
  for (int i = tid; i < Q * R / 8; i += NT) ((u32x4 *)s.embT)[i] = embsrc[i];
  const int nbias = L * 3 * R + S + H + Q + R;
  for (int i = tid; i < nbias; i += NT) bias[i] = a.mf_bias[i];
  for (int l = tid; l < L; l += NT) {
    const LayerDev ld = a.layers[l];
    roff[l] = ld.ring_off;
    dep[l] = ld.depth;
    slot[l] = (int)(a.t0 % (long long)ld.depth);
  }
  if (tid < ROWS) {
    int v = 0;
    if (tid < c.nrows) v = a.mode == MODE_TEACHER ? a.inputs[(long long)(c.b0 + tid) * a.n_steps] : a.last[c.b0 + tid];
    s.ins[tid] = v;
  }
  __syncthreads();

  const long long total = (long long)a.n_steps * c.NS;
  if (c.w < 4) a_role(c, total);
  else b_role<TP>(c, total);
  if (a.mode != MODE_TEACHER && tid < c.nrows) a.last[c.b0 + tid] = s.ins[tid];
}

}  // namespace mf

size_t mfma_lds_bytes(int L, int w) {
  if (w == 3) return mf::lds_fixed_bytes() + mf::lds_dyn_vb1_offset(L) + sizeof(uint16_t) * 2 * mf::ROWS * mf::PX;
  return mf::lds_fixed_bytes() + mf::lds_dyn_bias_offset(L) + sizeof(float) * mfma_bias_floats(L);
}

hipError_t launch_mfma_step(const StepArgs &a, hipStream_t s) {
  const size_t lds = mfma_lds_bytes(a.L, a.w);
  const dim3 grid((a.batch + kMfRows - 1) / kMfRows), block(kMfThreads);
  if (a.w == 3) hipLaunchKernelGGL(mf::mfma_step_kernel<2>, grid, block, lds, s, a);
  else hipLaunchKernelGGL(mf::mfma_step_kernel<1>, grid, block, lds, s, a);
  return hipGetLastError();
}

hipError_t set_mfma_lds_limit(size_t bytes) {
  hipError_t e = hipFuncSetAttribute((const void *)mf::mfma_step_kernel<1>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)bytes);
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute((const void *)mf::mfma_step_kernel<2>, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)bytes);
}

// ---------------------------------------------------------------------------
// Repacking into per-wave fragment streams.  Fragment (tile t, k-step ks) of a
// matrix M[out][k] gives lane l the 8 values M[16t + l%16][32ks + 8(l/16) + j].
// Stage k of the stream holds, for each of the 8 waves, F fragments of 1 KB.
namespace mf {

// element (output o, input channel c, tap j) of the conv weights [2R][R][w] (tap w - 1 multiplies the
// current input, tap w - 2 the input d steps back, tap 0 at width 3 the input 2d steps back)
__device__ __forceinline__ uint16_t conv_elem(const uint16_t *conv, int w, int o, int c, int j) {
  return conv[(o * R + c) * w + j];
}

__device__ __forceinline__ uint4 pack8(const uint16_t *v) {
  return make_uint4(v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16), v[6] | (v[7] << 16));
}

// Layer l's fragments.  Wave A (p = wave < 4), stage l: f0..f3 the conv's current-input tap (tanh
// tile p k-steps 0,1, sigmoid tile p k-steps 0,1), f4..f5 residual tile p, f6..f8 skip tiles 8p..8p+2 k-step 0,
// f9..f11 the same tiles k-step 1, f12 skip tile 8p+3 k-step 0.  Wave B (p = wave - 4), stage l:
// f4 skip tile 8p+3 k-step 1, f5..f8 skip tiles 8p+4..8p+7 k-step 0, f9..f12 k-step 1; the conv
// tap d steps back of layer l (tanh tile p k-steps 0,1, sigmoid tile p k-steps 0,1) goes to f0..f3 of stage
// l - 1, or for layer 0 to the last head stage (head stream positions GCV..GCV+3).  The last
// layer also zeroes its own wave-B f0..f3 (no next layer inside the step).  Width 3: the same four
// fragments of the oldest tap go to the tap stream after the stage streams, [l][p][f].
__global__ void repack_layer_kernel(const uint16_t *conv, const uint16_t *res, const uint16_t *skip, int l, int L,
                                    int w, uint4 *frags) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= kMfWaves * F * 64) return;
  const int lane = e % 64, f = (e / 64) % F, wv = e / (64 * F);
  const int m = lane % 16, kq = 8 * (lane / 16);
  const int NS = L + NHEAD;
  auto at = [&](int stage, int wave, int frag) {
    return frags + ((size_t)(stage * kMfWaves + wave) * F + frag) * 64 + lane;
  };
  uint16_t v[8];
  if (wv < 4) {
    const int p = wv;
    for (int j = 0; j < 8; ++j) {
      if (f < 4) {
        const int o = (f < 2 ? 0 : R) + 16 * p + m;
        v[j] = conv_elem(conv, w, o, 32 * (f & 1) + kq + j, w - 1);
      } else if (f < 6) {
        v[j] = res[(16 * p + m) * R + 32 * (f - 4) + kq + j];
      } else {
        const int t = f < 9 ? 8 * p + (f - 6) : f < 12 ? 8 * p + (f - 9) : 8 * p + 3;
        const int ks = (f >= 9 && f < 12) ? 1 : 0;
        v[j] = skip[(16 * t + m) * R + 32 * ks + kq + j];
      }
    }
    *at(l, wv, f) = pack8(v);
  } else {
    const int p = wv - 4;
    if (f < 4) {
      const int o = (f < 2 ? 0 : R) + 16 * p + m;
      for (int j = 0; j < 8; ++j) v[j] = conv_elem(conv, w, o, 32 * (f & 1) + kq + j, w - 2);
      if (l > 0) *at(l - 1, wv, f) = pack8(v);
      else *at(NS - 1, wv, GCV - F * (NHEAD - 1) + f) = pack8(v);
      if (l == L - 1) *at(l, wv, f) = make_uint4(0, 0, 0, 0);
      if (w == 3) {
        for (int j = 0; j < 8; ++j) v[j] = conv_elem(conv, w, o, 32 * (f & 1) + kq + j, 0);
        uint4 *tap = frags + mfma_frag_bytes(L) / 16;
        tap[((size_t)(l * 4 + p) * 4 + f) * 64 + lane] = pack8(v);
      }
    } else {
      for (int j = 0; j < 8; ++j) {
        const int t = f == 4 ? 8 * p + 3 : f < 9 ? 8 * p + 4 + (f - 5) : 8 * p + 4 + (f - 9);
        const int ks = (f == 4 || f >= 9) ? 1 : 0;
        v[j] = skip[(16 * t + m) * R + 32 * ks + kq + j];
      }
      *at(l, wv, f) = pack8(v);
    }
  }
}

// Head stages L .. L+7.  Wave stream g = 13 h + f: g < 64 first 1x1 tile (8p + g%4, wave B
// 8p + 4 + g%4) k-step g/4; 64 <= g < 96 output tile (4p + (g-64)%2, wave B 4p + 2 + ...) k-step
// (g-64)/2; the rest zero, except wave B's GCV..GCV+3 (layer 0's v-half, written by the layer
// repack and left alone here).
__global__ void repack_head_kernel(const uint16_t *head, const uint16_t *out, int L, uint4 *frags) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= NHEAD * kMfWaves * F * 64) return;
  const int lane = e % 64, f = (e / 64) % F, w = (e / (64 * F)) % kMfWaves, st = e / (64 * F * kMfWaves);
  const int m = lane % 16, kq = 8 * (lane / 16);
  const int g = F * st + f;
  const bool isA = w < 4;
  const int p = w & 3;
  if (!isA && g >= GCV && g < GCV + 4) return;
  uint16_t v[8];
  for (int j = 0; j < 8; ++j) {
    if (g < GH1) {
      const int t = 8 * p + (isA ? 0 : 4) + g % 4, ks = g / 4;
      v[j] = head[(16 * t + m) * S + 32 * ks + kq + j];
    } else if (g < GOUT) {
      const int t = 4 * p + (isA ? 0 : 2) + (g - GH1) % 2, ks = (g - GH1) / 2;
      v[j] = out[(16 * t + m) * H + 32 * ks + kq + j];
    } else {
      v[j] = 0;
    }
  }
  frags[((size_t)((L + st) * kMfWaves + w) * F + f) * 64 + lane] = pack8(v);
}

__global__ void embed_table_kernel(const uint16_t *embed, uint16_t *dst) {
  // dst [Q][R] from embed [R][Q]
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= Q * R) return;
  const int qq = e / R, ch = e % R;
  dst[e] = embed[ch * Q + qq];
}

// bias block: conv_b [L][2R], res_b [L][R], skip_sum [S] (sum over layers in layer order),
// head_b [H], out_b [Q], emb_b [R]
__global__ void bias_block_kernel(const float *const *conv_b, const float *const *res_b,
                                  const float *const *skip_b, const float *head_b, const float *out_b,
                                  const float *emb_b, int L, float *dst) {
  const int n = L * 3 * R + S + H + Q + R;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
    float v = 0.f;
    if (i < L * 2 * R) {
      const float *b = conv_b[i / (2 * R)];
      v = b ? b[i % (2 * R)] : 0.f;
    } else if (i < L * 3 * R) {
      const int j = i - L * 2 * R;
      const float *b = res_b[j / R];
      v = b ? b[j % R] : 0.f;
    } else if (i < L * 3 * R + S) {
      const int k = i - L * 3 * R;
      for (int l = 0; l < L; ++l) v += skip_b[l] ? skip_b[l][k] : 0.f;
    } else if (i < L * 3 * R + S + H) {
      v = head_b ? head_b[i - L * 3 * R - S] : 0.f;
    } else if (i < L * 3 * R + S + H + Q) {
      v = out_b ? out_b[i - L * 3 * R - S - H] : 0.f;
    } else {
      v = emb_b ? emb_b[i - L * 3 * R - S - H - Q] : 0.f;
    }
    dst[i] = v;
  }
}

}  // namespace mf

hipError_t launch_mfma_repack_layer(const void *conv, const void *res, const void *skip, int l, int L, int w,
                                    void *frags, hipStream_t s) {
  const int n = kMfWaves * kMfFrags * 64;
  hipLaunchKernelGGL(mf::repack_layer_kernel, dim3((n + 255) / 256), dim3(256), 0, s, (const uint16_t *)conv,
                     (const uint16_t *)res, (const uint16_t *)skip, l, L, w, (uint4 *)frags);
  return hipGetLastError();
}

hipError_t launch_mfma_repack_head(const void *head, const void *out, int L, void *frags, hipStream_t s) {
  const int n = kMfHeadStages * kMfWaves * kMfFrags * 64;
  hipLaunchKernelGGL(mf::repack_head_kernel, dim3((n + 255) / 256), dim3(256), 0, s, (const uint16_t *)head,
                     (const uint16_t *)out, L, (uint4 *)frags);
  return hipGetLastError();
}

hipError_t launch_mfma_embed_table(const void *embed, void *dst, hipStream_t s) {
  const int n = 256 * kMfR;
  hipLaunchKernelGGL(mf::embed_table_kernel, dim3((n + 255) / 256), dim3(256), 0, s, (const uint16_t *)embed,
                     (uint16_t *)dst);
  return hipGetLastError();
}

hipError_t launch_mfma_bias_block(const float *const *conv_b, const float *const *res_b, const float *const *skip_b,
                                  const float *head_b, const float *out_b, const float *emb_b, int L, float *dst,
                                  hipStream_t s) {
  hipLaunchKernelGGL(mf::bias_block_kernel, dim3(64), dim3(256), 0, s, conv_b, res_b, skip_b, head_b, out_b, emb_b, L,
                     dst);
  return hipGetLastError();
}

}  // namespace fwg
