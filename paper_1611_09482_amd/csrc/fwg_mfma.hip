// MFMA step kernel for gated stacks with bf16 operands, R = 64 residual
// channels, S = H = 512 skip/head channels and 256 classes (gfx950,
// v_mfma_f32_16x16x32_bf16, fp32 accumulation).
//
// One block of 4 waves owns 16 independent streams; one launch runs n_steps
// whole generation steps.  Per step and layer (paper Section 2.2): pop the
// layer's queue (the state pushed d_l steps earlier), compute the dilated
// width-2 product [W_r W_e] [v; x], the gate, the residual and skip 1x1
// products, then push the layer's input into the slot just popped.  After the
// last layer: relu(skip sum) -> 1x1 -> relu -> 1x1 -> logits, softmax and the
// inverse-CDF sample, which becomes the next step's input (Section 1).
//
// Products are computed transposed, D[channel][stream] = W[channel][k] X[stream][k]:
// weights are the MFMA A operand (16 output channels x 32 k), activations the B
// operand (32 k x 16 streams).  Each lane then holds 4 consecutive channels of
// one stream, so activation tiles move to and from LDS as 8- and 16-byte rows.
//
// Weights are streamed from L2: every wave reads its own pre-packed fragment
// sequence, one "stage" (a layer: 26 fragments; a head chunk: 16 fragments) at a
// time: as soon as a fragment register has fed its MFMA it is refilled with the
// same fragment of the next stage, so about one stage of loads is always in
// flight (every stage is 26 fragments, the head padded to whole stages, so the
// refill pattern is the same on every path).  Queue reads for stage i+2 are
// issued at the start of stage i and land in LDS at the end of stage i+1.  A lane that pushes a queue row is the
// lane that later pops it, so queue traffic needs no cross-wave ordering.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fwg_internal.h"

namespace fwg {
namespace mf {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f32x4 mfma(const u32x4 &a, const u32x4 &b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0,
                                                0, 0);
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
// two floats -> two bf16 (round to nearest even; one v_cvt_pk_bf16_f32 on gfx950)
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  const bf16x2 p = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, p);
}
__device__ __forceinline__ u32x2 pack4(const f32x4 &v) { return u32x2{pack2(v[0], v[1]), pack2(v[2], v[3])}; }
__device__ __forceinline__ float bf_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

__device__ __forceinline__ float sigmoidf_(float x) { return 1.f / (1.f + __expf(-x)); }
// tanh(a) * sigmoid(g) with one exp and one reciprocal each: tanh(a) = 1 - 2 / (exp(2a) + 1)
// (absolute error ~1e-7, far below the bf16 rounding this value goes through next)
__device__ __forceinline__ float gate(float a, float g) {
  const float t = 1.f - 2.f * __builtin_amdgcn_rcpf(__expf(2.f * a) + 1.f);
  return t * __builtin_amdgcn_rcpf(1.f + __expf(-g));
}

__device__ __forceinline__ u32x4 lds16(const uint16_t *p) { return *(const u32x4 *)p; }
__device__ __forceinline__ void lds8(uint16_t *p, u32x2 v) { *(u32x2 *)p = v; }
__device__ __forceinline__ f32x4 ldsf4(const float *p) {
  const float4 v = *(const float4 *)p;
  return f32x4{v.x, v.y, v.z, v.w};
}

// Inverse-CDF sample of one row of 256 logits by one wavefront (see fwg_kernels.hip).
__device__ __forceinline__ int sample256(const float *lg, float u) {
  const int lane = threadIdx.x & 63;
  const float4 l4 = *(const float4 *)(lg + 4 * lane);
  float m = fmaxf(fmaxf(l4.x, l4.y), fmaxf(l4.z, l4.w));
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off, 64));
  const float e0 = __expf(l4.x - m), e1 = __expf(l4.y - m), e2 = __expf(l4.z - m), e3 = __expf(l4.w - m);
  const float c0 = e0, c1 = c0 + e1, c2 = c1 + e2, c3 = c2 + e3;
  float incl = c3;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const float v = __shfl_up(incl, off, 64);
    if (lane >= off) incl += v;
  }
  float excl = __shfl_up(incl, 1, 64);
  if (lane == 0) excl = 0.f;
  const float Z = __shfl(excl + c3, 63, 64);
  const float target = u * Z;
  int first = 4;
  if (target < excl + c3) first = 3;
  if (target < excl + c2) first = 2;
  if (target < excl + c1) first = 1;
  if (target < excl + c0) first = 0;
  const unsigned long long hit = __ballot(first < 4);
  if (hit == 0ull) return 255;
  const int src = __ffsll((long long)hit) - 1;
  return 4 * src + __shfl(first, src, 64);
}

// ---------------------------------------------------------------------------
// Shapes and LDS layout (elements; activations bf16 with 8-element row padding)
constexpr int R = kMfR, S = kMfS, H = kMfH, Q = 256, ROWS = kMfRows;
constexpr int PX = R + 8;   // 64-channel activation rows
constexpr int PS = S + 8;   // 512-channel activation rows (skip / head hidden)
constexpr int PL = Q + 4;   // fp32 logits rows
constexpr int F = kMfFrags, NHEAD = kMfHeadStages;
// per-wave head fragment stream, k-step major: first 1x1 (g < G1: tile 8w + g%8, k-step g/8),
// output 1x1 (G1 <= g < G2: tile 4w + (g-G1)%4, k-step (g-G1)/4), then zero padding
constexpr int G1 = 128, G2 = 192;
constexpr int KCH = 64;  // steps per chunk of per-step inputs staged in LDS

struct Lds {
  uint16_t vbuf[2][ROWS * PX];
  uint16_t xbuf[2][ROWS * PX];
  uint16_t zbuf[ROWS * PX];
  uint16_t hbuf[ROWS * PS];
  union {
    uint16_t sbuf[ROWS * PS];
    float lg[ROWS * PL];
  } u;
  uint16_t embT[Q * R];  // embedding table, [class][channel]
  // per-step inputs of the block's streams for a chunk of KCH steps: uniforms (generation) or the
  // next forced input (teacher forcing), loaded once per chunk
  union {
    float u[ROWS][KCH];
    int in[ROWS][KCH];
  } chunk;
  int ins[ROWS];
  int pad_[ROWS];
  // followed by the per-layer tables (dynamic part): roff[L] (int64), slot[L], dil[L], then fp32 biases
};

__host__ __device__ constexpr size_t lds_fixed_bytes() { return (sizeof(Lds) + 15) & ~size_t(15); }
// dynamic part: roff[L] (8 B), slot[L], dil[L] (4 B each), then the bias block at a 16-byte boundary
__host__ __device__ inline size_t lds_dyn_bias_offset(int L) { return ((size_t)L * 16 + 15) & ~size_t(15); }

struct Frags {
  u32x4 f[F];
};

// Stage k of a step is layer k (k < L) or head chunk k - L; every stage is F fragments per wave.
struct Ctx {
  const StepArgs *a;
  Lds *s;
  int *slot, *dil;
  const long long *roff;
  const float *conv_b, *res_b, *skip_sum, *head_b, *out_b, *emb_b;
  __amdgpu_buffer_rsrc_t wrsrc;  // buffer resource over the fragment streams
  int wvoff;                     // this lane's byte offset inside a fragment (16 * lane)
  int L, NS, w, lane, n, q, b0, nrows;
};

// Byte offset (wave-uniform) of stage k's fragment stream for this wave: stage-major, 4 waves
// per stage, F fragments of 1 KB each.
__device__ __forceinline__ int stage_off(const Ctx &c, int k) { return (k * 4 + c.w) * F * 1024; }
__device__ __forceinline__ u32x4 load_frag(const Ctx &c, int off, int f) {
  return __builtin_amdgcn_raw_buffer_load_b128(c.wrsrc, c.wvoff, off + f * 1024, 0);
}
// Slot f has just been consumed: start loading the same slot of the next stage.
// The scheduling barrier keeps the compiler from hoisting the load above the MFMA that still
// reads the slot's previous contents (which would keep both copies live).
__device__ __forceinline__ void refill(const Ctx &c, Frags &W, int nx, int f) {
  __builtin_amdgcn_sched_barrier(0);
  W.f[f] = load_frag(c, nx, f);
  __builtin_amdgcn_sched_barrier(0);
}

__device__ __forceinline__ void load_stage(const Ctx &c, int k, Frags &fr) {
  const int off = stage_off(c, k);
#pragma unroll
  for (int f = 0; f < F; ++f) fr.f[f] = load_frag(c, off, f);
}

// Queue row a lane moves: stream row 4w + (lane%32)/8, 16-byte chunk lane%8 (lanes 32..63 mirror
// lanes 0..31 on loads and skip the stores).
__device__ __forceinline__ long long ring_elem(const Ctx &c, int l, int slotv) {
  const int r = 4 * c.w + ((c.lane & 31) >> 3);
  return c.roff[l] + ((long long)slotv * c.a->bmax + (c.b0 + r)) * R + 8 * (c.lane & 7);
}

// Issue the pop of stage k (a layer) for step offset `ahead` (0: the step the slot table
// describes, 1: the next one).  Head stages pop layer 0 as a harmless placeholder.
__device__ __forceinline__ u32x4 pop_issue(const Ctx &c, int k, int ahead) {
  const int l = k < c.L ? k : 0;
  int sl = c.slot[l] + ahead;
  if (sl >= c.dil[l]) sl -= c.dil[l];
  const uint16_t *ring = (const uint16_t *)c.a->ring;
  return __builtin_nontemporal_load((const u32x4 *)(ring + ring_elem(c, l, sl)));
}
__device__ __forceinline__ void pop_land(const Ctx &c, int parity, u32x4 v) {
  if (c.lane < 32) {
    const int r = 4 * c.w + (c.lane >> 3);
    *(u32x4 *)(c.s->vbuf[parity] + r * PX + 8 * (c.lane & 7)) = v;
  }
}

// Accumulators.  acc[] holds, in turn, the skip sum (layers; channels 128w + 16j + 4q + i),
// the first head 1x1's pre-activation (same channels) and the logits (acc[0..3], classes
// 64w + 16j + 4q + i).
struct Acc {
  f32x4 xres;  // residual stream: channels 16w + 4q + i of stream n
  f32x4 acc[8];
};

// One layer stage.  `par` = stage parity (selects vbuf); xbuf parity follows the layer index.
__device__ __forceinline__ void run_layer(const Ctx &c, int l, int par, Frags &W, int nx, Acc &A) {
  Lds &s = *c.s;
  const int n = c.n, q = c.q, w = c.w;
  u32x4 bx0, bx1;
  if (l == 0) {
    // embedding (current input h^0_e): row gather of the transposed 1x1 convolution plus bias
    const int in = s.ins[n];
    const uint16_t *e = s.embT + in * R;
    const u32x4 r0 = lds16(e + 8 * q), r1 = lds16(e + 32 + 8 * q);
    const float *eb = c.emb_b;
    auto cvt = [&](u32x4 raw, int k0) {
      u32x4 p;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        p[j] = pack2(bf_lo(raw[j]) + eb[k0 + 2 * j], bf_hi(raw[j]) + eb[k0 + 2 * j + 1]);
      return p;
    };
    bx0 = cvt(r0, 8 * q);
    bx1 = cvt(r1, 32 + 8 * q);
    // this wave's residual tile and its bf16 copy (pushed into queue 0 below)
    const int ch = 16 * w + 4 * q;
    const u32x2 raw = *(const u32x2 *)(e + ch);
    A.xres = f32x4{bf_lo(raw.x) + eb[ch], bf_hi(raw.x) + eb[ch + 1], bf_lo(raw.y) + eb[ch + 2],
                   bf_hi(raw.y) + eb[ch + 3]};
    lds8(s.xbuf[0] + n * PX + ch, pack4(A.xres));
#pragma unroll
    for (int j = 0; j < 8; ++j) A.acc[j] = ldsf4(c.skip_sum + 128 * w + 16 * j + 4 * q);
  } else {
    const uint16_t *xb = s.xbuf[l & 1] + n * PX;
    bx0 = lds16(xb + 8 * q);
    bx1 = lds16(xb + 32 + 8 * q);
  }
  const uint16_t *vb = s.vbuf[par] + n * PX;
  const u32x4 bv0 = lds16(vb + 8 * q), bv1 = lds16(vb + 32 + 8 * q);
  // dilated width-2 product: output rows 16w.. (tanh half) and 64 + 16w.. (sigmoid half)
  const float *cb = c.conv_b + l * 2 * R;
  f32x4 af = ldsf4(cb + 16 * w + 4 * q), ag = ldsf4(cb + R + 16 * w + 4 * q);
  af = mfma(W.f[0], bv0, af);
  ag = mfma(W.f[4], bv0, ag);
  af = mfma(W.f[1], bv1, af);
  ag = mfma(W.f[5], bv1, ag);
  af = mfma(W.f[2], bx0, af);
  ag = mfma(W.f[6], bx0, ag);
  af = mfma(W.f[3], bx1, af);
  ag = mfma(W.f[7], bx1, ag);
#pragma unroll
  for (int f = 0; f < 8; ++f) refill(c, W, nx, f);
  f32x4 z;
#pragma unroll
  for (int i = 0; i < 4; ++i) z[i] = gate(af[i], ag[i]);
  lds8(s.zbuf + n * PX + 16 * w + 4 * q, pack4(z));
  __syncthreads();
  // push phase: the layer's input x^{l-1}_t replaces the slot popped for this step
  if (c.lane < 32) {
    const int r = 4 * w + (c.lane >> 3);
    const u32x4 v = *(const u32x4 *)(s.xbuf[l & 1] + r * PX + 8 * (c.lane & 7));
    uint16_t *ring = (uint16_t *)c.a->ring;
    __builtin_nontemporal_store(v, (u32x4 *)(ring + ring_elem(c, l, c.slot[l])));
  }
  const uint16_t *zb = s.zbuf + n * PX;
  const u32x4 bz0 = lds16(zb + 8 * q), bz1 = lds16(zb + 32 + 8 * q);
  // residual 1x1
  f32x4 xr = A.xres + ldsf4(c.res_b + l * R + 16 * w + 4 * q);
  xr = mfma(W.f[8], bz0, xr);
  xr = mfma(W.f[9], bz1, xr);
  refill(c, W, nx, 8);
  refill(c, W, nx, 9);
  A.xres = xr;
  lds8(s.xbuf[(l + 1) & 1] + n * PX + 16 * w + 4 * q, pack4(xr));
  // skip 1x1, accumulated over layers (k-step major: consecutive MFMAs use different accumulators)
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    A.acc[j] = mfma(W.f[10 + j], bz0, A.acc[j]);
    refill(c, W, nx, 10 + j);
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    A.acc[j] = mfma(W.f[18 + j], bz1, A.acc[j]);
    refill(c, W, nx, 18 + j);
  }
}

// Head chunk C: fragments g = 26C .. 26C+25 of the head stream.
template <int C>
__device__ __forceinline__ void run_head(const Ctx &c, Frags &W, int nx, Acc &A) {
  Lds &s = *c.s;
  const int n = c.n, q = c.q, w = c.w;
  if (C == 0) {
    // relu(skip sum) becomes the first head 1x1's input
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      f32x4 r;
#pragma unroll
      for (int i = 0; i < 4; ++i) r[i] = fmaxf(A.acc[j][i], 0.f);
      lds8(s.u.sbuf + n * PS + 128 * w + 16 * j + 4 * q, pack4(r));
      A.acc[j] = ldsf4(c.head_b + 128 * w + 16 * j + 4 * q);
    }
    __syncthreads();
  }
  u32x4 b = u32x4{0, 0, 0, 0};
#pragma unroll
  for (int f = 0; f < F; ++f) {
    const int g = F * C + f;
    if (g < G1) {
      const int ks = g / 8, j = g % 8;
      if (j == 0 || f == 0) b = lds16(s.u.sbuf + n * PS + 32 * ks + 8 * q);
      A.acc[j] = mfma(W.f[f], b, A.acc[j]);
    } else if (g < G2) {
      if (g == G1) {
        // relu(head hidden) becomes the output 1x1's input
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          f32x4 r;
#pragma unroll
          for (int i = 0; i < 4; ++i) r[i] = fmaxf(A.acc[j][i], 0.f);
          lds8(s.hbuf + n * PS + 128 * w + 16 * j + 4 * q, pack4(r));
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) A.acc[j] = ldsf4(c.out_b + 64 * w + 16 * j + 4 * q);
        __syncthreads();
      }
      const int ks = (g - G1) / 4, j = (g - G1) % 4;
      if (j == 0 || f == 0) b = lds16(s.hbuf + n * PS + 32 * ks + 8 * q);
      A.acc[j] = mfma(W.f[f], b, A.acc[j]);
    }
    refill(c, W, nx, f);
  }
}

// Stage the per-step inputs of steps [s0, s0 + KCH) in LDS: the uniform of (row r, step s) for
// generation, the input of step s + 1 for teacher forcing.  Called by all threads once per chunk
// (in the first head stage, before its barrier); waiting for these loads here keeps every other
// wait in the step loop precise.
__device__ __forceinline__ void stage_chunk(const Ctx &c, long long s0) {
  const StepArgs &a = *c.a;
  Lds &s = *c.s;
  for (int i = threadIdx.x; i < ROWS * KCH; i += kThreads) {
    const int r = i / KCH, j = i % KCH;
    const long long st = s0 + j;
    if (a.forced) {
      int v = 0;
      if (r < c.nrows && st + 1 < a.n_steps) v = a.inputs[(long long)(c.b0 + r) * a.n_steps + st + 1];
      s.chunk.in[r][j] = v;
    } else {
      float v = 0.f;
      if (r < c.nrows && st < a.n_steps) v = a.uniforms[(long long)(c.b0 + r) * a.n_steps + st];
      s.chunk.u[r][j] = v;
    }
  }
}

// End of a step: logits to LDS, sample (or write logits), next inputs, queue slots advance.
__device__ __forceinline__ void finish_step(const Ctx &c, long long step, Acc &A) {
  Lds &s = *c.s;
  const StepArgs &a = *c.a;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    *(float4 *)(s.u.lg + c.n * PL + 64 * c.w + 16 * j + 4 * c.q) =
        make_float4(A.acc[j][0], A.acc[j][1], A.acc[j][2], A.acc[j][3]);
  __syncthreads();
  const int tid = threadIdx.x;
  if (a.forced) {
    for (int r = c.w; r < c.nrows; r += 4) {
      const float4 v = *(const float4 *)(s.u.lg + r * PL + 4 * c.lane);
      *(float4 *)(a.logits + ((long long)(c.b0 + r) * a.n_steps + step) * Q + 4 * c.lane) = v;
    }
    if (tid < c.nrows && step + 1 < a.n_steps) s.ins[tid] = s.chunk.in[tid][step % KCH];
  } else {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int r = c.w + 4 * kk;
      if (r >= c.nrows) break;
      const int k = sample256(s.u.lg + r * PL, s.chunk.u[r][step % KCH]);
      if (c.lane == 0) {
        a.samples[(long long)(c.b0 + r) * a.n_steps + step] = k;
        s.ins[r] = k;
      }
    }
  }
  for (int l = tid; l < c.L; l += kThreads) {
    const int nx = c.slot[l] + 1;
    c.slot[l] = nx == c.dil[l] ? 0 : nx;
  }
  __syncthreads();
}

// Stage position helpers.
struct Pos {
  long long step;
  int k;
};
__device__ __forceinline__ Pos advance(const Ctx &c, Pos p, int m) {
  p.k += m;
  if (p.k >= c.NS) { p.k -= c.NS; p.step += 1; }
  return p;
}

__device__ __forceinline__ void run_stage(const Ctx &c, Pos p, int par, Frags &W, int nx, Acc &A) {
  if (p.k < c.L) {
    run_layer(c, p.k, par, W, nx, A);
  } else {
    switch (p.k - c.L) {
      case 0:
        if (p.step % KCH == 0) stage_chunk(c, p.step);
        run_head<0>(c, W, nx, A);
        break;
      case 1: run_head<1>(c, W, nx, A); break;
      case 2: run_head<2>(c, W, nx, A); break;
      case 3: run_head<3>(c, W, nx, A); break;
      case 4: run_head<4>(c, W, nx, A); break;
      case 5: run_head<5>(c, W, nx, A); break;
      case 6: run_head<6>(c, W, nx, A); break;
      default: run_head<7>(c, W, nx, A); break;
    }
  }
  if (p.k == c.NS - 1) finish_step(c, p.step, A);
}

__global__ void __launch_bounds__(kThreads) mfma_step_kernel(StepArgs a) {
  extern __shared__ float4 lds_raw[];
  Lds &s = *(Lds *)lds_raw;
  const int tid = threadIdx.x;
  const int L = a.L;
  char *dyn = (char *)lds_raw + lds_fixed_bytes();
  long long *roff = (long long *)dyn;
  int *slot = (int *)(roff + L);
  int *dil = slot + L;
  // conv_b [L][2R], res_b [L][R], skip_sum [S], head_b [H], out_b [Q], emb_b [R]; 16-byte aligned
  float *bias = (float *)(dyn + lds_dyn_bias_offset(L));

  Ctx c;
  c.a = &a;
  c.s = &s;
  c.slot = slot;
  c.dil = dil;
  c.roff = roff;
  c.conv_b = bias;
  c.res_b = c.conv_b + L * 2 * R;
  c.skip_sum = c.res_b + L * R;
  c.head_b = c.skip_sum + S;
  c.out_b = c.head_b + H;
  c.emb_b = c.out_b + Q;
  c.L = L;
  c.NS = L + NHEAD;
  c.w = tid >> 6;
  c.lane = tid & 63;
  c.n = c.lane & 15;
  c.q = c.lane >> 4;
  c.b0 = blockIdx.x * ROWS;
  c.nrows = min(ROWS, a.batch - c.b0);
  c.w = __builtin_amdgcn_readfirstlane(c.w);
  c.wrsrc = __builtin_amdgcn_make_buffer_rsrc((void *)a.mf_frags, (short)0, mfma_frag_bytes(L), 0x00020000);
  c.wvoff = 16 * c.lane;

  // tables: embedding [Q][R], biases, queue offsets, dilations and slots
  const u32x4 *embsrc = (const u32x4 *)a.mf_embT;
  for (int i = tid; i < Q * R / 8; i += kThreads) ((u32x4 *)s.embT)[i] = embsrc[i];
  const int nbias = L * 3 * R + S + H + Q + R;
  for (int i = tid; i < nbias; i += kThreads) bias[i] = a.mf_bias[i];
  for (int l = tid; l < L; l += kThreads) {
    const LayerDev ld = a.layers[l];
    roff[l] = ld.ring_off;
    dil[l] = ld.dil;
    slot[l] = (int)(a.t0 % (long long)ld.dil);
  }
  if (tid < ROWS) {
    int v = 0;
    if (tid < c.nrows) v = a.forced ? a.inputs[(long long)(c.b0 + tid) * a.n_steps] : a.last[c.b0 + tid];
    s.ins[tid] = v;
  }
  __syncthreads();

  const long long total = (long long)a.n_steps * c.NS;
  Acc A;
  Frags W;  // one stage of fragments; each slot is refilled with the next stage's right after use
  Pos p0{0, 0};
  // prologue: stage 0's queue rows land now, stage 1's are in flight; stage 0's weights
  pop_land(c, 0, pop_issue(c, 0, 0));
  u32x4 vA, vB = pop_issue(c, 1 < L ? 1 : 0, 0);
  load_stage(c, 0, W);
  __syncthreads();

  for (long long i = 0; i < total; i += 2) {
    const Pos p1 = advance(c, p0, 1), p2 = advance(c, p0, 2), p3 = advance(c, p0, 3);
    // ---- even stage: queue rows of stage i+2 in flight into vA, rows of stage i+1 land
    vA = pop_issue(c, p2.k, (int)(p2.step - p0.step));
    __builtin_amdgcn_sched_barrier(0);  // issue the queue read before this stage's refills
    run_stage(c, p0, (int)(i & 1), W, stage_off(c, p1.k), A);
    if (p1.k < L && i + 1 < total) pop_land(c, (int)((i + 1) & 1), vB);
    __syncthreads();
    if (i + 1 >= total) break;
    // ---- odd stage: rows of stage i+3 in flight into vB, rows of stage i+2 land
    vB = pop_issue(c, p3.k, (int)(p3.step - p1.step));
    __builtin_amdgcn_sched_barrier(0);
    run_stage(c, p1, (int)((i + 1) & 1), W, stage_off(c, p2.k), A);
    if (p2.k < L && i + 2 < total) pop_land(c, (int)(i & 1), vA);
    __syncthreads();
    p0 = p2;
  }
  if (!a.forced && tid < c.nrows) a.last[c.b0 + tid] = s.ins[tid];
}

}  // namespace mf

size_t mfma_lds_bytes(int L) {
  return mf::lds_fixed_bytes() + mf::lds_dyn_bias_offset(L) + sizeof(float) * mfma_bias_floats(L);
}

hipError_t launch_mfma_step(const StepArgs &a, hipStream_t s) {
  const size_t lds = mfma_lds_bytes(a.L);
  const dim3 grid((a.batch + kMfRows - 1) / kMfRows), block(kThreads);
  hipLaunchKernelGGL(mf::mfma_step_kernel, grid, block, lds, s, a);
  return hipGetLastError();
}

hipError_t set_mfma_lds_limit(size_t bytes) {
  return hipFuncSetAttribute((const void *)mf::mfma_step_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)bytes);
}

// ---------------------------------------------------------------------------
// Repacking into per-wave fragment streams.  Fragment (tile t, k-step ks) of a
// matrix M[out][k] gives lane l the 8 values M[16t + l%16][32ks + 8(l/16) + j].
namespace mf {

// element of the conv matrix [2R][2R] with k < R the recurrent tap and k >= R the current tap
__device__ __forceinline__ uint16_t conv_elem(const uint16_t *conv, int o, int k) {
  return conv[(o * R + (k % R)) * 2 + (k >= R ? 1 : 0)];
}

__global__ void repack_layer_kernel(const uint16_t *conv, const uint16_t *res, const uint16_t *skip, uint4 *dst) {
  // dst: this layer's stage, 4 waves x F fragments x 64 lanes x 8 elements
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= 4 * F * 64) return;
  const int lane = e % 64, f = (e / 64) % F, w = e / (64 * F);
  const int m = lane % 16, kq = 8 * (lane / 16);
  uint16_t v[8];
  for (int j = 0; j < 8; ++j) {
    int o, k;
    if (f < 8) {
      const int t = f < 4 ? w : 4 + w, ks = f % 4;
      o = 16 * t + m;
      k = 32 * ks + kq + j;
      v[j] = conv_elem(conv, o, k);
    } else if (f < 10) {
      o = 16 * w + m;
      k = 32 * (f - 8) + kq + j;
      v[j] = res[o * R + k];
    } else {
      const int jj = (f - 10) % 8, ks = (f - 10) / 8;
      o = 16 * (8 * w + jj) + m;
      k = 32 * ks + kq + j;
      v[j] = skip[o * R + k];
    }
  }
  dst[e] = make_uint4(v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16), v[6] | (v[7] << 16));
}

__global__ void repack_head_kernel(const uint16_t *head, const uint16_t *out, uint4 *dst) {
  // dst: NHEAD stages of 4 waves x F fragments x 64 lanes; head fragment g = F*stage + f
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= NHEAD * 4 * F * 64) return;
  const int lane = e % 64, f = (e / 64) % F, w = (e / (64 * F)) % 4, st = e / (64 * F * 4);
  const int m = lane % 16, kq = 8 * (lane / 16);
  const int g = F * st + f;
  uint16_t v[8];
  for (int j = 0; j < 8; ++j) {
    if (g < G1) {
      const int t = 8 * w + g % 8, ks = g / 8;
      v[j] = head[(16 * t + m) * S + 32 * ks + kq + j];
    } else if (g < G2) {
      const int t = 4 * w + (g - G1) % 4, ks = (g - G1) / 4;
      v[j] = out[(16 * t + m) * H + 32 * ks + kq + j];
    } else {
      v[j] = 0;
    }
  }
  dst[e] = make_uint4(v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16), v[6] | (v[7] << 16));
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

hipError_t launch_mfma_repack_layer(const void *conv, const void *res, const void *skip, void *dst, hipStream_t s) {
  const int n = 4 * kMfFrags * 64;
  hipLaunchKernelGGL(mf::repack_layer_kernel, dim3((n + 255) / 256), dim3(256), 0, s, (const uint16_t *)conv,
                     (const uint16_t *)res, (const uint16_t *)skip, (uint4 *)dst);
  return hipGetLastError();
}

hipError_t launch_mfma_repack_head(const void *head, const void *out, void *dst, hipStream_t s) {
  const int n = kMfHeadStages * 4 * kMfFrags * 64;
  hipLaunchKernelGGL(mf::repack_head_kernel, dim3((n + 255) / 256), dim3(256), 0, s, (const uint16_t *)head,
                     (const uint16_t *)out, (uint4 *)dst);
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
