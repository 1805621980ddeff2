// HIP kernels of the Fast Wavenet generation library, written for gfx950.
//
// This file holds the general ("VALU") step-kernel family and the small
// utility kernels (weight repacking, fills).  One launch runs n_steps whole
// generation steps for a block of `RPW` independent streams: every step pops
// each layer's queue, runs the generation model (one step of a multi-layer
// RNN, paper Section 2.2, Fig. 4), pushes the new states, computes the output
// distribution and samples the next input (fed back, Section 1).
//
// Layout decisions:
//   * queues: one ring buffer per layer, ring_l[slot][stream][channel] with the
//     channel index contiguous, slot = t mod d_l (Section 2.1: depth = dilation);
//     popping reads the slot written d_l steps earlier, pushing overwrites it
//     after every lane has read it (pop before push, Section 2.2);
//   * weights: streamed from L2 in a 16-byte K-blocked layout, so consecutive
//     lanes read consecutive 16-byte chunks;
//   * activations of the block's streams: LDS, float32.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "fwg_bf16.h"
#include "fwg_internal.h"
#include "fwg_valu.h"
#include "fwg_sample.h"


namespace fwg {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Direct global-to-LDS copy of 16 bytes per lane (global_load_lds_dwordx4): lane i's bytes come
// from src_wave + lane_off (lane_off = 16 i) and land at LDS byte address lds_dst_wave + 16 i (the
// LDS base wave-uniform; the compiler sets M0 from it).  Consecutive copies issue back to back;
// callers wait for completion (vmcnt) before the data is read.
__device__ __forceinline__ void lds_copy16(const void *src_wave, uint32_t lane_off, const void *lds_dst_wave) {
  __builtin_amdgcn_global_load_lds((const char *)src_wave + lane_off,
                                   (__attribute__((address_space(3))) void *)lds_dst_wave, 16, 0, 0);
}

template <typename WT> struct WTraits;
template <> struct WTraits<float> {
  static constexpr int KB = 4;
  __device__ static __forceinline__ void unpack(u32x4 v, float *w) {
    w[0] = __uint_as_float(v.x); w[1] = __uint_as_float(v.y);
    w[2] = __uint_as_float(v.z); w[3] = __uint_as_float(v.w);
  }
  __device__ static __forceinline__ float load1(const void *p, long long i) { return ((const float *)p)[i]; }
  __device__ static __forceinline__ void store1(void *p, long long i, float v) { ((float *)p)[i] = v; }
  __device__ static __forceinline__ float opnd(float x) { return x; }
};
template <> struct WTraits<uint16_t> {
  static constexpr int KB = 8;
  __device__ static __forceinline__ void unpack(u32x4 v, float *w) {
    w[0] = bf16_lo(v.x); w[1] = bf16_hi(v.x); w[2] = bf16_lo(v.y); w[3] = bf16_hi(v.y);
    w[4] = bf16_lo(v.z); w[5] = bf16_hi(v.z); w[6] = bf16_lo(v.w); w[7] = bf16_hi(v.w);
  }
  __device__ static __forceinline__ float load1(const void *p, long long i) {
    return __uint_as_float(((uint32_t)((const uint16_t *)p)[i]) << 16);
  }
  __device__ static __forceinline__ void store1(void *p, long long i, float v) { ((uint16_t *)p)[i] = bf16_bits(v); }
  __device__ static __forceinline__ float opnd(float x) { return round_bf16(x); }
};

// ---------------------------------------------------------------------------
// Row-block product: part[kg][r][n] = sum over this K-group of W^T[k][n] * A(r, k)
// for r < RPW.  A(r, k) = A0[r*lda0 + k] for k < ksplit, else A1[r*lda1 + k - ksplit].
// N >= 256: each thread owns columns tid, tid+256, ... over all of K (one group).
// N < 256 : 256/N K-groups of N threads each.
// WP: the weight pointer type, a global (address space 1) or an LDS (address space 3) pointer to
// 16-byte vectors, so that staged weights are read with LDS instructions.
typedef __attribute__((address_space(3))) const u32x4 *lds_u4p;
typedef __attribute__((address_space(1))) const u32x4 *glb_u4p;

template <typename WT, int RPW, typename WP>
__device__ __forceinline__ void rows_product(WP W, int K, int N, const float *A0, int lda0,
                                             const float *A1, int lda1, int ksplit, float *part) {
  constexpr int KB = WTraits<WT>::KB;
  const int tid = threadIdx.x;
  const int nkb = K / KB;
  if (N >= kThreads) {
    for (int n = tid; n < N; n += kThreads) {
      float acc[RPW];
#pragma unroll
      for (int r = 0; r < RPW; ++r) acc[r] = 0.f;
      auto kstep = [&](int kb) {
        float w[KB];
        WTraits<WT>::unpack(W[(long long)kb * N + n], w);
        const int k0 = kb * KB;
        const bool lo = k0 < ksplit;
        const float *A = lo ? A0 + k0 : A1 + (k0 - ksplit);
        const int lda = lo ? lda0 : lda1;
#pragma unroll
        for (int r = 0; r < RPW; ++r) {
#pragma unroll
          for (int j = 0; j < KB; ++j) acc[r] = fmaf(w[j], A[r * lda + j], acc[r]);
        }
      };
      // staged (LDS) weights: 16 k-blocks per unrolled body keep more LDS reads in flight
      // (gated fp32 64-stream step 89.9 -> 80.3 us); weights read from L2 keep 4, whose
      // pipelining the compiler does best (16 made the 512-channel ReLU stack 4x slower)
      if constexpr (std::is_same<WP, lds_u4p>::value) {
#pragma unroll 16
        for (int kb = 0; kb < nkb; ++kb) kstep(kb);
      } else {
#pragma unroll 4
        for (int kb = 0; kb < nkb; ++kb) kstep(kb);
      }
#pragma unroll
      for (int r = 0; r < RPW; ++r) part[r * N + n] = acc[r];
    }
  } else {
    const int KG = kThreads / N;
    const int n = tid % N, kg = tid / N;
    const int per = nkb / KG;
    float acc[RPW];
#pragma unroll
    for (int r = 0; r < RPW; ++r) acc[r] = 0.f;
#pragma unroll 4
    for (int i = 0; i < per; ++i) {
      const int kb = kg * per + i;
      float w[KB];
      WTraits<WT>::unpack(W[(long long)kb * N + n], w);
      const int k0 = kb * KB;
      const bool lo = k0 < ksplit;
      const float *A = lo ? A0 + k0 : A1 + (k0 - ksplit);
      const int lda = lo ? lda0 : lda1;
#pragma unroll
      for (int r = 0; r < RPW; ++r) {
#pragma unroll
        for (int j = 0; j < KB; ++j) acc[r] = fmaf(w[j], A[r * lda + j], acc[r]);
      }
    }
#pragma unroll
    for (int r = 0; r < RPW; ++r) part[(kg * RPW + r) * N + n] = acc[r];
  }
}

// Sum of the K-group partials of output (r, n).
template <int RPW>
__device__ __forceinline__ float part_sum(const float *part, int N, int r, int n) {
  const int KG = N >= kThreads ? 1 : kThreads / N;
  float s = 0.f;
  for (int kg = 0; kg < KG; ++kg) s += part[(kg * RPW + r) * N + n];
  return s;
}

__device__ __forceinline__ float bias_or0(const float *b, int i) { return b ? b[i] : 0.f; }


// ---------------------------------------------------------------------------
// The general step kernel.  Block = RPW streams, 256 threads.
//
// Latency hiding: the states a layer pops do not depend on the current step (they were pushed
// at least d steps earlier), so the pops of layer l + 1 -- or of layer 0 of the next step -- are
// loaded into registers while layer l computes and land in the second of two LDS buffers at the
// end of the layer.  When two layers' weights fit in LDS (a.valu_wbytes > 0) the next layer's
// weights and biases are copied into the second weight buffer meanwhile, by direct
// global-to-LDS loads, so a layer's critical path touches LDS only.
typedef __attribute__((address_space(3))) const float *lds_f32p;
typedef __attribute__((address_space(1))) const float *glb_f32p;

// Model shapes known at compile time.  The general kernel reads the shape from its launch
// arguments; at one stream per block a layer is bound by instruction issue, and with the shape as
// constants the index arithmetic folds and fewer values stay live.  Fields: kind (-1: runtime), C,
// Q and w (0: runtime), S and H (-1: runtime).
struct ShapeAny {
  static constexpr int kind = -1, C = 0, S = -1, H = -1, Q = 0, w = 0;
};
template <int KIND, int C_, int S_, int H_, int W_>
struct ShapeFixed {
  static constexpr int kind = KIND, C = C_, S = S_, H = H_, Q = 256, w = W_;
};

template <typename WT, int RPW, bool STAGE, typename SH>
__global__ void __launch_bounds__(kThreads) valu_step_kernel(StepArgs a) {
  extern __shared__ float4 lds_raw[];
  float *lds = (float *)lds_raw;
  const int wfloats = a.valu_wbytes / 4;
  // the model shape: compile-time constants in a specialised instantiation, else launch arguments
  const int kind = SH::kind >= 0 ? SH::kind : a.kind;
  const int C = SH::C ? SH::C : a.C, S = SH::S >= 0 ? SH::S : a.S, H = SH::H >= 0 ? SH::H : a.H;
  const int Q = SH::Q ? SH::Q : a.Q, w = SH::w ? SH::w : a.w, L = a.L;
  const ValuLds lay = valu_lds_layout(kind, C, S, H, Q, L, RPW, w, wfloats);
  float *xf = lds + lay.xf, *xo = lds + lay.xo, *ao = lds + lay.ao;
  float *zo = lds + lay.zo, *so = lds + lay.so, *ho = lds + lay.ho, *h2 = lds + lay.h2;
  float *lg = lds + lay.lg, *partA = lds + lay.partA, *partB = lds + lay.partB;
  // the two buffers of popped states and of staged weights, selected by arithmetic on the LDS base
  // (a pointer array indexed at run time would turn LDS accesses into generic ones)
  auto vbuf = [&](int p) { return lds + (p ? lay.vo2 : lay.vo); };
  auto wbuf = [&](int p) { return (uint4 *)(lds + (p ? lay.wb1 : lay.wb0)); };
  int *slots = (int *)(lds + lay.slots);
  int *ins = (int *)(lds + lay.ins);
  ValuLayer *ltab = (ValuLayer *)(lds + lay.ltab);
  (void)ao;

  const int tid = threadIdx.x;
  const int Co = kind == 2 ? 2 * C : C;
  const int K = w * C;
  const int b0 = blockIdx.x * RPW;
  const int nrows = min(RPW, a.batch - b0);
  if (nrows <= 0) return;
  constexpr bool stage = STAGE;  // the host launches the staging variant iff a.valu_wbytes > 0
  const int nw16 = a.valu_wbytes / 16;       // 16-byte pieces of one layer's staged block
  const int VP = RPW * (w - 1) * C;          // popped elements per layer
  const int es = sizeof(WT);
  // offsets inside a layer's block: conv | res | skip weights, then conv_b | res_b | skip_b
  const size_t o_res = (size_t)K * Co * es, o_skip = o_res + (size_t)C * C * es;
  const size_t o_cb = kind == 2 ? o_skip + (size_t)S * C * es : o_res;
  const size_t o_rb = o_cb + (size_t)Co * 4, o_sb = o_rb + (size_t)C * 4;

  for (int l = tid; l < L; l += kThreads) {
    const LayerDev ld = a.layers[l];
    ValuLayer v;
    v.block = ld.conv;
    v.ring_off = ld.ring_off;
    v.dil = ld.dil;
    v.depth = ld.depth;
    v.pad_[0] = v.pad_[1] = 0;
    ltab[l] = v;
    slots[l] = (int)(a.t0 % (long long)ld.depth);
  }
  if (tid < RPW) {
    int v = 0;
    if (tid < nrows) v = a.mode == MODE_TEACHER ? a.inputs[(long long)(b0 + tid) * a.n_steps] : a.last[b0 + tid];
    ins[tid] = v;
  }
  __syncthreads();

  // prefetch registers of the next layer's popped states
  float pp[kValuPrefPops];
  const uint32_t lane16 = 16u * (uint32_t)(tid & 63);
  // tap k of layer l at the step whose slot is `slot`: the state k d slots after the oldest one;
  // with staging, the layer's weight block is copied straight into weight buffer `par`
  auto fetch = [&](int l, int slot, int par) {
    const ValuLayer ld = ltab[l];
#pragma unroll
    for (int j = 0; j < kValuPrefPops; ++j) {
      const int i = tid + j * kThreads;
      float v = 0.f;
      if (i < VP) {
        const int r = i / ((w - 1) * C), kc = i - r * ((w - 1) * C), k = kc / C, c = kc - k * C;
        int sk = slot + k * ld.dil;
        if (sk >= ld.depth) sk -= ld.depth;
        if (r < nrows)
          v = WTraits<WT>::load1(a.ring, ld.ring_off + (long long)sk * a.bmax * C + (long long)(b0 + r) * C + c);
      }
      pp[j] = v;
    }
    if (stage) {
      // each wave copies 64 consecutive 16-byte pieces per instruction
      const uint4 *src = (const uint4 *)ld.block;
      const int wv = tid >> 6;
#pragma unroll
      for (int j = 0; j < kValuStagePieces; ++j) {
        const int base = j * kThreads + wv * 64;
        if (base < nw16 && (tid & 63) + base < nw16) lds_copy16(src + base, lane16, wbuf(par) + base);
      }
    }
  };
  auto land = [&](int par) {
    float *vb = vbuf(par);
#pragma unroll
    for (int j = 0; j < kValuPrefPops; ++j) {
      const int i = tid + j * kThreads;
      if (i < VP) vb[i] = pp[j];
    }
    // the copies into the weight buffer have completed once the memory counter drains
    if (stage) __builtin_amdgcn_s_waitcnt(0);
  };

  fetch(0, slots[0], 0);
  land(0);
  __syncthreads();
  int par = 0;  // buffer holding the current layer's pops and weights

  for (int s = 0; s < a.n_steps; ++s) {
    // ---- current input (h^0_e) is ins[]: set before the loop and at the end of every step
    // ---- embedding: a row gather of the transposed 1x1 convolution
    for (int i = tid; i < RPW * C; i += kThreads) {
      const int r = i / C, c = i % C;
      const float v = WTraits<WT>::load1(a.embed, (long long)ins[r] * C + c) + bias_or0(a.embed_b, c);
      xf[i] = v;
      xo[i] = WTraits<WT>::opnd(v);
    }
    if (kind == 2)
      for (int i = tid; i < RPW * S; i += kThreads) so[i] = 0.f;
    __syncthreads();

    for (int l = 0; l < L; ++l) {
      const ValuLayer ld = ltab[l];
      // the layer that runs next: layer l + 1 now, or layer 0 at the next step (its slot one on)
      const bool more = l + 1 < L || s + 1 < a.n_steps;
      const int nl = l + 1 < L ? l + 1 : 0;
      int nslot = slots[nl];
      if (l + 1 == L) nslot = nslot + 1 == ltab[0].depth ? 0 : nslot + 1;
      // with one layer, the next step's pops include the state this layer pushes now: fetch after it
      if (more && L > 1) fetch(nl, nslot, par ^ 1);
      // ---- push phase for this queue: the layer's input x^{l-1}_t replaces the oldest state,
      // whose pop has landed in LDS already
      const long long qbase = ld.ring_off + (long long)slots[l] * a.bmax * C;
      for (int i = tid; i < RPW * C; i += kThreads) {
        const int r = i / C, c = i % C;
        if (r < nrows) WTraits<WT>::store1(a.ring, qbase + (long long)(b0 + r) * C + c, xo[i]);
      }
      if (more && L == 1) {
        __syncthreads();
        fetch(nl, nslot, par ^ 1);
      }
      const char *wb = stage ? (const char *)wbuf(par) : (const char *)ld.block;
      // staged weights and biases through LDS pointers (LDS loads), else global pointers
      typedef typename std::conditional<STAGE, lds_u4p, glb_u4p>::type WP;
      typedef typename std::conditional<STAGE, lds_f32p, glb_f32p>::type BP;
      auto wp = [&](size_t off) { return (WP)(wb + off); };
      const BP cb = (BP)(wb + o_cb);
      const float *vo = vbuf(par);
      // ---- dilated convolution of width w: [v_0 .. v_{w-2} x] . [W_0 ; .. ; W_{w-1}]
      rows_product<WT, RPW, WP>(wp(0), K, Co, vo, (w - 1) * C, xo, C, (w - 1) * C, partA);
      __syncthreads();
      if (kind == 2) {
        const BP rb = (BP)(wb + o_rb), sb = (BP)(wb + o_sb);
        // gate: z = tanh(a[0:R]) * sigmoid(a[R:2R])
        for (int i = tid; i < RPW * C; i += kThreads) {
          const int r = i / C, c = i % C;
          const float af = cb[c] + part_sum<RPW>(partA, Co, r, c);
          const float ag = cb[C + c] + part_sum<RPW>(partA, Co, r, C + c);
          // tanh(a) = 1 - 2 / (e^{2a} + 1) and sigmoid(g) = 1 / (1 + e^{-g}), one exp and one
          // reciprocal each (absolute error ~1e-7, saturating correctly at both ends)
          const float z = (1.f - 2.f * __builtin_amdgcn_rcpf(__expf(2.f * af) + 1.f)) *
                          __builtin_amdgcn_rcpf(1.f + __expf(-ag));
          zo[i] = WTraits<WT>::opnd(z);
        }
        __syncthreads();
        // residual and skip 1x1 products
        rows_product<WT, RPW, WP>(wp(o_res), C, C, zo, C, zo, C, C, partB);
        rows_product<WT, RPW, WP>(wp(o_skip), C, S, zo, C, zo, C, C, partA);
        __syncthreads();
        for (int i = tid; i < RPW * C; i += kThreads) {
          const int r = i / C, c = i % C;
          const float v = xf[i] + rb[c] + part_sum<RPW>(partB, C, r, c);
          xf[i] = v;
          xo[i] = WTraits<WT>::opnd(v);
        }
        for (int i = tid; i < RPW * S; i += kThreads) {
          const int r = i / S, k = i % S;
          so[i] += sb[k] + part_sum<RPW>(partA, S, r, k);
        }
      } else {
        for (int i = tid; i < RPW * C; i += kThreads) {
          const int r = i / C, c = i % C;
          const float pre = cb[c] + part_sum<RPW>(partA, Co, r, c);
          const float v = (kind == 1 ? xf[i] : 0.f) + fmaxf(pre, 0.f);
          xf[i] = v;
          xo[i] = WTraits<WT>::opnd(v);
        }
      }
      if (more) land(par ^ 1);
      __syncthreads();
      par ^= 1;
    }

    // ---- output head
    const float *top = xo;
    int Ktop = C;
    if (kind == 2) {
      for (int i = tid; i < RPW * S; i += kThreads) ho[i] = WTraits<WT>::opnd(fmaxf(so[i], 0.f));
      __syncthreads();
      rows_product<WT, RPW, glb_u4p>((glb_u4p)a.head, S, H, ho, S, ho, S, S, partA);
      __syncthreads();
      for (int i = tid; i < RPW * H; i += kThreads) {
        const int r = i / H, n = i % H;
        h2[i] = WTraits<WT>::opnd(fmaxf(bias_or0(a.head_b, n) + part_sum<RPW>(partA, H, r, n), 0.f));
      }
      __syncthreads();
      top = h2;
      Ktop = H;
    }
    rows_product<WT, RPW, glb_u4p>((glb_u4p)a.out, Ktop, Q, top, Ktop, top, Ktop, Ktop, partA);
    __syncthreads();
    for (int i = tid; i < RPW * Q; i += kThreads) {
      const int r = i / Q, q = i % Q;
      lg[i] = bias_or0(a.out_b, q) + part_sum<RPW>(partA, Q, r, q);
    }
    __syncthreads();

    if (a.mode != MODE_GENERATE) {
      if (a.logits)
        for (int i = tid; i < nrows * Q; i += kThreads) {
          const int r = i / Q, q = i % Q;
          a.logits[((long long)(b0 + r) * a.n_steps + s) * Q + q] = lg[i];
        }
      // the next input: the following element of the forced sequence (teacher forcing), or this
      // step's observed sample (online prediction)
      const int nx = s + forced_shift(a.mode);
      if (tid < nrows && nx < a.n_steps) ins[tid] = a.inputs[(long long)(b0 + tid) * a.n_steps + nx];
    } else {
      // ---- sample and feed back
      const int wv = tid >> 6;
      for (int r = wv; r < nrows; r += kThreads / 64) {
        const float u = a.uniforms[(long long)(b0 + r) * a.n_steps + s];
        const int k = sample_row_256(lg + r * Q, u);
        if ((tid & 63) == 0) {
          a.samples[(long long)(b0 + r) * a.n_steps + s] = k;
          ins[r] = k;
        }
      }
    }
    // ---- advance every queue's slot
    for (int l = tid; l < L; l += kThreads) {
      const int nx = slots[l] + 1;
      slots[l] = nx == ltab[l].depth ? 0 : nx;
    }
    __syncthreads();
  }
  if (a.mode != MODE_TEACHER && tid < nrows) a.last[b0 + tid] = ins[tid];
}

template <typename WT, bool STAGE, typename SH>
static hipError_t launch_valu_t(const StepArgs &a, int rpw, size_t lds, hipStream_t s) {
  const dim3 grid((a.batch + rpw - 1) / rpw), block(kThreads);
  switch (rpw) {
    case 1: hipLaunchKernelGGL((valu_step_kernel<WT, 1, STAGE, SH>), grid, block, lds, s, a); break;
    case 2: hipLaunchKernelGGL((valu_step_kernel<WT, 2, STAGE, SH>), grid, block, lds, s, a); break;
    case 4: hipLaunchKernelGGL((valu_step_kernel<WT, 4, STAGE, SH>), grid, block, lds, s, a); break;
    case 8: hipLaunchKernelGGL((valu_step_kernel<WT, 8, STAGE, SH>), grid, block, lds, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename WT, typename SH>
static hipError_t launch_valu_s(const StepArgs &a, int rpw, size_t lds, hipStream_t s) {
  return a.valu_wbytes > 0 ? launch_valu_t<WT, true, SH>(a, rpw, lds, s) : launch_valu_t<WT, false, SH>(a, rpw, lds, s);
}

// fp32 shapes with instantiations of their own: gated R = 32, S = H = 256 at widths 2 and 3.  (A
// 512-channel ReLU + residual instantiation ran 3x slower than the runtime-shaped kernel.)
typedef ShapeFixed<2, 32, 256, 256, 2> ShapeG32;
typedef ShapeFixed<2, 32, 256, 256, 3> ShapeG32W3;
template <typename SH>
static bool shape_is(const StepArgs &a) {
  return a.kind == SH::kind && a.C == SH::C && a.S == SH::S && a.H == SH::H && a.Q == SH::Q && a.w == SH::w;
}

hipError_t launch_valu_step(const StepArgs &a, int rpw, size_t lds, hipStream_t s) {
  if (a.dtype == 1) return launch_valu_s<uint16_t, ShapeAny>(a, rpw, lds, s);
  if (shape_is<ShapeG32>(a)) return launch_valu_s<float, ShapeG32>(a, rpw, lds, s);
  if (shape_is<ShapeG32W3>(a)) return launch_valu_s<float, ShapeG32W3>(a, rpw, lds, s);
  return launch_valu_s<float, ShapeAny>(a, rpw, lds, s);
}

template <typename WT, int RPW, typename SH>
static hipError_t set_lds_sh(size_t bytes) {
  hipError_t e = hipFuncSetAttribute((const void *)valu_step_kernel<WT, RPW, true, SH>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute((const void *)valu_step_kernel<WT, RPW, false, SH>,
                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}
template <typename WT, int RPW>
static hipError_t set_lds_one(size_t bytes) {
  hipError_t e = set_lds_sh<WT, RPW, ShapeAny>(bytes);
  if constexpr (sizeof(WT) == 4) {
    if (e != hipSuccess) return e;
    if ((e = set_lds_sh<WT, RPW, ShapeG32>(bytes)) != hipSuccess) return e;
    e = set_lds_sh<WT, RPW, ShapeG32W3>(bytes);
  }
  return e;
}

hipError_t set_valu_lds_limit(size_t bytes) {
  hipError_t e;
  if ((e = set_lds_one<float, 1>(bytes)) != hipSuccess) return e;
  if ((e = set_lds_one<float, 2>(bytes)) != hipSuccess) return e;
  if ((e = set_lds_one<float, 4>(bytes)) != hipSuccess) return e;
  if ((e = set_lds_one<float, 8>(bytes)) != hipSuccess) return e;
  if ((e = set_lds_one<uint16_t, 1>(bytes)) != hipSuccess) return e;
  if ((e = set_lds_one<uint16_t, 2>(bytes)) != hipSuccess) return e;
  if ((e = set_lds_one<uint16_t, 4>(bytes)) != hipSuccess) return e;
  return set_lds_one<uint16_t, 8>(bytes);
}

// ---------------------------------------------------------------------------
// Weight repacking (once, at create): dst in the VALU K-blocked layout
// Wp[kb][n][j] = W^T[kb*KB + j][n], or the embedding's row-gather table.
template <typename T>
__global__ void repack_kernel(const T *__restrict__ src, T *__restrict__ dst, int mode, int K, int N, int C, int KB) {
  const long long total = (long long)K * N;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (long long)gridDim.x * blockDim.x) {
    if (mode == REPACK_EMBED) {
      // dst [Q][C] from src [C][Q]; here K = Q, N = C
      const long long q = i / N, c = i % N;
      dst[i] = src[c * K + q];
      continue;
    }
    const long long j = i % KB, rest = i / KB;
    const long long n = rest % N, kb = rest / N;
    const long long k = kb * KB + j;
    long long si;
    if (mode == REPACK_CONV) si = (n * C + (k % C)) * (K / C) + k / C;  // tap k / C of K / C
    else si = n * K + k;
    dst[i] = src[si];
  }
}

hipError_t launch_repack(const void *src, void *dst, int mode, int dtype, int K, int N, int C, hipStream_t s) {
  const long long total = (long long)K * N;
  const int blocks = (int)((total + 255) / 256 < 4096 ? (total + 255) / 256 : 4096);
  if (dtype == 1)
    hipLaunchKernelGGL(repack_kernel<uint16_t>, dim3(blocks), dim3(256), 0, s, (const uint16_t *)src,
                       (uint16_t *)dst, mode, K, N, C, valu_kb_elems(1));
  else
    hipLaunchKernelGGL(repack_kernel<float>, dim3(blocks), dim3(256), 0, s, (const float *)src, (float *)dst,
                       mode, K, N, C, valu_kb_elems(0));
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Fills (used instead of memset nodes so the calls stay safe under stream capture).
// Zero `bytes` bytes at dst (16-byte aligned): whole 16-byte units, then the tail byte by byte.
__global__ void fill_zero_kernel(uint4 *dst, size_t bytes) {
  const size_t n16 = bytes / 16;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (size_t)gridDim.x * blockDim.x)
    dst[i] = make_uint4(0, 0, 0, 0);
  if (blockIdx.x == 0 && threadIdx.x < bytes % 16) ((unsigned char *)dst)[n16 * 16 + threadIdx.x] = 0;
}
__global__ void fill_i32_kernel(int32_t *dst, int32_t v, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) dst[i] = v;
}
__global__ void copy_bias_kernel(const float *src, float *dst, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) dst[i] = src ? src[i] : 0.f;
}

hipError_t launch_fill_zero(void *dst, size_t bytes, hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  const size_t n16 = bytes / 16;  // regions start 256-byte aligned
  const int blocks = (int)(n16 / 256 + 1 < 8192 ? n16 / 256 + 1 : 8192);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks), dim3(256), 0, s, (uint4 *)dst, bytes);
  return hipGetLastError();
}
hipError_t launch_fill_i32(int32_t *dst, int32_t v, int n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_i32_kernel, dim3((n + 255) / 256), dim3(256), 0, s, dst, v, n);
  return hipGetLastError();
}
hipError_t launch_copy_bias(const float *src, float *dst, int n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(copy_bias_kernel, dim3((n + 255) / 256), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

}  // namespace fwg
