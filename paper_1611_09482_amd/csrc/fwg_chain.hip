// Chain step kernel for small float32 ReLU stacks (channels C = 32, filter width 2, at most six
// layers): one block per stream, every weight and every queue of the stream in LDS for the whole
// launch, each wave's half of the dilated products in its registers.
//
// A sample's work is a chain of dependent steps (the layers in order, then the output 1x1 and the
// sample, which is the next input: Section 1, Section 2.2); at one stream nothing else can run beside
// it, so the kernel shortens that chain instead of widening it:
//  - wave 0 (the chain) holds the layer input as lane o -> channel o % 32 and computes output o in
//    lanes o and o + 32, each over half of K: the lane's 16 weights stay in its registers for the
//    launch, the 16 inputs of its half are read back from the queue row it has just pushed (one
//    LDS broadcast per half-wave), and the halves' partial sums meet with one cross-half lane
//    swap; the output 1x1 gives lane l the classes 4l..4l+3, and the sampler reduces them with DPP
//    row moves and lane reads;
//  - wave 1 computes W_r v + b of every layer for the next step (v = the state popped from the
//    layer's queue: pushed d_l >= 1 steps earlier, so known before that step starts; for d_l = 1 it
//    waits for the chain's push of this step through an LDS flag) and stages the per-step uniforms
//    or forced inputs; one block barrier per step orders the two waves.
// The queues live in LDS as [layer][slot][C] (slot = t mod d); they are loaded from the workspace at
// launch and written back at its end, so the generation state carries across calls.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "fwg_chain.h"
#include "fwg_internal.h"
#include "fwg_sample.h"
#include "fwg_xchg.h"

namespace fwg {
namespace ch {

constexpr int C = kChainC, Q = 256;
constexpr int LR = kChainMaxLayers;  // layers whose weights the waves hold in registers
static_assert(LR <= 8, "the per-layer flags fit the 8 words before the broadcast row");
constexpr int NT = 128;      // wave 0: the chain; wave 1: recurrent halves and staging
constexpr int KCH = 64;      // steps per chunk of staged uniforms / forced inputs
constexpr int SPIN_MAX = 1 << 24;

// v of lane i plus v of lane i ^ 32, in every lane (the two half-waves' partial sums of one dot product).
__device__ __forceinline__ float halves_sum(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, v), __builtin_bit_cast(unsigned, v),
                                                 false, false);
  return __builtin_bit_cast(float, (unsigned)r[0]) + __builtin_bit_cast(float, (unsigned)r[1]);
}

// Dot product of a register row (this lane's half: 16 weights) with 16 values read from LDS as a
// broadcast within the half-wave (v points at the half's first value), two accumulation chains.
__device__ __forceinline__ float half_dot(const float (&w)[C / 2], const float *v) {
  const float4 *v4 = (const float4 *)v;
  float a0 = 0.f, a1 = 0.f;
#pragma unroll
  for (int i = 0; i < C / 8; ++i) {
    const float4 x = v4[i];
    a0 = fmaf(w[4 * i], x.x, a0);
    a1 = fmaf(w[4 * i + 1], x.y, a1);
    a0 = fmaf(w[4 * i + 2], x.z, a0);
    a1 = fmaf(w[4 * i + 3], x.w, a1);
  }
  return a0 + a1;
}

// LDS areas of a launch (offsets from the ChainArgs layout, in floats).
struct Lay {
  const float *img;   // the weight image
  float *ring;        // queues: layer l at ring + qoff[l], [slot][C]
  float *pbuf;        // [2][LR][C]: W_r v + b of every layer, by step parity
  volatile int *flag; // per layer: step index + 1 once the chain pushed this step's input
  float *xrow;        // [C] the last layer's output, broadcast to the output 1x1
  float *u;           // [2][KCH] staged uniforms (generation)
  int *fin;           // [2][KCH] staged forced next inputs
};

__global__ void __launch_bounds__(NT) chain_step_kernel(StepArgs a, ChainArgs g) {
  extern __shared__ float4 lds4[];
  float *lds = (float *)lds4;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int b = blockIdx.x, L = a.L;
  Lay s;
  s.img = lds;
  s.ring = lds + g.image_floats;
  s.pbuf = s.ring + g.ring_floats;
  s.u = s.pbuf + 2 * LR * C;
  s.fin = (int *)(s.u + 2 * KCH);
  s.flag = (volatile int *)(s.fin + 2 * KCH);
  s.xrow = (float *)(s.fin + 2 * KCH + 8);  // 16-byte aligned after the flags

  // per-layer queue offsets, dilations and slots, in wave-uniform registers
  int qoff[LR], dil[LR], slot[LR];
  {
    int off = 0;
#pragma unroll
    for (int l = 0; l < LR; ++l) {
      const int d = l < L ? a.layers[l].dil : 1;
      qoff[l] = off;
      dil[l] = d;
      slot[l] = (int)(a.t0 % (long long)d);
      off += l < L ? d * C : 0;
    }
  }
  // ---- launch: image, queues of this stream, flags, first chunk of per-step inputs
  for (int i = tid; i < g.image_floats / 4; i += NT) lds4[i] = ((const float4 *)g.image)[i];
#pragma unroll
  for (int l = 0; l < LR; ++l) {
    if (l < L) {
      const float *src = (const float *)a.ring + a.layers[l].ring_off;
      for (int i = tid; i < dil[l] * C; i += NT) {
        const int sl = i / C, ch = i % C;
        s.ring[qoff[l] + i] = src[((long long)sl * a.bmax + b) * C + ch];
      }
    }
  }
  if (tid < LR) s.flag[tid] = 0;
  for (int j = tid; j < KCH; j += NT) {
    if (a.mode == MODE_GENERATE) s.u[j] = j < a.n_steps ? a.uniforms[(long long)b * a.n_steps + j] : 0.f;
    else {
      const long long nx = j + forced_shift(a.mode);
      s.fin[j] = nx < a.n_steps ? a.inputs[(long long)b * a.n_steps + nx] : 0;
    }
  }
  __syncthreads();

  const int o = lane & (C - 1);
  const bool residual = a.kind == 1;  // relu + residual (FWG_RELU_RESIDUAL)
  // this wave's half of every layer's dilated product, in registers for the launch: lanes o and
  // o + 32 hold row o over K halves 0 and 1 (wave 0: W_e, the current-input tap; wave 1: W_r, the
  // popped tap)
  const int h = lane >> 5;
  float wt[LR][C / 2];
#pragma unroll
  for (int l = 0; l < LR; ++l)
#pragma unroll
    for (int j = 0; j < C / 2; ++j)
      wt[l][j] = l < L ? s.img[g.o_layer + l * g.layer_floats + (1 - wave) * C * C + (16 * h + j) * C + o] : 0.f;

  if (wave == 1) {
    // ---- W_r v + b of every layer for step 0 (its pops were all pushed before the launch)
#pragma unroll
    for (int l = 0; l < LR; ++l) {
      if (l < L) {
        const float acc = halves_sum(half_dot(wt[l], s.ring + qoff[l] + slot[l] * C + 16 * h)) +
                          s.img[g.o_layer + l * g.layer_floats + 2 * C * C + o];
        if (lane < C) s.pbuf[l * C + o] = acc;
      }
    }
  }
  __syncthreads();  // step 0's W_r v + b is in LDS
  if (wave == 1) {
    for (int step = 0; step < a.n_steps; ++step) {
      // ---- W_r v + b of every layer for the next step, into the other parity
      const int np = (step & 1) ^ 1;
#pragma unroll
      for (int l = 0; l < LR; ++l) {
        if (l < L) {
          const int sl = slot[l] + 1 == dil[l] ? 0 : slot[l] + 1;
          if (dil[l] == 1) {
            // the state popped next step is this step's input of the layer: wait for the chain's push
            for (int it = 0; s.flag[l] != step + 1 && it < SPIN_MAX; ++it) __builtin_amdgcn_s_sleep(1);
          }
          const float acc = halves_sum(half_dot(wt[l], s.ring + qoff[l] + sl * C + 16 * h)) +
                            s.img[g.o_layer + l * g.layer_floats + 2 * C * C + o];
          if (lane < C) s.pbuf[(np * LR + l) * C + o] = acc;
          slot[l] = sl;
        }
      }
      // staging of the next chunk, one chunk ahead
      if (step % KCH == 0) {
        const int base = step + KCH, buf = (step / KCH + 1) & 1;
        for (int j = lane; j < KCH; j += 64) {
          const long long sj = base + j;
          if (a.mode == MODE_GENERATE) {
            s.u[buf * KCH + j] = sj < a.n_steps ? a.uniforms[(long long)b * a.n_steps + sj] : 0.f;
          } else {
            const long long nx = sj + forced_shift(a.mode);
            s.fin[buf * KCH + j] = nx < a.n_steps ? a.inputs[(long long)b * a.n_steps + nx] : 0;
          }
        }
      }
      __syncthreads();
    }
  } else {
    // ---- the chain: embedding, layers, output 1x1, sample
    const float *embT = s.img + g.o_emb;                  // [Q][C]
    const float *embb = s.img + g.o_embb;                 // [C]
    const float4 *woT4 = (const float4 *)(s.img + g.o_out);  // [C][Q / 4]
    const float4 *wob4 = (const float4 *)(s.img + g.o_outb);
    int in = a.mode == MODE_TEACHER ? a.inputs[(long long)b * a.n_steps] : a.last[b];
    for (int step = 0; step < a.n_steps; ++step) {
      const int par = step & 1;
      float x = embT[in * C + o] + embb[o];
      float pv[LR];
#pragma unroll
      for (int l = 0; l < LR; ++l) pv[l] = l < L ? s.pbuf[(par * LR + l) * C + o] : 0.f;
      float4 wo[2][4];
#pragma unroll
      for (int l = 0; l < LR; ++l) {
        if (l < L) {
          // push: this layer's input replaces the slot the step pops (its value was read for this
          // step's W_r v one step earlier)
          if (lane < C) s.ring[qoff[l] + slot[l] * C + o] = x;
          if (lane == 0) s.flag[l] = step + 1;
          const int slot_pushed = slot[l];
          slot[l] = slot[l] + 1 == dil[l] ? 0 : slot[l] + 1;
          if (l + 1 == L) {
            // the output 1x1's first weights, read while the last layer computes
#pragma unroll
            for (int j = 0; j < 4; ++j) wo[0][j] = woT4[j * (Q / 4) + lane];
          }
          // the pushed row read back as this half's 16 inputs (LDS operations of a wave execute in order)
          const float acc = halves_sum(half_dot(wt[l], s.ring + qoff[l] + slot_pushed * C + 16 * h)) + pv[l];
          const float r = fmaxf(acc, 0.f);
          x = residual ? x + r : r;
        }
      }
      // output 1x1: lane l takes classes 4l..4l+3; the last layer's output reaches every lane through
      // an LDS row, the weights are read four k-steps ahead
      if (lane < C) s.xrow[o] = x;
      float xs[C];
#pragma unroll
      for (int i = 0; i < C / 4; ++i) {
        const float4 v = ((const float4 *)s.xrow)[i];
        xs[4 * i] = v.x;
        xs[4 * i + 1] = v.y;
        xs[4 * i + 2] = v.z;
        xs[4 * i + 3] = v.w;
      }
      float4 lg = wob4[lane];
#pragma unroll
      for (int kb = 0; kb < C / 4; ++kb) {
        if (kb + 1 < C / 4) {
#pragma unroll
          for (int j = 0; j < 4; ++j) wo[(kb + 1) & 1][j] = woT4[((kb + 1) * 4 + j) * (Q / 4) + lane];
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float xk = xs[kb * 4 + j];
          const float4 wv = wo[kb & 1][j];
          lg.x = fmaf(wv.x, xk, lg.x);
          lg.y = fmaf(wv.y, xk, lg.y);
          lg.z = fmaf(wv.z, xk, lg.z);
          lg.w = fmaf(wv.w, xk, lg.w);
        }
      }
      if (a.mode == MODE_GENERATE) {
        in = sample_row4(lg, s.u[(step / KCH & 1) * KCH + step % KCH]);
        if (lane == 0) a.samples[(long long)b * a.n_steps + step] = in;
      } else {
        if (a.logits) ((float4 *)(a.logits + ((long long)b * a.n_steps + step) * Q))[lane] = lg;
        in = s.fin[(step / KCH & 1) * KCH + step % KCH];
      }
      __syncthreads();
    }
    if (tid == 0 && a.mode != MODE_TEACHER) a.last[b] = in;
  }
  __syncthreads();

  // ---- launch end: queues back to the workspace
#pragma unroll
  for (int l = 0; l < LR; ++l) {
    if (l < L) {
      float *dst = (float *)a.ring + a.layers[l].ring_off;
      for (int i = tid; i < dil[l] * C; i += NT) {
        const int sl = i / C, ch = i % C;
        dst[((long long)sl * a.bmax + b) * C + ch] = s.ring[qoff[l] + i];
      }
    }
  }
}

// Image of the weights: per layer W_r^T [C][C] (tap 0), W_e^T [C][C] (tap 1), bias [C]; the
// embedding transposed [Q][C] and its bias; the output 1x1 transposed [C][Q] and its bias.
__global__ void chain_image_kernel(const float *conv, const float *conv_b, float *layer_dst, int C_) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= 2 * C_ * C_ + C_) return;
  float v;
  if (i < 2 * C_ * C_) {
    const int tap = i / (C_ * C_), r = i % (C_ * C_), k = r / C_, oo = r % C_;
    v = conv[((size_t)oo * C_ + k) * 2 + tap];
  } else {
    v = conv_b ? conv_b[i - 2 * C_ * C_] : 0.f;
  }
  layer_dst[i] = v;
}
__global__ void chain_transpose_kernel(const float *src, float *dst, int rows, int cols) {
  // dst[c][r] = src[r][c]
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * cols) return;
  const int r = i / cols, c = i % cols;
  dst[(size_t)c * rows + r] = src[i];
}
__global__ void chain_vec_kernel(const float *src, float *dst, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = src ? src[i] : 0.f;
}

}  // namespace ch

bool chain_layout(int kind, int dtype, int C, int Q, int L, int w, const int32_t *dil, ChainArgs *g, size_t *lds) {
  if ((kind != 0 && kind != 1) || dtype != 0 || C != kChainC || Q != 256 || w != 2 || L < 1 || L > kChainMaxLayers)
    return false;
  long long ring = 0;
  for (int l = 0; l < L; ++l) ring += (long long)dil[l] * C;
  g->o_emb = 0;
  g->o_embb = Q * C;
  g->o_layer = g->o_embb + C;
  g->layer_floats = 2 * C * C + C;
  g->o_out = g->o_layer + L * g->layer_floats;
  g->o_outb = g->o_out + C * Q;
  g->image_floats = (g->o_outb + Q + 3) & ~3;
  g->ring_floats = (int)((ring + 3) & ~3ll);
  const long long floats = (long long)g->image_floats + g->ring_floats + 2LL * kChainMaxLayers * C + 2 * ch::KCH +
                           2 * ch::KCH + 8 + kChainC;
  *lds = (size_t)floats * 4;
  return ring < (1 << 20) && *lds <= 160 * 1024;
}

hipError_t set_chain_lds_limit(size_t bytes) {
  return hipFuncSetAttribute((const void *)ch::chain_step_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)bytes);
}

hipError_t launch_chain_step(const StepArgs &a, const ChainArgs &g, size_t lds, hipStream_t s) {
  hipLaunchKernelGGL(ch::chain_step_kernel, dim3(a.batch), dim3(ch::NT), lds, s, a, g);
  return hipGetLastError();
}

hipError_t launch_chain_image(const void *embed, const float *embed_b, const void *const *conv,
                              const float *const *conv_b, const void *out, const float *out_b, int L,
                              const ChainArgs &g, float *img, hipStream_t s) {
  const int C = kChainC, Q = 256;
  hipLaunchKernelGGL(ch::chain_transpose_kernel, dim3((C * Q + 255) / 256), dim3(256), 0, s, (const float *)embed,
                     img + g.o_emb, C, Q);
  hipLaunchKernelGGL(ch::chain_vec_kernel, dim3(1), dim3(256), 0, s, embed_b, img + g.o_embb, C);
  for (int l = 0; l < L; ++l)
    hipLaunchKernelGGL(ch::chain_image_kernel, dim3((2 * C * C + C + 255) / 256), dim3(256), 0, s,
                       (const float *)conv[l], conv_b ? conv_b[l] : nullptr, img + g.o_layer + l * g.layer_floats, C);
  hipLaunchKernelGGL(ch::chain_transpose_kernel, dim3((C * Q + 255) / 256), dim3(256), 0, s, (const float *)out,
                     img + g.o_out, Q, C);
  hipLaunchKernelGGL(ch::chain_vec_kernel, dim3(1), dim3(256), 0, s, out_b, img + g.o_outb, Q);
  return hipGetLastError();
}

}  // namespace fwg

// ---------------------------------------------------------------------------
// Gated variant: float32 gated stacks with R = 32, S = H = 256 (the WaveNet-style unit: z =
// tanh(a[0:R]) sigmoid(a[R:2R]), residual and skip 1x1s, the skip sum through relu -> 1x1 -> relu
// -> 1x1 to the logits; Section 2.1, Fig. 2), at most 64 layers, filter width 2 or 3 (Section 3.1).
// One block of four waves per stream:
//  - wave 0 (the chain): lane o computes gate pre-activation o (tanh half for o < 32, sigmoid half
//    for o >= 32) from the layer input broadcast through LDS; the halves meet with one cross-half
//    lane swap, which leaves z in both halves; the residual 1x1 splits K over the half-waves.  It
//    pushes each layer input to the layer's queue in the workspace and to an LDS row;
//  - wave 1: the recurrent taps of every layer's product for the next step (W_r v + b at width 2):
//    states pushed at least one step earlier (before a block barrier) are read from the workspace
//    queues; the newest tap of a layer with d = 1 is this step's LDS row (an LDS flag per layer);
//  - waves 2, 3: the skip sum, two of the 256 skip channels per lane, each layer as soon as its z
//    row is in LDS (an LDS flag per layer);
//  - then all four waves compute the head, one hidden channel and then one class per thread, and
//    wave 0 draws the sample.
// Every weight is streamed from the workspace once per step (the model, about 1.6 MB at 20 layers,
// stays in L2), into registers one layer ahead.  The per-layer queue offset and slot of layer l live
// in lane l of the waves that need them and are read with lane reads.
namespace fwg {
namespace chg {

constexpr int R = kChainGR, S = kChainGS, H = kChainGS, Q = 256, NT = 256, KCH = 64;
constexpr int FCH = 12, FREC = 8, FSK = 16, FH = 64, FHR = 8;  // float4 chunks per lane (FHR: per head round)
constexpr int FZ = R / 4;  // float4 chunks of one 32-wide row
constexpr int SPIN_MAX = 1 << 20;

// Flags in LDS, addressed as LDS: through a generic pointer a volatile access stays a flat access,
// whose wait also drains every global load in flight (the weights fetched one layer ahead).
typedef __attribute__((address_space(3))) volatile int lds_flag;

struct Lay {
  float *embT, *embb;   // [Q][R], [R]
  float *P;             // [2][L][2R]: W_r v + b by step parity
  float *xrow, *zrow;   // [L][R]: this step's layer inputs and gate outputs
  float *resb;          // [L][R]
  float *srow, *hrow, *lrow;  // [S]: relu(skip sum); [H]: relu(hidden); [Q]: logits
  float *u;             // [2][KCH]
  int *fin;             // [2][KCH]
  lds_flag *fx, *fz;     // [L]: step + 1 once the chain wrote xrow[l] / zrow[l]
  lds_flag *abort_;      // set once a flag wait ran out: later waits of the launch return at once
};

__host__ __device__ inline size_t lds_floats(int L) {
  return (size_t)Q * R + R + 2ull * L * 2 * R + 3ull * L * R + S + H + Q + 2 * KCH + 2 * KCH + 2ull * L + 4;
}
// offset (in 4-byte words) of the flags
__host__ __device__ inline int lay_flag_off(int L) { return Q * R + R + 2 * L * 2 * R + 3 * L * R + S + H + Q + 4 * KCH; }
__device__ __forceinline__ Lay make_lay(float *lds, int L) {
  Lay s;
  s.embT = lds;
  s.embb = s.embT + Q * R;
  s.P = s.embb + R;
  s.xrow = s.P + 2 * L * 2 * R;
  s.zrow = s.xrow + L * R;
  s.resb = s.zrow + L * R;
  s.srow = s.resb + L * R;
  s.hrow = s.srow + S;
  s.lrow = s.hrow + H;
  s.u = s.lrow + Q;
  s.fin = (int *)(s.u + 2 * KCH);
  s.fx = (lds_flag *)(lds + lay_flag_off(L));
  s.fz = s.fx + L;
  s.abort_ = s.fz + L;
  return s;
}

// Weight streams are read as raw buffer loads from one resource over the packed weights: the
// per-lane part of the address is one constant VGPR offset and the per-chunk part an SGPR offset,
// so that no 64-bit address per chunk is kept in registers.
typedef __amdgpu_buffer_rsrc_t Rsrc;
__device__ __forceinline__ Rsrc make_rsrc(const void *base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, bytes, 0x00020000);
}
template <int N>
__device__ __forceinline__ void load_chunks(float4 (&dst)[N], Rsrc r, int voff, int soff, int stride) {
#pragma unroll
  for (int i = 0; i < N; ++i)
    dst[i] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff + i * stride, 0));
}
// keeps the compiler from moving LDS accesses across a flag store or a flag wait (the hardware runs
// a wave's LDS operations in order)
__device__ __forceinline__ void compiler_fence() { asm volatile("" ::: "memory"); }

// Waits until flag == want, at most SPIN_MAX polls (the chain wave sets every flag of a step
// unconditionally; the bound only keeps a fault from turning into a hang).
template <class S>
__device__ __forceinline__ void wait_flag(const S &s, lds_flag *flag, int want) {
  for (int it = 0; *flag != want; ++it) {
    if (it >= SPIN_MAX || *s.abort_) {
      *s.abort_ = 1;
      break;
    }
    __builtin_amdgcn_s_sleep(1);
  }
  compiler_fence();
}

__device__ __forceinline__ float gate_half(float a, bool tanh_half) {
  // tanh(a) = 1 - 2 / (exp(2a) + 1) for the first half, sigmoid(a) = 1 / (1 + exp(-a)) for the second
  const float e = __expf(tanh_half ? 2.f * a : -a);
  const float r = __builtin_amdgcn_rcpf(e + 1.f);
  return tanh_half ? 1.f - 2.f * r : r;
}

__device__ __forceinline__ long long lane_i64(long long v, int l) {
  const int lo = __builtin_amdgcn_readlane((int)(unsigned)(v & 0xffffffffll), l);
  const int hi = __builtin_amdgcn_readlane((int)(v >> 32), l);
  return (long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo);
}

// The chain wave's layer l with its weights in Wc (W_e row chunks, then W_res half-row chunks); the
// next layer's weights are fetched into Wn first.  x: the layer input in (lane o and o + 32 both
// hold channel o), the layer output out.  qptr: this step's push address of the layer's queue.
// zw (pair variant): z of the layer also goes out as 32 tagged words zw[32 l + o].
__device__ __forceinline__ void chain_gated_layer(const Lay &s, float4 (&Wc)[FCH], float4 (&Wn)[FCH], Rsrc rw,
                                                  int next_off, float *qptr, int l, int L, int par, int step,
                                                  int lane, float &x, xg::u64 *zw = nullptr,
                                                  bool local = false) {
  const int o = lane & (R - 1), h = lane >> 5;
  if (lane < R) {
    qptr[o] = x;
    s.xrow[l * R + o] = x;
  }
  compiler_fence();
  if (lane == 0) s.fx[l] = step + 1;
  load_chunks(Wn, rw, lane * 16, next_off, 1024);
  const float4 *xr4 = (const float4 *)(s.xrow + l * R);
  float a0 = s.P[(par * L + l) * 2 * R + lane], a1 = 0.f;
#pragma unroll
  for (int c = 0; c < R / 4; ++c) {
    const float4 xv = xr4[c];
    a0 = fmaf(Wc[c].x, xv.x, a0);
    a1 = fmaf(Wc[c].y, xv.y, a1);
    a0 = fmaf(Wc[c].z, xv.z, a0);
    a1 = fmaf(Wc[c].w, xv.w, a1);
  }
  const float v = gate_half(a0 + a1, lane < R);
  const auto sw = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, v), __builtin_bit_cast(unsigned, v),
                                                   false, false);
  // lanes o and o + 32 both hold tanh(a_o) and sigmoid(a_{o+32})
  const float z = __builtin_bit_cast(float, (unsigned)sw[0]) * __builtin_bit_cast(float, (unsigned)sw[1]);
  if (lane < R) s.zrow[l * R + o] = z;
  compiler_fence();
  if (lane == 0) s.fz[l] = step + 1;
  if (zw != nullptr && lane < R) xg::put_word(zw + l * R + o, __builtin_bit_cast(uint32_t, z), step + 1, local);
  // the residual 1x1 over this half of K, z read back from its row
  const float4 *zr4 = (const float4 *)(s.zrow + l * R + 16 * h);
  float r0 = 0.f, r1 = 0.f;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const float4 zv = zr4[c];
    r0 = fmaf(Wc[8 + c].x, zv.x, r0);
    r1 = fmaf(Wc[8 + c].y, zv.y, r1);
    r0 = fmaf(Wc[8 + c].z, zv.z, r0);
    r1 = fmaf(Wc[8 + c].w, zv.w, r1);
  }
  x = x + s.resb[l * R + o] + ch::halves_sum(r0 + r1);
}

// Wave 1's layer l: the recurrent taps of the dilated product for the next step, sum over k < W - 1
// of W_k v_k + b, v_k = the state tap k reads then (x_{t+1-(W-1-k)d}, Section 3.1; W = 2: the one
// popped state).  taps[k]: the state's queue row in the workspace, loaded before the next layer's
// weights so that its wait leaves them in flight; with last_row, the newest tap (distance d = 1) is
// this step's LDS row of the layer instead, read once the chain has written it.
template <int W, class S>
__device__ __forceinline__ void rec_layer(const S &s, const float4 (&Wc)[FREC * (W - 1)],
                                          float4 (&Wn)[FREC * (W - 1)], Rsrc rw, int next_off,
                                          const float *const (&taps)[W - 1], bool last_row, const float *convb, int l,
                                          int L, int np, int step, int lane) {
  constexpr int F = FREC * (W - 1);
  float4 vv[F];
#pragma unroll
  for (int k = 0; k < W - 1; ++k) {
    if (k + 2 < W || !last_row) {
#pragma unroll
      for (int c = 0; c < FREC; ++c) vv[FREC * k + c] = ((const float4 *)taps[k])[c];
    }
  }
  load_chunks(Wn, rw, lane * 16, next_off, 1024);
  if (last_row) {
    // the newest state tapped next step is this step's input of the layer
    wait_flag(s, s.fx + l, step + 1);
    const float4 *x4 = (const float4 *)(s.xrow + l * R);
#pragma unroll
    for (int c = 0; c < FREC; ++c) vv[FREC * (W - 2) + c] = x4[c];
  }
  float a0 = convb[l * 2 * R + lane], a1 = 0.f;
#pragma unroll
  for (int c = 0; c < F; ++c) {
    a0 = fmaf(Wc[c].x, vv[c].x, a0);
    a1 = fmaf(Wc[c].y, vv[c].y, a1);
    a0 = fmaf(Wc[c].z, vv[c].z, a0);
    a1 = fmaf(Wc[c].w, vv[c].w, a1);
  }
  s.P[(np * L + l) * 2 * R + lane] = a0 + a1;
}

// A skip wave's layer l: skip channels m0 and m0 + 1 accumulate W_s z of the layer.
__device__ __forceinline__ void skip_layer(const Lay &s, const float4 (&Wc)[FSK], float4 (&Wn)[FSK], Rsrc rw,
                                           int next_off, int lane, int l, int step, float &s0, float &s1) {
  load_chunks(Wn, rw, lane * 16, next_off, 1024);
  wait_flag(s, s.fz + l, step + 1);
  const float4 *zr4 = (const float4 *)(s.zrow + l * R);
  float p0 = 0.f, p1 = 0.f;
#pragma unroll
  for (int c = 0; c < R / 4; ++c) {
    const float4 zv = zr4[c];
    s0 = fmaf(Wc[c].x, zv.x, s0);
    s1 = fmaf(Wc[8 + c].x, zv.x, s1);
    p0 = fmaf(Wc[c].y, zv.y, p0);
    p1 = fmaf(Wc[8 + c].y, zv.y, p1);
    s0 = fmaf(Wc[c].z, zv.z, s0);
    s1 = fmaf(Wc[8 + c].z, zv.z, s1);
    p0 = fmaf(Wc[c].w, zv.w, p0);
    p1 = fmaf(Wc[8 + c].w, zv.w, p1);
  }
  s0 += p0;
  s1 += p1;
}

// One head 1x1 for output channel tid: the row (chunk c of thread t = 64 w + lane at byte
// off + 65536 w + 1024 c + 16 lane) streamed in rounds of FHR chunks (the first round already in HA),
// the input vector broadcast from LDS.  voff: this thread's 65536 w + 16 lane.
__device__ __forceinline__ void head_round(const float4 (&Wc)[FHR], const float *in, float &a0, float &a1) {
  const float4 *in4 = (const float4 *)in;
#pragma unroll
  for (int c = 0; c < FHR; ++c) {
    const float4 xv = in4[c];
    a0 = fmaf(Wc[c].x, xv.x, a0);
    a1 = fmaf(Wc[c].y, xv.y, a1);
    a0 = fmaf(Wc[c].z, xv.z, a0);
    a1 = fmaf(Wc[c].w, xv.w, a1);
  }
}
__device__ __forceinline__ float head_row(float4 (&HA)[FHR], float4 (&HB)[FHR], Rsrc rw, int voff, int off,
                                          const float *inrow, float bias) {
  constexpr int NR = FH / FHR;  // rounds, an even number
  float a0 = bias, a1 = 0.f;
  // two rounds per iteration, not unrolled: the compiler cannot hoist later rounds' loads and LDS
  // reads (their registers would spill)
#pragma unroll 1
  for (int r = 0; r < NR; r += 2) {
    load_chunks(HB, rw, voff, off + (r + 1) * FHR * 1024, 1024);
    head_round(HA, inrow + r * FHR * 4, a0, a1);
    if (r + 2 < NR) load_chunks(HA, rw, voff, off + (r + 2) * FHR * 1024, 1024);
    head_round(HB, inrow + (r + 1) * FHR * 4, a0, a1);
  }
  return a0 + a1;
}

template <int W>
__global__ void __launch_bounds__(NT) chain_gated_kernel(StepArgs a, ChainGatedArgs g) {
  constexpr int FR = FREC * (W - 1);  // wave 1's weight chunks per layer
  extern __shared__ float4 lds4[];
  float *lds = (float *)lds4;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int b = blockIdx.x, L = a.L;
  const Lay s = make_lay(lds, L);

  // ---- launch: tables into LDS, flags, the first chunk of per-step inputs
  for (int i = tid; i < Q * R / 4; i += NT) ((float4 *)s.embT)[i] = ((const float4 *)g.embT)[i];
  for (int i = tid; i < R; i += NT) s.embb[i] = g.embb[i];
  for (int i = tid; i < L * R; i += NT) s.resb[i] = g.resb[i];
  for (int i = tid; i < L; i += NT) {
    s.fx[i] = 0;
    s.fz[i] = 0;
  }
  if (tid == 0) *s.abort_ = 0;
  for (int j = tid; j < KCH; j += NT) {
    if (a.mode == MODE_GENERATE) s.u[j] = j < a.n_steps ? a.uniforms[(long long)b * a.n_steps + j] : 0.f;
    else {
      const long long nx = j + forced_shift(a.mode);
      s.fin[j] = nx < a.n_steps ? a.inputs[(long long)b * a.n_steps + nx] : 0;
    }
  }
  // lane l: layer l's queue (element offset of this stream's row in slot 0), dilation d, depth
  // (W - 1) d and the slot of the current step, t mod depth (wave 1 keeps the slot of the next
  // step); at slot t mod depth the queue holds x_{t-(W-1)d}, and tap k reads the state k d slots on
  const long long slot_stride = (long long)a.bmax * R;
  long long qoff = 0;
  int qdil = 1, qdep = W - 1, qslot = 0;
  if (lane < L) {
    const LayerDev ld = a.layers[lane];
    qoff = ld.ring_off + (long long)b * R;
    qdil = ld.dil;
    qdep = ld.depth;
    qslot = (int)(a.t0 % (long long)qdep);
  }
  float *ring = (float *)a.ring;
  // the recurrent taps of every layer for step 0 (wave 1; every state they read was pushed before
  // the launch)
  if (wave == 1) {
    for (int l = 0; l < L; ++l) {
      const float4 *w = g.wrec + (size_t)l * FR * 64 + lane;
      float acc = g.convb[l * 2 * R + lane];
#pragma unroll
      for (int k = 0; k < W - 1; ++k) {
        int sk = qslot + k * qdil;
        sk = sk >= qdep ? sk - qdep : sk;
        const float *v = ring + lane_i64(qoff + sk * slot_stride, l);
#pragma unroll
        for (int c = 0; c < FREC; ++c) {
          const float4 wv = w[(FREC * k + c) * 64];
          const float4 vv = *(const float4 *)(v + 4 * c);
          acc = fmaf(wv.x, vv.x, acc);
          acc = fmaf(wv.y, vv.y, acc);
          acc = fmaf(wv.z, vv.z, acc);
          acc = fmaf(wv.w, vv.w, acc);
        }
      }
      s.P[l * 2 * R + lane] = acc;
    }
    qslot = qslot + 1 == qdep ? 0 : qslot + 1;  // wave 1 works one step ahead
  }
  __syncthreads();

  int in = a.mode == MODE_TEACHER ? a.inputs[(long long)b * a.n_steps] : a.last[b];
  const int o = lane & (R - 1);
  // the packed weights, wchain first: byte offsets of the streams
  const char *wbase = (const char *)g.wchain;
  const Rsrc rw = make_rsrc(wbase, (int)((const char *)g.convb - wbase));
  const int o_rec = (int)((const char *)g.wrec - wbase), o_skip = (int)((const char *)g.wskip - wbase);
  const int o_head = (int)((const char *)g.whead - wbase), o_out = (int)((const char *)g.wout - wbase);
  const int hvoff = wave * 65536 + lane * 16;  // this thread's part of a head chunk address
  const float hbias = g.headb[tid], obias = g.outb[tid];
  float4 HA[FHR], HB[FHR];
  if (wave == 0) {
    // ---------------- the chain, then its share of the head
    const int lstr = FCH * 1024;
    float4 WA[FCH], WB[FCH];
    load_chunks(WA, rw, lane * 16, 0, 1024);
    for (int step = 0; step < a.n_steps; ++step) {
      const int par = step & 1;
      float x = s.embT[in * R + o] + s.embb[o];
      for (int l = 0; l < L; l += 2) {
        {
          float *qp = ring + lane_i64(qoff + qslot * slot_stride, l);
          const int ln = l + 1 < L ? l + 1 : 0;
          chain_gated_layer(s, WA, WB, rw, ln * lstr, qp, l, L, par, step, lane, x);
        }
        if (l + 1 < L) {
          float *qp = ring + lane_i64(qoff + qslot * slot_stride, l + 1);
          const int ln = l + 2 < L ? l + 2 : 0;
          chain_gated_layer(s, WB, WA, rw, ln * lstr, qp, l + 1, L, par, step, lane, x);
        }
      }
      if (L & 1) {
#pragma unroll
        for (int c = 0; c < FCH; ++c) WA[c] = WB[c];
      }
      qslot = qslot + 1 == qdep ? 0 : qslot + 1;
      load_chunks(HA, rw, hvoff, o_head, 1024);
      __syncthreads();  // the skip sum is in LDS
      const float hv = head_row(HA, HB, rw, hvoff, o_head, s.srow, hbias);
      s.hrow[tid] = fmaxf(hv, 0.f);
      load_chunks(HA, rw, hvoff, o_out, 1024);
      __syncthreads();
      const float lv = head_row(HA, HB, rw, hvoff, o_out, s.hrow, obias);
      s.lrow[tid] = lv;
      if (a.mode != MODE_GENERATE && a.logits) a.logits[((long long)b * a.n_steps + step) * Q + tid] = lv;
      __syncthreads();
      if (a.mode == MODE_GENERATE) {
        const float4 lg = ((const float4 *)s.lrow)[lane];
        in = sample_row4(lg, s.u[(step / KCH & 1) * KCH + step % KCH]);
        if (lane == 0) a.samples[(long long)b * a.n_steps + step] = in;
      } else {
        in = s.fin[(step / KCH & 1) * KCH + step % KCH];
      }
      __syncthreads();  // the step's LDS rows and logits are consumed
    }
    if (lane == 0 && a.mode != MODE_TEACHER) a.last[b] = in;
  } else if (wave == 1) {
    // ---------------- the recurrent taps for the next step, staging, its share of the head
    const int lstr = FR * 1024;
    float4 WA[FR], WB[FR];
    load_chunks(WA, rw, lane * 16, o_rec, 1024);
    for (int step = 0; step < a.n_steps; ++step) {
      const int np = (step & 1) ^ 1;
      // lane l: the queue rows layer l's taps read next step
      long long toff[W - 1];
#pragma unroll
      for (int k = 0; k < W - 1; ++k) {
        int sk = qslot + k * qdil;
        sk = sk >= qdep ? sk - qdep : sk;
        toff[k] = qoff + sk * slot_stride;
      }
      for (int l = 0; l < L; l += 2) {
        {
          const float *taps[W - 1];
#pragma unroll
          for (int k = 0; k < W - 1; ++k) taps[k] = ring + lane_i64(toff[k], l);
          const int ln = l + 1 < L ? l + 1 : 0;
          rec_layer<W>(s, WA, WB, rw, o_rec + ln * lstr, taps, __builtin_amdgcn_readlane(qdil, l) == 1, g.convb, l,
                       L, np, step, lane);
        }
        if (l + 1 < L) {
          const float *taps[W - 1];
#pragma unroll
          for (int k = 0; k < W - 1; ++k) taps[k] = ring + lane_i64(toff[k], l + 1);
          const int ln = l + 2 < L ? l + 2 : 0;
          rec_layer<W>(s, WB, WA, rw, o_rec + ln * lstr, taps, __builtin_amdgcn_readlane(qdil, l + 1) == 1,
                       g.convb, l + 1, L, np, step, lane);
        }
      }
      if (L & 1) {
#pragma unroll
        for (int c = 0; c < FR; ++c) WA[c] = WB[c];
      }
      qslot = qslot + 1 == qdep ? 0 : qslot + 1;
      // staging of the next chunk of per-step inputs, one chunk ahead
      if (step % KCH == 0) {
        const int base = step + KCH, buf = (step / KCH + 1) & 1;
        for (int j = lane; j < KCH; j += 64) {
          const long long sj = base + j;
          if (a.mode == MODE_GENERATE) {
            s.u[buf * KCH + j] = sj < a.n_steps ? a.uniforms[(long long)b * a.n_steps + sj] : 0.f;
          } else {
            const long long nx = sj + forced_shift(a.mode);
            s.fin[buf * KCH + j] = nx < a.n_steps ? a.inputs[(long long)b * a.n_steps + nx] : 0;
          }
        }
      }
      load_chunks(HA, rw, hvoff, o_head, 1024);
      __syncthreads();
      const float hv = head_row(HA, HB, rw, hvoff, o_head, s.srow, hbias);
      s.hrow[tid] = fmaxf(hv, 0.f);
      load_chunks(HA, rw, hvoff, o_out, 1024);
      __syncthreads();
      const float lv = head_row(HA, HB, rw, hvoff, o_out, s.hrow, obias);
      s.lrow[tid] = lv;
      if (a.mode != MODE_GENERATE && a.logits) a.logits[((long long)b * a.n_steps + step) * Q + tid] = lv;
      __syncthreads();
      __syncthreads();
    }
  } else {
    // ---------------- the skip sum: channels 128 (wave - 2) + 2 lane and + 1, then the head
    const int wst = o_skip + (wave - 2) * FSK * 1024;
    const int lstr = 2 * FSK * 1024;
    const int m0 = 128 * (wave - 2) + 2 * lane;
    const float b0 = g.skipb[m0], b1 = g.skipb[m0 + 1];
    float4 WA[FSK], WB[FSK];
    load_chunks(WA, rw, lane * 16, wst, 1024);
    for (int step = 0; step < a.n_steps; ++step) {
      float s0 = b0, s1 = b1;
      for (int l = 0; l < L; l += 2) {
        skip_layer(s, WA, WB, rw, wst + (l + 1 < L ? l + 1 : 0) * lstr, lane, l, step, s0, s1);
        if (l + 1 < L) skip_layer(s, WB, WA, rw, wst + (l + 2 < L ? l + 2 : 0) * lstr, lane, l + 1, step, s0, s1);
      }
      if (L & 1) {
#pragma unroll
        for (int c = 0; c < FSK; ++c) WA[c] = WB[c];
      }
      s.srow[m0] = fmaxf(s0, 0.f);
      s.srow[m0 + 1] = fmaxf(s1, 0.f);
      load_chunks(HA, rw, hvoff, o_head, 1024);
      __syncthreads();
      const float hv = head_row(HA, HB, rw, hvoff, o_head, s.srow, hbias);
      s.hrow[tid] = fmaxf(hv, 0.f);
      load_chunks(HA, rw, hvoff, o_out, 1024);
      __syncthreads();
      const float lv = head_row(HA, HB, rw, hvoff, o_out, s.hrow, obias);
      s.lrow[tid] = lv;
      if (a.mode != MODE_GENERATE && a.logits) a.logits[((long long)b * a.n_steps + step) * Q + tid] = lv;
      __syncthreads();
      __syncthreads();
    }
  }
}

// ---------------------------------------------------------------------------
// Pair variant: the step of a stream on two blocks of one XCD, with the layer recurrence taken one
// layer ahead so that a single 32-wide product lies between consecutive gates.
//
// With x^l the input of layer l, z^l its gate output and x^{l+1} = x^l + W_res^l z^l + b_res^l, the
// gate pre-activation of layer l + 1 is
//   a^{l+1} = [W_r v + b + W_e^{l+1} b_res^l] + W_e^{l+1} x^l + (W_e^{l+1} W_res^l) z^l,
// the same sum regrouped (float32, products of the layer's weights formed once per fwg_create in
// float64).  The first bracket is the recurrent part (its constant folded into the bias), the
// second is known once x^l is, a layer before z^l; only M^l z^l (M^l = W_e^{l+1} W_res^l, 64 x 32)
// waits for the gate of layer l.
//
// Chain block (h = 0), four waves:
//  - wave 0, the gates: a^l = P^l + U^l + M^{l-1} z^{l-1} (z^{l-1} broadcast from its LDS row), the
//    gate, z^l to LDS (+ flag) and to the helper as 32 tagged words;
//  - wave 1, the residual stream: x^0 from the embedding, then x^{l+1} = x^l + W_res^l z^l + b_res^l
//    (K split over the half-waves), each layer input to LDS (+ flag) and pushed to its queue;
//  - wave 2: the recurrent taps of every layer for the next step (as in the one-block kernel) and
//    the staging of per-step inputs;
//  - wave 3: U^l = W_e^l x^{l-1} (x^0 for l = 0), to LDS (+ flag).
// Helper block (h = 1): the skip sum, 64 channels per wave (wave 0 also receives the z words into
// its LDS row).  Head, both blocks, with each thread's weights resident in registers for the launch:
// the helper publishes relu(skip sum) and each block computes half of the hidden channels (thread:
// one K half of one row of the first 1x1).  Width 2: from its half of the hidden channels alone each
// block forms the partial logits of every class (thread: one class row of the output 1x1 over that
// half), the helper publishes its partials and the chain block adds them, so the hidden channels
// never cross between the blocks.  Width 3 (whose other weights leave no room for the output 1x1's
// partial products without spilling): the blocks exchange their hidden halves, each computes half of
// the classes (thread: one K half of one class row) and in generation the helper publishes its
// logits.  The chain block samples.
//
// Hand-offs are the tagged words of fwg_xchg.h (tag = step index in the launch + 1; zeroed before
// every launch).  No block overwrites a word before the other has read it: each block's next write
// of a word depends, through the step's hand-offs, on the other's read of the previous one.  Block i
// of the launch: XCD slot i mod 8, pair (i / 16) 8 + i mod 8, role (i / 8) mod 2, so a pair's blocks
// i and i + 8 share an XCD under round-robin dispatch (a launch handshake checks; words go through
// memory when they do not).

constexpr int PH = FH / 2;  // head chunks per thread (one K half of a 256-wide row)
__host__ __device__ inline size_t pair_words(int L) { return 736 + (size_t)32 * L; }
constexpr int PW_HS = 0, PW_Z = 96;  // handshake slots (chain block, helper, mode: 32 words each), z rows
__host__ __device__ inline int pw_s(int L) { return 96 + 32 * L; }                // 256: relu(skip sum)
__host__ __device__ inline int pw_h(int L, int h) { return 96 + 32 * L + 256 + 128 * h; }
__host__ __device__ inline int pw_l(int L) { return 96 + 32 * L + 512; }           // the helper's logits
__host__ __device__ inline int pw_p(int L) { return pw_h(L, 0); }  // 256: the helper's partial logits (width 2)

// LDS of the pair variant (in 4-byte words): embedding table and bias, P [2][L][64], U [L][64],
// xrow, zrow, resb [L][32], srow, hrow, lrow, part [256], u, fin [2][KCH], flags.
struct PL {
  float *embT, *embb, *P, *U, *xrow, *zrow, *resb, *srow, *hrow, *lrow, *part, *u;
  int *fin;
  lds_flag *fx, *fz, *fu;  // [L]: step + 1 once x^l / z^l / U^l of the step is in LDS
  lds_flag *abort_, *mode, *inval;
};
__host__ __device__ inline int pl_flag_off(int L) {
  return Q * R + R + 2 * L * 2 * R + L * 2 * R + 3 * L * R + 4 * 256 + 4 * KCH;
}
__host__ __device__ inline size_t pair_lds_floats(int L) { return (size_t)pl_flag_off(L) + 3 * L + 8; }
__device__ __forceinline__ PL make_pl(float *lds, int L) {
  PL s;
  s.embT = lds;
  s.embb = s.embT + Q * R;
  s.P = s.embb + R;
  s.U = s.P + 2 * L * 2 * R;
  s.xrow = s.U + L * 2 * R;
  s.zrow = s.xrow + L * R;
  s.resb = s.zrow + L * R;
  s.srow = s.resb + L * R;
  s.hrow = s.srow + 256;
  s.lrow = s.hrow + 256;
  s.part = s.lrow + 256;
  s.u = s.part + 256;
  s.fin = (int *)(s.u + 2 * KCH);
  s.fx = (lds_flag *)(lds + pl_flag_off(L));
  s.fz = s.fx + L;
  s.fu = s.fz + L;
  s.abort_ = s.fu + L;
  s.mode = s.abort_ + 1;
  s.inval = s.abort_ + 2;
  return s;
}

// 32-wide dot product of 8 weight chunks with a row broadcast from LDS, two accumulation chains.
__device__ __forceinline__ float dot32(const float4 (&w)[FZ], const float *row, float acc) {
  const float4 *r4 = (const float4 *)row;
  float a1 = 0.f;
#pragma unroll
  for (int c = 0; c < FZ; ++c) {
    const float4 v = r4[c];
    acc = fmaf(w[c].x, v.x, acc);
    a1 = fmaf(w[c].y, v.y, a1);
    acc = fmaf(w[c].z, v.z, acc);
    a1 = fmaf(w[c].w, v.w, a1);
  }
  return acc + a1;
}

struct PairX {
  xg::u64 *pw;            // this pair's words
  uint32_t *abort_w, *sticky;
  bool local;             // both blocks on one XCD
};

// Half of a head 1x1 from resident weights: one row over one half of the input channels (PH
// chunks), the input vector broadcast from LDS.
__device__ __forceinline__ float head_dot(const float4 (&Wt)[PH], const float *in) {
  const float4 *i4 = (const float4 *)in;
  float a0 = 0.f, a1 = 0.f;
#pragma unroll
  for (int c = 0; c < PH; ++c) {
    const float4 v = i4[c];
    a0 = fmaf(Wt[c].x, v.x, a0);
    a1 = fmaf(Wt[c].y, v.y, a1);
    a0 = fmaf(Wt[c].z, v.z, a0);
    a1 = fmaf(Wt[c].w, v.w, a1);
  }
  return a0 + a1;
}

// The head of one step in block h (every thread of both blocks).  Block h computes hidden channels
// 128 h .. 128 h + 127 (thread t: K half t / 128 of row t mod 128).  KS (width 2): over those
// channels alone, thread t computes the partial logit of class t; the helper publishes its partials
// and the chain block adds them to its own, so a logit is (hidden half 0 + hidden half 1) + bias, and
// on return the chain block holds all 256 logits in LDS and in forced modes has written them out.
// Otherwise the blocks exchange their hidden halves and block h computes classes 128 h .. 128 h + 127
// (thread t: K half t / 128 of class row t mod 128); on return the chain block holds all 256 logits
// in LDS in generation, and in forced modes each block has written its 128 classes out.  The helper's
// relu(skip sum) is already in its srow.
template <bool KS>
__device__ __forceinline__ void pair_head(const PL &s, const float4 (&W1)[PH], const float4 (&W2)[PH],
                                          const PairX &px, const StepArgs &a, int L, int b, int h, int step,
                                          float hbias, float obias) {
  const int tid = threadIdx.x, kh = tid >> 7, t2 = tid & 127;
  const uint32_t tag = step + 1;
  __syncthreads();  // the helper: every skip channel in LDS
  if (h == 1) {
    xg::put_word(px.pw + pw_s(L) + tid, __builtin_bit_cast(uint32_t, s.srow[tid]), tag, px.local);
  } else {
    uint32_t v[1];
    xg::wait_words<1, 1>(px.pw + pw_s(L) + tid, tag, v, px.abort_w, px.sticky);
    s.srow[tid] = __builtin_bit_cast(float, v[0]);
    __syncthreads();  // relu(skip sum) of all 256 channels
  }
  s.part[tid] = head_dot(W1, s.srow + 128 * kh);
  __syncthreads();
  if (KS) {
    if (tid < 128) s.hrow[128 * h + tid] = fmaxf(s.part[tid] + s.part[tid + 128] + hbias, 0.f);
    __syncthreads();  // this block's half of the hidden layer
    const float pl = head_dot(W2, s.hrow + 128 * h);
    if (h == 1) {
      xg::put_word(px.pw + pw_p(L) + tid, __builtin_bit_cast(uint32_t, pl), tag, px.local);
    } else {
      uint32_t v[1];
      xg::wait_words<1, 1>(px.pw + pw_p(L) + tid, tag, v, px.abort_w, px.sticky);
      const float lv = pl + __builtin_bit_cast(float, v[0]) + obias;
      s.lrow[tid] = lv;
      if (a.mode != MODE_GENERATE && a.logits) a.logits[((long long)b * a.n_steps + step) * Q + tid] = lv;
    }
    __syncthreads();  // the chain block has every logit
    return;
  }
  if (tid < 128) {
    const float hv = fmaxf(s.part[tid] + s.part[tid + 128] + hbias, 0.f);
    s.hrow[128 * h + tid] = hv;
    xg::put_word(px.pw + pw_h(L, h) + tid, __builtin_bit_cast(uint32_t, hv), tag, px.local);
  } else {
    uint32_t v[1];
    xg::wait_words<1, 1>(px.pw + pw_h(L, 1 - h) + t2, tag, v, px.abort_w, px.sticky);
    s.hrow[128 * (1 - h) + t2] = __builtin_bit_cast(float, v[0]);
  }
  __syncthreads();  // the hidden layer
  s.part[tid] = head_dot(W2, s.hrow + 128 * kh);
  __syncthreads();
  if (tid < 128) {
    const float lv = s.part[tid] + s.part[tid + 128] + obias;
    s.lrow[128 * h + tid] = lv;
    if (a.mode != MODE_GENERATE) {
      if (a.logits) a.logits[((long long)b * a.n_steps + step) * Q + 128 * h + tid] = lv;
    } else if (h == 1) {
      xg::put_word(px.pw + pw_l(L) + tid, __builtin_bit_cast(uint32_t, lv), tag, px.local);
    }
  } else if (h == 0 && a.mode == MODE_GENERATE) {
    uint32_t v[1];
    xg::wait_words<1, 1>(px.pw + pw_l(L) + t2, tag, v, px.abort_w, px.sticky);
    s.lrow[128 + t2] = __builtin_bit_cast(float, v[0]);
  }
  __syncthreads();  // the chain block has every logit in generation
}

template <int W>
__global__ void __launch_bounds__(NT) chain_pair_kernel(StepArgs a, ChainGatedArgs g) {
  constexpr int FR = FREC * (W - 1);  // wave 2's weight chunks per layer
  extern __shared__ float4 lds4[];
  float *lds = (float *)lds4;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kq = blockIdx.x >> 3, h = kq & 1, b = (kq >> 1) * 8 + (blockIdx.x & 7);
  if (b >= a.batch) return;  // the last pairs of the grid beyond the batch
  const int L = a.L;
  const PL s = make_pl(lds, L);
  PairX px;
  px.pw = (xg::u64 *)((char *)a.sp_comm + 256) + (size_t)b * pair_words(L);
  px.abort_w = (uint32_t *)a.sp_comm;
  px.sticky = a.sp_sticky;

  // ---- launch handshake: both blocks report their XCD; the chain block tells the helper whether
  // they share one
  if (tid == 0) {
    xg::put_word(px.pw + PW_HS + 32 * h, xg::xcd_id(), 1, false);
    uint32_t v[1];
    if (h == 0) {
      xg::wait_words<1, 1>(px.pw + PW_HS + 32, 1, v, px.abort_w, px.sticky);
      const uint32_t loc = v[0] == xg::xcd_id() ? 1u : 0u;
      xg::put_word(px.pw + PW_HS + 64, loc, 1, false);
      *s.mode = (int)loc;
    } else {
      xg::wait_words<1, 1>(px.pw + PW_HS + 64, 1, v, px.abort_w, px.sticky);
      *s.mode = (int)v[0];
    }
  }
  // ---- tables into LDS (the chain block), flags, the first chunk of per-step inputs.  Every
  // thread issues all of its loads before its first LDS store, so the launch waits for one memory
  // round trip here instead of one per loop iteration.
  if (h == 0) {
    typedef unsigned int v4u __attribute__((ext_vector_type(4)));
    constexpr int NE = Q * R / 4 / NT;  // 16-byte pieces of the embedding table per thread
    constexpr int NRB = 4;              // residual biases per thread in the first batch
    static_assert(Q * R / 4 == NE * NT && R <= NT && KCH <= NT, "tables split over the block");
    v4u ev[NE];
#pragma unroll
    for (int k = 0; k < NE; ++k) ev[k] = ((const v4u *)g.embT)[tid + k * NT];
    const float eb = tid < R ? g.embb[tid] : 0.f;
    float rb[NRB];
#pragma unroll
    for (int k = 0; k < NRB; ++k) rb[k] = tid + k * NT < L * R ? g.resb[tid + k * NT] : 0.f;
    float uj = 0.f;
    int fj = 0;
    if (tid < KCH) {
      if (a.mode == MODE_GENERATE) {
        if (tid < a.n_steps) uj = a.uniforms[(long long)b * a.n_steps + tid];
      } else {
        const long long nx = tid + forced_shift(a.mode);
        if (nx < a.n_steps) fj = a.inputs[(long long)b * a.n_steps + nx];
      }
    }
    int in0 = 0;
    if (tid == 0) in0 = a.mode == MODE_TEACHER ? a.inputs[(long long)b * a.n_steps] : a.last[b];
#pragma unroll
    for (int k = 0; k < NE; ++k) ((v4u *)s.embT)[tid + k * NT] = ev[k];
    if (tid < R) s.embb[tid] = eb;
#pragma unroll
    for (int k = 0; k < NRB; ++k)
      if (tid + k * NT < L * R) s.resb[tid + k * NT] = rb[k];
    for (int i = tid + NRB * NT; i < L * R; i += NT) s.resb[i] = g.resb[i];  // more than 32 layers
    if (tid < KCH) {
      if (a.mode == MODE_GENERATE) s.u[tid] = uj;
      else s.fin[tid] = fj;
    }
    if (tid == 0) *s.inval = in0;
  }
  for (int i = tid; i < L; i += NT) {
    s.fx[i] = 0;
    s.fz[i] = 0;
    s.fu[i] = 0;
  }
  if (tid == 0) *s.abort_ = 0;
  // lane l: layer l's queue (row offset of slot 0), dilation, depth (W - 1) d, slot of the step
  const long long slot_stride = (long long)a.bmax * R;
  long long qoff = 0;
  int qdil = 1, qdep = W - 1, qslot = 0;
  if (lane < L) {
    const LayerDev ld = a.layers[lane];
    qoff = ld.ring_off + (long long)b * R;
    qdil = ld.dil;
    qdep = ld.depth;
    qslot = (int)(a.t0 % (long long)qdep);
  }
  float *ring = (float *)a.ring;
  if (h == 0 && wave == 2) {
    // the recurrent taps of every layer for step 0 (bias with the folded W_e b_res term)
    for (int l = 0; l < L; ++l) {
      const float4 *w = g.wrec + (size_t)l * FR * 64 + lane;
      float acc = g.convb[l * 2 * R + lane];
#pragma unroll
      for (int k = 0; k < W - 1; ++k) {
        int sk = qslot + k * qdil;
        sk = sk >= qdep ? sk - qdep : sk;
        const float *v = ring + lane_i64(qoff + sk * slot_stride, l);
#pragma unroll
        for (int c = 0; c < FREC; ++c) {
          const float4 wv = w[(FREC * k + c) * 64];
          const float4 vv = *(const float4 *)(v + 4 * c);
          acc = fmaf(wv.x, vv.x, acc);
          acc = fmaf(wv.y, vv.y, acc);
          acc = fmaf(wv.z, vv.z, acc);
          acc = fmaf(wv.w, vv.w, acc);
        }
      }
      s.P[l * 2 * R + lane] = acc;
    }
    qslot = qslot + 1 == qdep ? 0 : qslot + 1;  // wave 2 works one step ahead
  }
  // this thread's K half of its rows of both head 1x1s, resident for the launch
  const char *wbase = (const char *)g.wchain;
  const Rsrc rw = make_rsrc(wbase, (int)((const char *)g.convb - wbase));
  const int o_rec = (int)((const char *)g.wrec - wbase), o_skip = (int)((const char *)g.wskip - wbase);
  const int o_head = (int)((const char *)g.whead - wbase), o_out = (int)((const char *)g.wout - wbase);
  const int o_m = (int)((const char *)g.wm - wbase);
  float4 W1[PH], W2[PH];
  load_chunks(W1, rw, lane * 16, o_head + (h * 4 + wave) * PH * 1024, 1024);
  load_chunks(W2, rw, lane * 16, o_out + (h * 4 + wave) * PH * 1024, 1024);
  constexpr bool KS = W == 2;  // the output 1x1 split by K (partial logits of every class per block)
  const float hbias = g.headb[128 * h + (tid & 127)], obias = KS ? g.outb[tid] : g.outb[128 * h + (tid & 127)];
  __syncthreads();
  px.local = *s.mode != 0;
  const int o = lane & (R - 1), hl = lane >> 5;

  if (h == 1) {
    // ---------------- helper: skip channel 64 wave + lane (wave 0 receives z), then the head
    const int wst = o_skip + wave * FZ * 1024, lstr = 4 * FZ * 1024;
    const int m = 64 * wave + lane;
    const float bm = g.skipb[m];
    float4 WA[FZ], WB[FZ];
    load_chunks(WA, rw, lane * 16, wst, 1024);
    for (int step = 0; step < a.n_steps; ++step) {
      float s0 = bm;
      for (int l = 0; l < L; l += 2) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const int le = l + e;
          if (le < L) {
            float4 (&Wc)[FZ] = e ? WB : WA;
            float4 (&Wn)[FZ] = e ? WA : WB;
            if (wave == 0) {
              if (lane < R) {
                uint32_t v[1];
                xg::wait_words<1, 1>(px.pw + PW_Z + le * R + lane, step + 1, v, px.abort_w, px.sticky);
                s.zrow[le * R + lane] = __builtin_bit_cast(float, v[0]);
              }
              compiler_fence();
              if (lane == 0) s.fz[le] = step + 1;
            } else {
              wait_flag(s, s.fz + le, step + 1);
            }
            s0 = dot32(Wc, s.zrow + le * R, s0);
            load_chunks(Wn, rw, lane * 16, wst + (le + 1 < L ? le + 1 : 0) * lstr, 1024);
          }
        }
      }
      if (L & 1) {
#pragma unroll
        for (int c = 0; c < FZ; ++c) WA[c] = WB[c];
      }
      s.srow[m] = fmaxf(s0, 0.f);
      pair_head<KS>(s, W1, W2, px, a, L, b, 1, step, hbias, obias);
      __syncthreads();
    }
  } else if (wave == 0) {
    // ---------------- the gates (publishing z), then the head and the sample
    const int lstr = FZ * 1024;
    float4 WA[FZ], WB[FZ];  // M^{l-1} rows at slot l
    load_chunks(WA, rw, lane * 16, o_m, 1024);
    int in = *s.inval;
    for (int step = 0; step < a.n_steps; ++step) {
      const int par = step & 1;
      float z = 0.f;
      for (int l = 0; l < L; l += 2) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const int le = l + e;
          if (le < L) {
            float4 (&Wc)[FZ] = e ? WB : WA;
            float4 (&Wn)[FZ] = e ? WA : WB;
            wait_flag(s, s.fu + le, step + 1);
            float acc = s.P[(par * L + le) * 2 * R + lane] + s.U[le * 2 * R + lane];
            if (le > 0) acc = dot32(Wc, s.zrow + (le - 1) * R, acc);
            const float v = gate_half(acc, lane < R);
            const auto sw = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, v),
                                                             __builtin_bit_cast(unsigned, v), false, false);
            z = __builtin_bit_cast(float, (unsigned)sw[0]) * __builtin_bit_cast(float, (unsigned)sw[1]);
            if (lane < R) s.zrow[le * R + o] = z;
            compiler_fence();
            if (lane == 0) s.fz[le] = step + 1;
            if (lane < R) xg::put_word(px.pw + PW_Z + le * R + o, __builtin_bit_cast(uint32_t, z), step + 1, px.local);
            // the next layer's weights, fetched once this layer's result is out
            load_chunks(Wn, rw, lane * 16, o_m + (le + 1 < L ? le + 1 : 0) * lstr, 1024);
          }
        }
      }
      if (L & 1) {
#pragma unroll
        for (int c = 0; c < FZ; ++c) WA[c] = WB[c];
      }
      pair_head<KS>(s, W1, W2, px, a, L, b, 0, step, hbias, obias);
      if (a.mode == MODE_GENERATE) {
        const float4 lg = ((const float4 *)s.lrow)[lane];
        in = sample_row4(lg, s.u[(step / KCH & 1) * KCH + step % KCH]);
        if (lane == 0) a.samples[(long long)b * a.n_steps + step] = in;
      } else {
        in = s.fin[(step / KCH & 1) * KCH + step % KCH];
      }
      if (lane == 0) *s.inval = in;
      __syncthreads();  // the step's LDS rows and logits are consumed; the next input is in LDS
    }
    if (lane == 0 && a.mode != MODE_TEACHER) a.last[b] = in;
  } else if (wave == 1) {
    // ---------------- the residual stream and the pushes, then the head
    const int lstr = FCH * 1024;
    float4 WA[4], WB[4];  // W_res half rows: chunks 8..11 of the layer's chain block
    load_chunks(WA, rw, lane * 16, 8 * 1024, 1024);
    for (int step = 0; step < a.n_steps; ++step) {
      const long long qrow = qoff + qslot * slot_stride;  // lane l: layer l's push row of this step
      const int in = *s.inval;
      float x = s.embT[in * R + o] + s.embb[o];
      for (int l = 0; l < L; l += 2) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const int le = l + e;
          if (le < L) {
            float4 (&Wc)[4] = e ? WB : WA;
            float4 (&Wn)[4] = e ? WA : WB;
            // x = x^le, the input of layer le, to its queue (and, for layer 0, to LDS: the rows of later
            // layers are written as soon as they are computed)
            if (lane < R) {
              if (le == 0) s.xrow[o] = x;
              ring[lane_i64(qrow, le) + o] = x;
            }
            compiler_fence();
            if (le == 0 && lane == 0) s.fx[0] = step + 1;
            if (le + 1 < L) {
              wait_flag(s, s.fz + le, step + 1);
              const float4 *z4 = (const float4 *)(s.zrow + le * R + 16 * hl);
              float r0 = 0.f, r1 = 0.f;
#pragma unroll
              for (int c = 0; c < 4; ++c) {
                const float4 zv = z4[c];
                r0 = fmaf(Wc[c].x, zv.x, r0);
                r1 = fmaf(Wc[c].y, zv.y, r1);
                r0 = fmaf(Wc[c].z, zv.z, r0);
                r1 = fmaf(Wc[c].w, zv.w, r1);
              }
              x = x + s.resb[le * R + o] + ch::halves_sum(r0 + r1);
              if (lane < R) s.xrow[(le + 1) * R + o] = x;
              compiler_fence();
              if (lane == 0) s.fx[le + 1] = step + 1;
              load_chunks(Wn, rw, lane * 16, (le + 1) * lstr + 8 * 1024, 1024);
            } else {
              load_chunks(Wn, rw, lane * 16, 8 * 1024, 1024);  // layer 0's, for the next step
            }
          }
        }
      }
      if (L & 1) {
#pragma unroll
        for (int c = 0; c < 4; ++c) WA[c] = WB[c];
      }
      qslot = qslot + 1 == qdep ? 0 : qslot + 1;
      pair_head<KS>(s, W1, W2, px, a, L, b, 0, step, hbias, obias);
      __syncthreads();
    }
  } else if (wave == 2) {
    // ---------------- the recurrent taps for the next step, staging, then the head
    const int lstr = FR * 1024;
    float4 WA[FR], WB[FR];
    load_chunks(WA, rw, lane * 16, o_rec, 1024);
    for (int step = 0; step < a.n_steps; ++step) {
      const int np = (step & 1) ^ 1;
      long long toff[W - 1];
#pragma unroll
      for (int k = 0; k < W - 1; ++k) {
        int sk = qslot + k * qdil;
        sk = sk >= qdep ? sk - qdep : sk;
        toff[k] = qoff + sk * slot_stride;
      }
      for (int l = 0; l < L; l += 2) {
        {
          const float *taps[W - 1];
#pragma unroll
          for (int k = 0; k < W - 1; ++k) taps[k] = ring + lane_i64(toff[k], l);
          const int ln = l + 1 < L ? l + 1 : 0;
          rec_layer<W>(s, WA, WB, rw, o_rec + ln * lstr, taps, __builtin_amdgcn_readlane(qdil, l) == 1, g.convb, l,
                       L, np, step, lane);
        }
        if (l + 1 < L) {
          const float *taps[W - 1];
#pragma unroll
          for (int k = 0; k < W - 1; ++k) taps[k] = ring + lane_i64(toff[k], l + 1);
          const int ln = l + 2 < L ? l + 2 : 0;
          rec_layer<W>(s, WB, WA, rw, o_rec + ln * lstr, taps, __builtin_amdgcn_readlane(qdil, l + 1) == 1,
                       g.convb, l + 1, L, np, step, lane);
        }
      }
      if (L & 1) {
#pragma unroll
        for (int c = 0; c < FR; ++c) WA[c] = WB[c];
      }
      qslot = qslot + 1 == qdep ? 0 : qslot + 1;
      if (step % KCH == 0) {
        const int base = step + KCH, buf = (step / KCH + 1) & 1;
        for (int j = lane; j < KCH; j += 64) {
          const long long sj = base + j;
          if (a.mode == MODE_GENERATE) {
            s.u[buf * KCH + j] = sj < a.n_steps ? a.uniforms[(long long)b * a.n_steps + sj] : 0.f;
          } else {
            const long long nx = sj + forced_shift(a.mode);
            s.fin[buf * KCH + j] = nx < a.n_steps ? a.inputs[(long long)b * a.n_steps + nx] : 0;
          }
        }
      }
      pair_head<KS>(s, W1, W2, px, a, L, b, 0, step, hbias, obias);
      __syncthreads();
    }
  } else {
    // ---------------- U^l = W_e^l x^{l-1} (x^0 for l = 0), then the head
    const int lstr = FCH * 1024;
    float4 WA[FZ], WB[FZ];  // W_e rows: chunks 0..7 of the layer's chain block
    load_chunks(WA, rw, lane * 16, 0, 1024);
    for (int step = 0; step < a.n_steps; ++step) {
      for (int l = 0; l < L; l += 2) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const int le = l + e;
          if (le < L) {
            float4 (&Wc)[FZ] = e ? WB : WA;
            float4 (&Wn)[FZ] = e ? WA : WB;
            const int src = le > 0 ? le - 1 : 0;
            wait_flag(s, s.fx + src, step + 1);
            s.U[le * 2 * R + lane] = dot32(Wc, s.xrow + src * R, 0.f);
            compiler_fence();
            if (lane == 0) s.fu[le] = step + 1;
            load_chunks(Wn, rw, lane * 16, (le + 1 < L ? le + 1 : 0) * lstr, 1024);
          }
        }
      }
      if (L & 1) {
#pragma unroll
        for (int c = 0; c < FZ; ++c) WA[c] = WB[c];
      }
      pair_head<KS>(s, W1, W2, px, a, L, b, 0, step, hbias, obias);
      __syncthreads();
    }
  }
}

// ---- packing (once per fwg_create)
// pair: the pair variant's skip layout ([L][4 waves][8 chunks][64]: channel 64 wave + lane).
__global__ void pack_layer_kernel(const float *conv, const float *res, const float *skip, int l, int w, int pair,
                                  ChainGatedArgs g) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  const int nchain = FCH * 64, nrec = FREC * (w - 1) * 64, nskip = 2 * FSK * 64;
  float v[4];
  if (e < nchain) {
    const int c = e / 64, ln = e % 64;
    for (int q = 0; q < 4; ++q) {
      if (c < 8) v[q] = conv[((size_t)ln * R + 4 * c + q) * w + w - 1];           // W_e[ln][k] (current-input tap)
      else v[q] = res[(size_t)(ln % R) * R + 16 * (ln / R) + 4 * (c - 8) + q];    // W_res row, this lane's half
    }
    ((float4 *)g.wchain)[(size_t)l * nchain + e] = make_float4(v[0], v[1], v[2], v[3]);
  } else if (e < nchain + nrec) {
    // recurrent tap t = c / 8 (t = 0: the oldest state), columns 4 (c mod 8) ..
    const int f = e - nchain, c = f / 64, ln = f % 64, t = c / FREC, cc = c % FREC;
    for (int q = 0; q < 4; ++q) v[q] = conv[((size_t)ln * R + 4 * cc + q) * w + t];
    ((float4 *)g.wrec)[(size_t)l * nrec + f] = make_float4(v[0], v[1], v[2], v[3]);
  } else if (e < nchain + nrec + nskip) {
    const int f = e - nchain - nrec;
    int m, k0;
    if (pair) {
      const int wv = f / (FZ * 64), c = (f / 64) % FZ, ln = f % 64;
      m = 64 * wv + ln;
      k0 = 4 * c;
    } else {
      const int wv = f / (FSK * 64), c = (f / 64) % FSK, ln = f % 64;
      m = 128 * wv + 2 * ln + (c >= 8 ? 1 : 0);
      k0 = 4 * (c & 7);
    }
    for (int q = 0; q < 4; ++q) v[q] = skip[(size_t)m * R + k0 + q];
    ((float4 *)g.wskip)[(size_t)l * nskip + f] = make_float4(v[0], v[1], v[2], v[3]);
  }
}
// Single block: f = (wave, chunk, lane), row t = 64 wave + lane, columns 4 chunk .. 4 chunk + 3.
// Pair (pair = 1, 2): f = (block h, wave, j, lane), thread t = 64 wave + lane, row 128 h + t mod 128,
// chunk PH (t / 128) + j (the thread's K half); with pair = 2 the output 1x1 instead gives thread t
// class row t, chunk PH h + j (the block's half of the hidden channels).
__global__ void pack_head_kernel(const float *head, const float *out, int pair, ChainGatedArgs g) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= 2 * FH * NT) return;
  const int which = e / (FH * NT), f = e % (FH * NT);
  int t, c;
  if (pair) {
    const int hb = f / (4 * PH * 64), wv = (f / (PH * 64)) % 4, j = (f / 64) % PH, tt = 64 * wv + f % 64;
    const bool ks = pair == 2 && which;
    t = ks ? tt : 128 * hb + (tt & 127);
    c = ks ? PH * hb + j : PH * (tt >> 7) + j;
  } else {
    const int wv = f / (FH * 64);
    c = (f / 64) % FH;
    t = 64 * wv + f % 64;
  }
  const float *src = which ? out : head;
  float v[4];
  for (int q = 0; q < 4; ++q) v[q] = src[(size_t)t * 256 + 4 * c + q];
  ((float4 *)(which ? g.wout : g.whead))[f] = make_float4(v[0], v[1], v[2], v[3]);
}
// Pair variant: M^l = W_e^{l+1} W_res^l (64 x 32, float64 sums) at slot l + 1 of wm, rows per lane.
__global__ void pack_m_kernel(const float *conv_next, const float *res, int slot, int w, ChainGatedArgs g) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= FZ * 64) return;
  const int c = e / 64, o = e % 64;
  float v[4];
  for (int q = 0; q < 4; ++q) {
    const int k = 4 * c + q;
    double acc = 0.0;
    for (int j = 0; j < R; ++j) acc += (double)conv_next[((size_t)o * R + j) * w + w - 1] * (double)res[(size_t)j * R + k];
    v[q] = (float)acc;
  }
  ((float4 *)g.wm)[(size_t)slot * FZ * 64 + e] = make_float4(v[0], v[1], v[2], v[3]);
}
// Pair variant: the bias of layer l's recurrent part gains W_e^l b_res^{l-1} (float64 sum).
__global__ void pack_fold_kernel(const float *conv, const float *res_b_prev, int l, int w, ChainGatedArgs g) {
  const int o = blockIdx.x * blockDim.x + threadIdx.x;
  if (o >= 2 * R || res_b_prev == nullptr) return;
  double acc = 0.0;
  for (int j = 0; j < R; ++j) acc += (double)conv[((size_t)o * R + j) * w + w - 1] * (double)res_b_prev[j];
  float *cb = (float *)g.convb + (size_t)l * 2 * R;
  cb[o] = (float)((double)cb[o] + acc);
}
__global__ void pack_vec_kernel(const float *src, float *dst, int n, int accumulate) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= n) return;
  const float v = src ? src[e] : 0.f;
  dst[e] = accumulate ? dst[e] + v : v;
}

}  // namespace chg

bool chain_gated_ok(int kind, int dtype, int C, int S, int H, int Q, int L, int w, size_t *img_bytes, size_t *lds) {
  if (kind != 2 || dtype != 0 || C != kChainGR || S != kChainGS || H != kChainGS || Q != 256 || w < 2 ||
      w > kChainGMaxWidth || L < 1 || L > kChainGMaxLayers)
    return false;
  const ChainGatedArgs g = chain_gated_arrays(nullptr, L, w);
  *img_bytes = (size_t)(uintptr_t)(g.embb + kChainGR);
  *lds = chg::lds_floats(L) * 4;
  return *lds <= 160 * 1024;
}

ChainGatedArgs chain_gated_arrays(void *base, int L, int w) {
  using namespace chg;
  uintptr_t p = (uintptr_t)base;
  auto take = [&](size_t bytes) {
    const uintptr_t at = p;
    p += (bytes + 255) & ~(size_t)255;
    return at;
  };
  ChainGatedArgs g;
  g.wchain = (const float4 *)take((size_t)L * FCH * 64 * 16);
  g.wrec = (const float4 *)take((size_t)L * FREC * (w - 1) * 64 * 16);
  g.wskip = (const float4 *)take((size_t)L * 2 * FSK * 64 * 16);
  g.whead = (const float4 *)take((size_t)FH * NT * 16);
  g.wout = (const float4 *)take((size_t)FH * NT * 16);
  g.wm = (const float4 *)take((size_t)L * FZ * 64 * 16);
  g.convb = (const float *)take((size_t)L * 2 * R * 4);
  g.resb = (const float *)take((size_t)L * R * 4);
  g.skipb = (const float *)take((size_t)S * 4);
  g.headb = (const float *)take((size_t)H * 4);
  g.outb = (const float *)take((size_t)Q * 4);
  g.embT = (const float *)take((size_t)Q * R * 4);
  g.embb = (const float *)take((size_t)R * 4);
  return g;
}

static_assert(kChainGMaxWidth == 3, "the launcher instantiates filter widths 2 and 3");
hipError_t set_chain_gated_lds_limit(size_t bytes) {
  hipError_t e = hipFuncSetAttribute((const void *)chg::chain_gated_kernel<2>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute((const void *)chg::chain_gated_kernel<3>, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)bytes);
}

size_t chain_pair_lds_bytes(int L) { return chg::pair_lds_floats(L) * 4; }
size_t chain_pair_comm_bytes(int L, int batch) { return 256 + chg::pair_words(L) * 8 * (size_t)batch; }
int chain_pair_grid(int batch) { return 16 * ((batch + 7) / 8); }

hipError_t chain_pair_setup(size_t lds, int bmax, int *coresident_ok) {
  *coresident_ok = 0;
  hipError_t e;
  if ((e = hipFuncSetAttribute((const void *)chg::chain_pair_kernel<2>, hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)lds)) != hipSuccess)
    return e;
  if ((e = hipFuncSetAttribute((const void *)chg::chain_pair_kernel<3>, hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)lds)) != hipSuccess)
    return e;
  int dev = 0, cus = 0, per2 = 0, per3 = 0;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
  if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per2, chg::chain_pair_kernel<2>, chg::NT, lds)) != hipSuccess)
    return e;
  if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per3, chg::chain_pair_kernel<3>, chg::NT, lds)) != hipSuccess)
    return e;
  // every block of the largest launch resident at once (the blocks of a pair wait for each other)
  *coresident_ok = (long long)std::min(per2, per3) * cus >= (long long)chain_pair_grid(bmax);
  return hipSuccess;
}

hipError_t launch_chain_pair_step(const StepArgs &a, const ChainGatedArgs &g, size_t lds, hipStream_t s) {
  const dim3 grid(chain_pair_grid(a.batch));
  if (a.w == 3) hipLaunchKernelGGL(chg::chain_pair_kernel<3>, grid, dim3(chg::NT), lds, s, a, g);
  else hipLaunchKernelGGL(chg::chain_pair_kernel<2>, grid, dim3(chg::NT), lds, s, a, g);
  return hipGetLastError();
}

hipError_t launch_chain_gated_step(const StepArgs &a, const ChainGatedArgs &g, size_t lds, hipStream_t s) {
  if (a.w == 3) hipLaunchKernelGGL(chg::chain_gated_kernel<3>, dim3(a.batch), dim3(chg::NT), lds, s, a, g);
  else hipLaunchKernelGGL(chg::chain_gated_kernel<2>, dim3(a.batch), dim3(chg::NT), lds, s, a, g);
  return hipGetLastError();
}

hipError_t launch_chain_gated_pack(const void *embed, const float *embed_b, const void *const *conv,
                                   const float *const *conv_b, const void *const *res, const float *const *res_b,
                                   const void *const *skip, const float *const *skip_b, const void *head,
                                   const float *head_b, const void *out, const float *out_b, int L, int w, bool pair,
                                   const ChainGatedArgs &g, hipStream_t s) {
  using namespace chg;
  const int n = FCH * 64 + FREC * (w - 1) * 64 + 2 * FSK * 64;
  for (int l = 0; l < L; ++l) {
    hipLaunchKernelGGL(pack_layer_kernel, dim3((n + 255) / 256), dim3(256), 0, s, (const float *)conv[l],
                       (const float *)res[l], (const float *)skip[l], l, w, pair ? 1 : 0, g);
    hipLaunchKernelGGL(pack_vec_kernel, dim3(1), dim3(256), 0, s, conv_b ? conv_b[l] : nullptr,
                       (float *)g.convb + (size_t)l * 2 * R, 2 * R, 0);
    hipLaunchKernelGGL(pack_vec_kernel, dim3(1), dim3(256), 0, s, res_b ? res_b[l] : nullptr,
                       (float *)g.resb + (size_t)l * R, R, 0);
    hipLaunchKernelGGL(pack_vec_kernel, dim3(1), dim3(256), 0, s, skip_b ? skip_b[l] : nullptr, (float *)g.skipb, S,
                       l > 0);
  }
  // the pair kernel's output 1x1 is split by K at width 2 (pair_head)
  hipLaunchKernelGGL(pack_head_kernel, dim3((2 * FH * NT + 255) / 256), dim3(256), 0, s, (const float *)head,
                     (const float *)out, pair ? (w == 2 ? 2 : 1) : 0, g);
  hipLaunchKernelGGL(pack_vec_kernel, dim3(1), dim3(256), 0, s, head_b, (float *)g.headb, H, 0);
  hipLaunchKernelGGL(pack_vec_kernel, dim3(1), dim3(256), 0, s, out_b, (float *)g.outb, Q, 0);
  hipLaunchKernelGGL(ch::chain_transpose_kernel, dim3((R * Q + 255) / 256), dim3(256), 0, s, (const float *)embed,
                     (float *)g.embT, R, Q);
  hipLaunchKernelGGL(pack_vec_kernel, dim3(1), dim3(256), 0, s, embed_b, (float *)g.embb, R, 0);
  if (pair) {
    // slot 0 of wm is never read; zero it all the same
    hipLaunchKernelGGL(pack_vec_kernel, dim3(FZ * 64 * 4 / 256), dim3(256), 0, s, nullptr, (float *)g.wm, FZ * 64 * 4,
                       0);
    for (int l = 0; l + 1 < L; ++l)
      hipLaunchKernelGGL(pack_m_kernel, dim3((FZ * 64 + 255) / 256), dim3(256), 0, s, (const float *)conv[l + 1],
                         (const float *)res[l], l + 1, w, g);
    for (int l = 1; l < L; ++l)
      hipLaunchKernelGGL(pack_fold_kernel, dim3(1), dim3(2 * R), 0, s, (const float *)conv[l],
                         res_b ? res_b[l - 1] : nullptr, l, w, g);
  }
  return hipGetLastError();
}

}  // namespace fwg
