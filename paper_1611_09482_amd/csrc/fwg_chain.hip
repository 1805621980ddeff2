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

#include "fwg_chain.h"
#include "fwg_internal.h"
#include "fwg_sample.h"

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
