// Chain step kernel for small float32 ReLU stacks (channels C = 32, filter width 2): one block per
// stream, every weight and every queue of the stream in LDS for the whole launch.
//
// A sample's work is a chain of dependent steps (the layers in order, then the output 1x1 and the
// sample, which is the next input: Section 1, Section 2.2); at one stream nothing else can run beside
// it, so the kernel shortens that chain instead of widening it:
//  - wave 0 (the chain) keeps the layer input in lanes 0..31 (lane o holds channel o) and computes
//    each output o in lane o: the input values reach every lane as scalars read from their lanes
//    (v_readlane), the weights W_e^T[k][o] come from LDS (consecutive lanes, consecutive words);
//    the output 1x1 gives lane l the classes 4l..4l+3, and the sampler reduces them with DPP row
//    moves and lane reads;
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

namespace fwg {
namespace ch {

constexpr int C = kChainC, Q = 256;
constexpr int NT = 128;      // wave 0: the chain; wave 1: recurrent halves and staging
constexpr int KCH = 64;      // steps per chunk of staged uniforms / forced inputs
constexpr int SPIN_MAX = 1 << 24;

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}
__device__ __forceinline__ float lane_f(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}

// Inverse-CDF sample of one row of 256 logits held 4 per lane (lane l: classes 4l..4l+3): max, exp,
// inclusive prefix sums in class order (in-lane, then DPP shifts inside rows of 16 lanes, then the
// row totals), and the first class k with u Z < S_k, else the last class.  Wave-uniform result.
__device__ __forceinline__ int sample_row(float4 lg, float u, int lane) {
  float m = fmaxf(fmaxf(lg.x, lg.y), fmaxf(lg.z, lg.w));
  m = fmaxf(m, dpp<0xB1>(m));   // quad_perm [1,0,3,2]
  m = fmaxf(m, dpp<0x4E>(m));   // quad_perm [2,3,0,1]
  m = fmaxf(m, dpp<0x141>(m));  // row_half_mirror
  m = fmaxf(m, dpp<0x140>(m));  // row_mirror
  m = fmaxf(fmaxf(lane_f(m, 0), lane_f(m, 16)), fmaxf(lane_f(m, 32), lane_f(m, 48)));
  float c[4];
  c[0] = __expf(lg.x - m);
  c[1] = c[0] + __expf(lg.y - m);
  c[2] = c[1] + __expf(lg.z - m);
  c[3] = c[2] + __expf(lg.w - m);
  float incl = c[3];
  incl += dpp<0x111>(incl);  // row_shr:1
  incl += dpp<0x112>(incl);  // row_shr:2
  incl += dpp<0x114>(incl);  // row_shr:4
  incl += dpp<0x118>(incl);  // row_shr:8
  const float t0 = lane_f(incl, 15), t1 = lane_f(incl, 31), t2 = lane_f(incl, 47), t3 = lane_f(incl, 63);
  const int row = lane >> 4;
  incl += (row >= 1 ? t0 : 0.f) + (row >= 2 ? t1 : 0.f) + (row >= 3 ? t2 : 0.f);
  const float excl = incl - c[3];
  const float target = u * (((t0 + t1) + t2) + t3);
  int first = 4;
#pragma unroll
  for (int k = 3; k >= 0; --k)
    if (target < excl + c[k]) first = k;
  const unsigned long long hit = __ballot(first < 4);
  if (hit == 0ull) return Q - 1;
  const int src = __ffsll((long long)hit) - 1;
  return 4 * src + __builtin_amdgcn_readlane(first, src);
}

// The queue slot of layer l at time t, and byte offsets into the LDS image.
struct Lay {
  const float *img;   // LDS image (ChainArgs offsets, in floats)
  float *ring;        // LDS queues: layer l at ring + qoff[l] floats, [slot][C]
  float *pbuf;        // [2][L][C]: W_r v + b of every layer, by step parity
  int *qoff, *dil, *slot;  // per layer: float offset of the queue, dilation, slot at the current step
  volatile int *flag;      // per layer: step index + 1 once the chain pushed this step's input
  float *u;           // [2][KCH] staged uniforms (generation)
  int *fin;           // [2][KCH] staged forced next inputs
  float *lgs;         // [Q] logits of the step (forced modes, for the store)
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
  s.u = s.pbuf + 2 * L * C;
  s.fin = (int *)(s.u + 2 * KCH);
  s.qoff = s.fin + 2 * KCH;
  s.dil = s.qoff + L;
  s.slot = s.dil + L;
  s.flag = s.slot + L;
  int *cur_in = (int *)(s.flag + L);
  s.lgs = (float *)(cur_in + 4);

  // ---- launch: image, queues of this stream, per-layer tables, first input
  for (int i = tid; i < g.image_floats / 4; i += NT) lds4[i] = ((const float4 *)g.image)[i];
  {
    int off = 0;
    for (int l = 0; l < L; ++l) {
      const int d = a.layers[l].dil;
      if (tid == 0) {
        s.qoff[l] = off;
        s.dil[l] = d;
        s.slot[l] = (int)(a.t0 % (long long)d);
        s.flag[l] = 0;
      }
      const float *src = (const float *)a.ring + a.layers[l].ring_off;
      for (int i = tid; i < d * C; i += NT) {
        const int sl = i / C, ch = i % C;
        s.ring[off + i] = src[((long long)sl * a.bmax + b) * C + ch];
      }
      off += d * C;
    }
  }
  if (tid == 0) cur_in[0] = a.mode == MODE_TEACHER ? a.inputs[(long long)b * a.n_steps] : a.last[b];
  // stage chunk 0
  for (int j = tid; j < KCH; j += NT) {
    if (a.mode == MODE_GENERATE) s.u[j] = j < a.n_steps ? a.uniforms[(long long)b * a.n_steps + j] : 0.f;
    else {
      const long long nx = j + forced_shift(a.mode);
      s.fin[j] = nx < a.n_steps ? a.inputs[(long long)b * a.n_steps + nx] : 0;
    }
  }
  __syncthreads();

  const float *embT = s.img + g.o_emb;    // [Q][C]
  const float *embb = s.img + g.o_embb;   // [C]
  const float *woT = s.img + g.o_out;     // [C][Q]
  const float *wob = s.img + g.o_outb;    // [Q]
  const int o = lane & (C - 1);
  const bool residual = a.kind == 1;  // relu + residual (FWG_RELU_RESIDUAL)

  if (wave == 1) {
    // W_r v + b of every layer for step 0 (pops of step 0: all pushed before the launch)
    for (int l = 0; l < L; ++l) {
      const float *wrT = s.img + g.o_layer + l * g.layer_floats;  // W_r^T [C][C], then W_e^T, then b
      const float *v = s.ring + s.qoff[l] + s.slot[l] * C;
      float acc = wrT[2 * C * C + o];
      for (int k = 0; k < C; ++k) acc = fmaf(wrT[k * C + o], v[k], acc);
      if (lane < C) s.pbuf[l * C + o] = acc;
    }
  }
  __syncthreads();

  for (int step = 0; step < a.n_steps; ++step) {
    const int par = step & 1;
    if (wave == 0) {
      // ---- the chain: embedding, layers, output 1x1, sample
      const int in = cur_in[0];
      float x = embT[in * C + o] + embb[o];
      for (int l = 0; l < L; ++l) {
        const float *we = s.img + g.o_layer + l * g.layer_floats + C * C;  // W_e^T [C][C]
        // push: this layer's input replaces the slot the step pops (its value was read for this
        // step's W_r v one step earlier)
        if (lane < C) s.ring[s.qoff[l] + s.slot[l] * C + o] = x;
        if (lane == 0) s.flag[l] = step + 1;
        float w[C];
#pragma unroll
        for (int k = 0; k < C; ++k) w[k] = we[k * C + o];
        float acc = s.pbuf[(par * L + l) * C + o];
#pragma unroll
        for (int k = 0; k < C; ++k) acc = fmaf(w[k], lane_f(x, k), acc);
        const float r = fmaxf(acc, 0.f);
        x = residual ? x + r : r;
      }
      // output 1x1: lane l takes classes 4l..4l+3
      float4 lg = ((const float4 *)wob)[lane];
#pragma unroll 8
      for (int k = 0; k < C; ++k) {
        const float4 wv = ((const float4 *)(woT + k * Q))[lane];
        const float xk = lane_f(x, k);
        lg.x = fmaf(wv.x, xk, lg.x);
        lg.y = fmaf(wv.y, xk, lg.y);
        lg.z = fmaf(wv.z, xk, lg.z);
        lg.w = fmaf(wv.w, xk, lg.w);
      }
      int nxt;
      if (a.mode == MODE_GENERATE) {
        nxt = sample_row(lg, s.u[(step / KCH & 1) * KCH + step % KCH], lane);
        if (lane == 0) a.samples[(long long)b * a.n_steps + step] = nxt;
      } else {
        if (a.logits) ((float4 *)(a.logits + ((long long)b * a.n_steps + step) * Q))[lane] = lg;
        nxt = s.fin[(step / KCH & 1) * KCH + step % KCH];
      }
      if (lane == 0) cur_in[0] = nxt;
    } else {
      // ---- W_r v + b of every layer for the next step, into the other parity
      const int np = par ^ 1;
      for (int l = 0; l < L; ++l) {
        const int d = s.dil[l];
        const int sl = s.slot[l] + 1 == d ? 0 : s.slot[l] + 1;
        if (d == 1) {
          // the state popped next step is this step's input of the layer: wait for the chain's push
          for (int it = 0; s.flag[l] != step + 1 && it < SPIN_MAX; ++it) __builtin_amdgcn_s_sleep(1);
        }
        const float *wrT = s.img + g.o_layer + l * g.layer_floats;
        const float *v = s.ring + s.qoff[l] + sl * C;
        float acc = wrT[2 * C * C + o];
#pragma unroll 8
        for (int k = 0; k < C; ++k) acc = fmaf(wrT[k * C + o], v[k], acc);
        if (lane < C) s.pbuf[(np * L + l) * C + o] = acc;
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
    }
    __syncthreads();
    // slot advance (wave 1 read slot + 1 above; the chain reads the slots during the step)
    if (tid < L) s.slot[tid] = s.slot[tid] + 1 == s.dil[tid] ? 0 : s.slot[tid] + 1;
    __syncthreads();
  }

  // ---- launch end: queues and the pending input back to the workspace
  {
    for (int l = 0; l < L; ++l) {
      const int d = s.dil[l];
      float *dst = (float *)a.ring + a.layers[l].ring_off;
      for (int i = tid; i < d * C; i += NT) {
        const int sl = i / C, ch = i % C;
        dst[((long long)sl * a.bmax + b) * C + ch] = s.ring[s.qoff[l] + i];
      }
    }
    if (tid == 0 && a.mode != MODE_TEACHER) a.last[b] = cur_in[0];
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
  if ((kind != 0 && kind != 1) || dtype != 0 || C != kChainC || Q != 256 || w != 2 || L < 1 || L > 64) return false;
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
  const long long floats = (long long)g->image_floats + g->ring_floats + 2LL * L * C + 2 * ch::KCH +
                           2 * ch::KCH + 4LL * L + 4 + Q;
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
