// Wave-per-stream step kernel for models whose weights fit in LDS (gfx950).
//
// Small stacks (the toy ReLU stack of the paper's illustration, C = 32, L = 5) are bound by
// latency, not arithmetic: a 256-thread block pays a barrier and an L2 round trip on every layer.
// Here each wavefront carries one stream through the whole generation step (paper Section 2.2:
// pop, compute, push) on its own: every weight lives in LDS for the whole launch (copied once at
// the start from a float image prepared at create), the popped states of all layers of the next
// step are loaded into registers while the current step finishes (a pop never depends on the
// current step), and all exchanges between lanes go through the wave's own LDS scratch, so no
// block barrier is needed after the weight copy.  Four waves share one block and its weights.
//
// Products y[n] = b[n] + sum_k W^T[k][n] in[k] (wave_product): W^T rows are read contiguously
// across lanes and in[k] is broadcast.  Rounding points, layer kinds,
// filter width, sampling and forced modes are those of the other step kernels.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fwg_bf16.h"
#include "fwg_internal.h"
#include "fwg_wave.h"
#include "fwg_sample.h"

namespace fwg {
namespace wv {

// Orders this wave's LDS writes before its later reads by other lanes: LDS instructions of one wave
// execute in order, so only the compiler has to be kept from moving accesses across this point.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// y[n] += sum_k W^T[k][n] in[k] for W^T [K][N] (row stride N) and in[0..K).  Wide products
// (N > 32): lane n takes columns n, n + 64, ... over all of K.  Narrow ones (N <= 32): the wave
// splits into G = 64 / N' lane groups (N' = N rounded up to a power of two) that take K / G each
// (when 4 G divides K), and the partial sums are combined across groups, so every lane of every
// group ends with its column's full sum.  in[] is read four values at a time.
template <int NMAX>
__device__ __forceinline__ void wave_product(const float *WT, int K, int N, const float *in, float (&acc)[NMAX],
                                             int lane) {
  if (N <= 32) {
    int np = 1;
    while (np < N) np <<= 1;
    int G = 64 / np;
    while (G > 1 && K % (4 * G)) G >>= 1;
    const int n = lane & (np - 1), grp = lane / np;
    const int kper = K / G, k0 = grp * kper;
    float s = 0.f;
    if (n < N && grp < G) {
      const float *w = WT + (long long)k0 * N + n;
#pragma unroll 4
      for (int k = 0; k < kper; k += 4) {
        const float4 v = *(const float4 *)(in + k0 + k);
        s = fmaf(w[0], v.x, s);
        s = fmaf(w[N], v.y, s);
        s = fmaf(w[2 * N], v.z, s);
        s = fmaf(w[3 * N], v.w, s);
        w += 4 * N;
      }
    }
    for (int off = np; off < 64; off <<= 1) s += __shfl_xor(s, off, 64);
    acc[0] += s;  // lanes n, n + np, ... all hold column n
    return;
  }
#pragma unroll 2
  for (int k = 0; k < K; k += 4) {
    const float4 v = *(const float4 *)(in + k);
#pragma unroll
    for (int j = 0; j < NMAX; ++j) {
      const int n = lane + 64 * j;
      if (n < N) {
        const float *w = WT + (long long)k * N + n;
        acc[j] = fmaf(w[0], v.x, acc[j]);
        acc[j] = fmaf(w[N], v.y, acc[j]);
        acc[j] = fmaf(w[2 * N], v.z, acc[j]);
        acc[j] = fmaf(w[3 * N], v.w, acc[j]);
      }
    }
  }
}

// Column of a lane's acc[j] after wave_product: n = lane + 64 j for wide products; for narrow ones
// (N <= 32) column lane mod N' is held by several lanes, and only the first group writes it.
__device__ __forceinline__ int wave_col(int N, int lane, int j) {
  if (N <= 32) {
    int np = 1;
    while (np < N) np <<= 1;
    return (j == 0 && lane < np) ? lane : 1 << 30;
  }
  return lane + 64 * j;
}

template <bool BF16>
__device__ __forceinline__ float opnd(float v) {
  return BF16 ? round_bf16(v) : v;
}
template <bool BF16>
__device__ __forceinline__ float ring_load(const void *ring, long long i) {
  return BF16 ? __uint_as_float(((uint32_t)((const uint16_t *)ring)[i]) << 16) : ((const float *)ring)[i];
}
template <bool BF16>
__device__ __forceinline__ void ring_store(void *ring, long long i, float v) {
  if (BF16) ((uint16_t *)ring)[i] = bf16_bits(v);
  else ((float *)ring)[i] = v;
}

constexpr int NMAX = 4;   // columns per lane: products up to 256 outputs (the 256 logits)
constexpr int PMAX = 16;  // popped values per lane and step held in registers

// CR: channels per lane (C <= 64 CR).
template <bool BF16, int CR>
__global__ void __launch_bounds__(256) wave_step_kernel(StepArgs a, WaveArgs g) {
  extern __shared__ float4 lds4[];
  float *lds = (float *)lds4;
  // the weight image, once per launch
  {
    const float4 *src = (const float4 *)g.image;
    for (int i = threadIdx.x; i < g.image_floats / 4; i += 256) lds4[i] = src[i];
  }
  __syncthreads();
  const int wvi = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int b = blockIdx.x * 4 + wvi;
  if (b >= a.batch) return;  // no block barrier follows

  const int C = a.C, S = a.S, H = a.H, Q = a.Q, L = a.L, w = a.w;
  const bool gated = a.kind == 2;
  const int Co = gated ? 2 * C : C, K = w * C;
  float *scr = lds + g.image_floats + wvi * g.scr_floats;
  float *pin = scr;                   // [L][w C] layer inputs: taps 0 .. w-2 popped, tap w-1 current
  float *xs = pin + g.ain_floats;     // [C] float32 stream x^l
  float *zb = xs + g.c_floats;        // [C] gate output (operand)
  float *sb = zb + g.c_floats;        // [S] skip sum
  float *rs = sb + g.s_floats;        // [S] operand of relu(s)
  float *hb = rs + g.s_floats;        // [H] head hidden (operand)
  float *lg = hb + g.h_floats;        // [Q] logits

  // lane l < L: layer l's queue (offset, depth, slot of the current step) for its push
  int depth_l = 1, slot_l = 0;
  long long roff_l = 0;
  if (lane < L) {
    const LayerDev ld = a.layers[lane];
    depth_l = ld.depth;
    roff_l = ld.ring_off;
    slot_l = (int)(a.t0 % (long long)ld.depth);
  }
  // lane j < L (w - 1): pop pair j = (layer j / (w - 1), tap j % (w - 1)): its slot counter (the
  // state k d slots after the oldest one of that layer), the address of this stream's row in that
  // slot, and where the popped row goes in the layer inputs
  const int W1 = w - 1, npair = L * W1;
  int pj_slot = 0, pj_depth = 1, pj_dst = 0;
  long long pj_addr = 0, pj_base = 0;
  const long long slot_stride = (long long)a.bmax * C;
  if (lane < npair) {
    const int l = lane / W1, k = lane - l * W1;
    const LayerDev ld = a.layers[l];
    pj_depth = ld.depth;
    pj_base = ld.ring_off + (long long)b * C;
    pj_slot = (int)((a.t0 + (long long)k * ld.dil) % (long long)ld.depth);
    pj_addr = pj_base + pj_slot * slot_stride;
    pj_dst = l * K + k * C;
  }
  float pp[PMAX];
  // the pops of the step whose slot counters are current: entry i = (pair i / CR, channel block i % CR)
  auto fetch = [&]() {
#pragma unroll
    for (int i = 0; i < PMAX; ++i) {
      float v = 0.f;
      const int j = i / CR, cr = i % CR;
      if (j < npair) {
        const int c = lane + 64 * cr;
        const long long addr = ((long long)__builtin_amdgcn_readlane((int)(pj_addr >> 32), j) << 32) |
                               (uint32_t)__builtin_amdgcn_readlane((int)pj_addr, j);
        if (c < C) v = ring_load<BF16>(a.ring, addr + c);
      }
      pp[i] = v;
    }
  };
  auto land = [&]() {
#pragma unroll
    for (int i = 0; i < PMAX; ++i) {
      const int j = i / CR, cr = i % CR;
      if (j < npair) {
        const int c = lane + 64 * cr;
        if (c < C) pin[__builtin_amdgcn_readlane(pj_dst, j) + c] = pp[i];
      }
    }
  };

  int in = a.mode == MODE_TEACHER ? a.inputs[(long long)b * a.n_steps] : a.last[b];
  fetch();
  const float *embT = lds + g.o_emb, *embB = lds + g.o_embb;

  for (int s = 0; s < a.n_steps; ++s) {
    // ---- h^0_e: the embedding row of the current input; this step's pops into the layer inputs
    for (int c = lane; c < C; c += 64) xs[c] = embT[(long long)in * C + c] + embB[c];
    if (gated)
      for (int m = lane; m < S; m += 64) sb[m] = 0.f;
    land();
    wave_sync();
    for (int l = 0; l < L; ++l) {
      const float *blk = lds + g.o_layer + (long long)l * g.layer_floats;
      float *ain = pin + l * K;
      const int sl = __builtin_amdgcn_readlane(slot_l, l);
      const long long ro = ((long long)__builtin_amdgcn_readlane((int)(roff_l >> 32), l) << 32) |
                           (uint32_t)__builtin_amdgcn_readlane((int)roff_l, l);
      // the current state completes the layer input and replaces the popped oldest state
      // (pop before push, Section 2.2)
      for (int c = lane; c < C; c += 64) {
        const float x = opnd<BF16>(xs[c]);
        ain[(w - 1) * C + c] = x;
        ring_store<BF16>(a.ring, ro + ((long long)sl * a.bmax + b) * C + c, x);
      }
      wave_sync();
      // dilated product of width w
      const float *convT = blk, *convB = blk + g.o_convb;
      float acc[NMAX];
      if (gated) {
        // lane n: the tanh row n and the sigmoid row C + n of one channel
        float acc2[NMAX];
#pragma unroll
        for (int j = 0; j < NMAX; ++j) {
          const int n = lane + 64 * j;
          acc[j] = n < C ? convB[n] : 0.f;
          acc2[j] = n < C ? convB[C + n] : 0.f;
        }
#pragma unroll 2
        for (int k = 0; k < K; k += 4) {
          const float4 v = *(const float4 *)(ain + k);
#pragma unroll
          for (int j = 0; j < NMAX; ++j) {
            const int n = lane + 64 * j;
            if (n < C) {
              const float *wt = convT + (long long)k * Co + n;
              acc[j] = fmaf(wt[0], v.x, fmaf(wt[Co], v.y, fmaf(wt[2 * Co], v.z, fmaf(wt[3 * Co], v.w, acc[j]))));
              const float *ws = wt + C;
              acc2[j] = fmaf(ws[0], v.x, fmaf(ws[Co], v.y, fmaf(ws[2 * Co], v.z, fmaf(ws[3 * Co], v.w, acc2[j]))));
            }
          }
        }
#pragma unroll
        for (int j = 0; j < NMAX; ++j) {
          const int n = lane + 64 * j;
          if (n < C) {
            const float t = 1.f - 2.f * __builtin_amdgcn_rcpf(__expf(2.f * acc[j]) + 1.f);
            const float sg = __builtin_amdgcn_rcpf(1.f + __expf(-acc2[j]));
            zb[n] = opnd<BF16>(t * sg);
          }
        }
        wave_sync();
        // residual and skip 1x1 products
        const float *resT = blk + g.o_res, *resB = blk + g.o_resb, *skT = blk + g.o_skip, *skB = blk + g.o_skipb;
#pragma unroll
        for (int j = 0; j < NMAX; ++j) acc[j] = 0.f;
        wave_product<NMAX>(resT, C, C, zb, acc, lane);
#pragma unroll
        for (int j = 0; j < NMAX; ++j) {
          const int n = wave_col(C, lane, j);
          if (n < C) xs[n] += resB[n] + acc[j];
        }
        float acs[NMAX];
#pragma unroll
        for (int j = 0; j < NMAX; ++j) acs[j] = 0.f;
        wave_product<NMAX>(skT, C, S, zb, acs, lane);
#pragma unroll
        for (int j = 0; j < NMAX; ++j) {
          const int m = wave_col(S, lane, j);
          if (m < S) sb[m] += skB[m] + acs[j];
        }
      } else {
#pragma unroll
        for (int j = 0; j < NMAX; ++j) acc[j] = 0.f;
        wave_product<NMAX>(convT, K, Co, ain, acc, lane);
#pragma unroll
        for (int j = 0; j < NMAX; ++j) {
          const int n = wave_col(Co, lane, j);
          if (n < C) xs[n] = (a.kind == 1 ? xs[n] : 0.f) + fmaxf(convB[n] + acc[j], 0.f);
        }
      }
      wave_sync();
    }
    // the next step's pops (every push of this step has been made); slot counters advance
    {
      int nx = slot_l + 1;
      slot_l = nx == depth_l ? 0 : nx;
      nx = pj_slot + 1;
      pj_slot = nx == pj_depth ? 0 : nx;
      pj_addr = pj_base + pj_slot * slot_stride;
    }
    if (s + 1 < a.n_steps) fetch();

    // ---- output head
    float acc[NMAX];
    const float *outT = lds + g.o_out, *outB = lds + g.o_outb;
    if (gated) {
      for (int m = lane; m < S; m += 64) rs[m] = opnd<BF16>(fmaxf(sb[m], 0.f));
      wave_sync();
      const float *hT = lds + g.o_head, *hB = lds + g.o_headb;
#pragma unroll
      for (int j = 0; j < NMAX; ++j) acc[j] = 0.f;
      wave_product<NMAX>(hT, S, H, rs, acc, lane);
#pragma unroll
      for (int j = 0; j < NMAX; ++j) {
        const int n = wave_col(H, lane, j);
        if (n < H) hb[n] = opnd<BF16>(fmaxf(hB[n] + acc[j], 0.f));
      }
      wave_sync();
#pragma unroll
      for (int j = 0; j < NMAX; ++j) acc[j] = 0.f;
      wave_product<NMAX>(outT, H, Q, hb, acc, lane);
    } else {
      for (int c = lane; c < C; c += 64) zb[c] = opnd<BF16>(xs[c]);
      wave_sync();
#pragma unroll
      for (int j = 0; j < NMAX; ++j) acc[j] = 0.f;
      wave_product<NMAX>(outT, C, Q, zb, acc, lane);
    }
#pragma unroll
    for (int j = 0; j < NMAX; ++j) {
      const int q = wave_col(Q, lane, j);
      if (q < Q) lg[q] = outB[q] + acc[j];
    }
    wave_sync();
    if (a.mode != MODE_GENERATE) {
      if (a.logits)
        for (int q = lane; q < Q; q += 64) a.logits[((long long)b * a.n_steps + s) * Q + q] = lg[q];
      const int nx = s + forced_shift(a.mode);
      if (nx < a.n_steps) in = a.inputs[(long long)b * a.n_steps + nx];
    } else {
      const int k = sample_row_256(lg, a.uniforms[(long long)b * a.n_steps + s]);
      if (lane == 0) a.samples[(long long)b * a.n_steps + s] = k;
      in = k;
    }
    wave_sync();
  }
  if (a.mode != MODE_TEACHER && lane == 0) a.last[b] = in;
}

// ---------------------------------------------------------------------------
// The weight image (floats): W^T of every product, k-major, so lanes read consecutive columns.
template <typename T>
__device__ __forceinline__ float to_f(T v);
template <>
__device__ __forceinline__ float to_f<float>(float v) { return v; }
template <>
__device__ __forceinline__ float to_f<uint16_t>(uint16_t v) { return __uint_as_float(((uint32_t)v) << 16); }

// dst[k * N + n] = W[n][k] of a PyTorch [N][K] matrix; conv [Co][C][w] with k = tap * C + c
template <typename T>
__global__ void wave_image_kernel(const T *src, float *dst, int N, int K, int C, int conv) {
  const long long total = (long long)N * K;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (long long)gridDim.x * blockDim.x) {
    const int k = (int)(i / N), n = (int)(i - (long long)k * N);
    long long si;
    if (conv) {
      const int w = K / C, tap = k / C, c = k - tap * C;
      si = ((long long)n * C + c) * w + tap;
    } else {
      si = (long long)n * K + k;
    }
    dst[i] = to_f<T>(src[si]);
  }
}

__global__ void wave_vec_kernel(const float *src, float *dst, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = src ? src[i] : 0.f;
}

}  // namespace wv

template <bool BF16>
static hipError_t launch_wave_t(const StepArgs &a, const WaveArgs &g, hipStream_t s) {
  const dim3 grid((a.batch + 3) / 4), block(256);
  const size_t lds = sizeof(float) * ((size_t)g.image_floats + 4 * (size_t)g.scr_floats);
  const int cr = (a.C + 63) / 64;
  if (cr == 1) hipLaunchKernelGGL((wv::wave_step_kernel<BF16, 1>), grid, block, lds, s, a, g);
  else if (cr == 2) hipLaunchKernelGGL((wv::wave_step_kernel<BF16, 2>), grid, block, lds, s, a, g);
  else hipLaunchKernelGGL((wv::wave_step_kernel<BF16, 4>), grid, block, lds, s, a, g);
  return hipGetLastError();
}

hipError_t launch_wave_step(const StepArgs &a, const WaveArgs &g, hipStream_t s) {
  return a.dtype == 1 ? launch_wave_t<true>(a, g, s) : launch_wave_t<false>(a, g, s);
}

template <bool BF16, int CR>
static hipError_t set_wave_lds_one(size_t bytes) {
  return hipFuncSetAttribute((const void *)wv::wave_step_kernel<BF16, CR>, hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)bytes);
}

hipError_t set_wave_lds_limit(size_t bytes) {
  hipError_t e;
  if ((e = set_wave_lds_one<true, 1>(bytes)) != hipSuccess) return e;
  if ((e = set_wave_lds_one<true, 2>(bytes)) != hipSuccess) return e;
  if ((e = set_wave_lds_one<true, 4>(bytes)) != hipSuccess) return e;
  if ((e = set_wave_lds_one<false, 1>(bytes)) != hipSuccess) return e;
  if ((e = set_wave_lds_one<false, 2>(bytes)) != hipSuccess) return e;
  return set_wave_lds_one<false, 4>(bytes);
}

hipError_t launch_wave_image(const void *src, float *dst, int dtype, int N, int K, int C, int conv, hipStream_t s) {
  const long long total = (long long)N * K;
  const int grid = (int)((total + 255) / 256 < 4096 ? (total + 255) / 256 : 4096);
  if (dtype == 1)
    hipLaunchKernelGGL(wv::wave_image_kernel<uint16_t>, dim3(grid), dim3(256), 0, s, (const uint16_t *)src, dst, N,
                       K, C, conv);
  else
    hipLaunchKernelGGL(wv::wave_image_kernel<float>, dim3(grid), dim3(256), 0, s, (const float *)src, dst, N, K, C,
                       conv);
  return hipGetLastError();
}

hipError_t launch_wave_vec(const float *src, float *dst, int n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(wv::wave_vec_kernel, dim3((n + 255) / 256), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

}  // namespace fwg
