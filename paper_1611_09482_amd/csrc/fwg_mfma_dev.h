// Device helpers shared by the bf16 MFMA step kernels (fwg_mfma.hip, fwg_split.hip): the
// v_mfma_f32_16x16x32_bf16 wrapper, bf16 packing, the gate, LDS row moves and the wave-wide
// inverse-CDF sampler over 256 classes.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fwg {
namespace mfd {

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
__device__ __forceinline__ void stf4(float *p, const f32x4 &v) { *(float4 *)p = make_float4(v[0], v[1], v[2], v[3]); }
__device__ __forceinline__ f32x4 relu4(const f32x4 &v) {
  return f32x4{fmaxf(v[0], 0.f), fmaxf(v[1], 0.f), fmaxf(v[2], 0.f), fmaxf(v[3], 0.f)};
}

// Cross-lane moves inside rows of 16 lanes (DPP) and lane reads, for the wave-wide max and scan of
// the sampler.  Control codes: quad permutations, row_shr:n = 0x110 + n, row_mirror = 0x140,
// row_half_mirror = 0x141; bound_ctrl makes a source lane outside the row read 0.
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}
__device__ __forceinline__ float lane_f(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}

// Inverse-CDF samples of two rows of 256 logits by one wavefront: lanes 0..31 take row A,
// lanes 32..63 row B, each lane 8 consecutive classes.  Per row: max-subtracted exp, inclusive
// prefix sum over the classes in order, first class k with u * Z < S_k (255 if none).  The two
// rows' dependent chains of cross-lane moves run together.  Returns (class of A, class of B), wave-uniform.
__device__ __forceinline__ int2 sample256x2(const float *lgA, const float *lgB, float uA, float uB) {
  const int lane = threadIdx.x & 63, half = lane >> 5, row = lane >> 4;
  const float *lg = (half ? lgB : lgA) + 8 * (lane & 31);
  const float4 la = *(const float4 *)lg, lb = *(const float4 *)(lg + 4);
  float m = fmaxf(fmaxf(fmaxf(la.x, la.y), fmaxf(la.z, la.w)), fmaxf(fmaxf(lb.x, lb.y), fmaxf(lb.z, lb.w)));
  m = fmaxf(m, dpp<0xB1>(m));   // quad_perm [1,0,3,2]
  m = fmaxf(m, dpp<0x4E>(m));   // quad_perm [2,3,0,1]
  m = fmaxf(m, dpp<0x141>(m));  // row_half_mirror
  m = fmaxf(m, dpp<0x140>(m));  // row_mirror
  // rows of 16 lanes 0, 1 hold row A, rows 2, 3 row B
  const float mA = fmaxf(lane_f(m, 0), lane_f(m, 16)), mB = fmaxf(lane_f(m, 32), lane_f(m, 48));
  m = half ? mB : mA;
  float c[8];
  c[0] = __expf(la.x - m);
  c[1] = c[0] + __expf(la.y - m);
  c[2] = c[1] + __expf(la.z - m);
  c[3] = c[2] + __expf(la.w - m);
  c[4] = c[3] + __expf(lb.x - m);
  c[5] = c[4] + __expf(lb.y - m);
  c[6] = c[5] + __expf(lb.z - m);
  c[7] = c[6] + __expf(lb.w - m);
  // inclusive scan of the lane sums inside each row of 16, then row 1 (3) adds row 0's (2's) total
  float incl = c[7];
  incl += dpp<0x111>(incl);  // row_shr:1
  incl += dpp<0x112>(incl);  // row_shr:2
  incl += dpp<0x114>(incl);  // row_shr:4
  incl += dpp<0x118>(incl);  // row_shr:8
  const float t0 = lane_f(incl, 15), t1 = lane_f(incl, 31), t2 = lane_f(incl, 47), t3 = lane_f(incl, 63);
  incl += (row == 1 ? t0 : 0.f) + (row == 3 ? t2 : 0.f);
  const float excl = incl - c[7];
  const float target = half ? uB * (t2 + t3) : uA * (t0 + t1);
  int first = 8;
#pragma unroll
  for (int k = 7; k >= 0; --k)
    if (target < excl + c[k]) first = k;
  const unsigned long long hit = __ballot(first < 8);
  const unsigned int hA = (unsigned int)hit, hB = (unsigned int)(hit >> 32);
  int kA = 255, kB = 255;
  if (hA != 0u) {
    const int src = __ffs((int)hA) - 1;
    kA = 8 * src + __builtin_amdgcn_readlane(first, src);
  }
  if (hB != 0u) {
    const int src = __ffs((int)hB) - 1;
    kB = 8 * src + __builtin_amdgcn_readlane(first, 32 + src);
  }
  return make_int2(kA, kB);
}

}  // namespace mfd
}  // namespace fwg
