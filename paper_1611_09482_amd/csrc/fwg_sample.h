// Inverse-CDF sampling shared by the general step kernels, the naive generator, and (the DPP form)
// the chain and wide step kernels.
#pragma once

#include <hip/hip_runtime.h>

namespace fwg {

// Inverse-CDF sampling of one row of 256 logits by one wavefront: 4 classes per
// lane, wave max, exp, per-lane running sums, wave-wide exclusive scan, and the
// first class whose running sum exceeds u * Z (else the last class).
__device__ __forceinline__ int sample_row_256(const float *lg, float u) {
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

// The same rule for a row held 4 classes per lane (lane l: classes 4l..4l+3) with DPP row moves and
// lane reads instead of LDS shuffles: max, exp, inclusive prefix sums in class order (in-lane, then
// shifts inside rows of 16 lanes, then the row totals), the first class k with u Z < S_k, else the
// last class.  Wave-uniform result.
template <int CTRL>
__device__ __forceinline__ float dpp_move(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}
__device__ __forceinline__ float read_lane(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}
__device__ __forceinline__ int sample_row4(float4 lg, float u) {
  const int lane = threadIdx.x & 63;
  float m = fmaxf(fmaxf(lg.x, lg.y), fmaxf(lg.z, lg.w));
  m = fmaxf(m, dpp_move<0xB1>(m));   // quad_perm [1,0,3,2]
  m = fmaxf(m, dpp_move<0x4E>(m));   // quad_perm [2,3,0,1]
  m = fmaxf(m, dpp_move<0x141>(m));  // row_half_mirror
  m = fmaxf(m, dpp_move<0x140>(m));  // row_mirror
  m = fmaxf(fmaxf(read_lane(m, 0), read_lane(m, 16)), fmaxf(read_lane(m, 32), read_lane(m, 48)));
  float c[4];
  c[0] = __expf(lg.x - m);
  c[1] = c[0] + __expf(lg.y - m);
  c[2] = c[1] + __expf(lg.z - m);
  c[3] = c[2] + __expf(lg.w - m);
  float incl = c[3];
  incl += dpp_move<0x111>(incl);  // row_shr:1
  incl += dpp_move<0x112>(incl);  // row_shr:2
  incl += dpp_move<0x114>(incl);  // row_shr:4
  incl += dpp_move<0x118>(incl);  // row_shr:8
  const float t0 = read_lane(incl, 15), t1 = read_lane(incl, 31), t2 = read_lane(incl, 47), t3 = read_lane(incl, 63);
  const int row = lane >> 4;
  incl += (row >= 1 ? t0 : 0.f) + (row >= 2 ? t1 : 0.f) + (row >= 3 ? t2 : 0.f);
  const float excl = incl - c[3];
  const float target = u * (((t0 + t1) + t2) + t3);
  int first = 4;
#pragma unroll
  for (int k = 3; k >= 0; --k)
    if (target < excl + c[k]) first = k;
  const unsigned long long hit = __ballot(first < 4);
  if (hit == 0ull) return 255;
  const int src = __ffsll((long long)hit) - 1;
  return 4 * src + __builtin_amdgcn_readlane(first, src);
}

}  // namespace fwg
