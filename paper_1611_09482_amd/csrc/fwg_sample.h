// Inverse-CDF sampling shared by the general step kernels and the naive generator.
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

}  // namespace fwg
