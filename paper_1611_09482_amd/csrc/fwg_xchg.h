// Hand-offs between the cooperating blocks of one launch (the split, wide and gated chain pair
// step-kernel families): 8-byte words of (32-bit payload, 32-bit tag), loaded with relaxed
// device-scope atomics.  A word is fresh once its tag equals the step's tag (no tag is used twice
// between two zero fills of the exchange region), so no fence or flag has to order the payload.
// Every wait is bounded: a wait that runs out writes the launch's abort mark into the abort word,
// which ends every other wait of that launch, and sets a sticky word the host reports.  Not part of
// the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fwg {
namespace xg {

typedef unsigned long long u64;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kSpinMax = 1 << 21;  // polls of one wait before the launch is aborted

// `local`: every reader shares this block's XCD (and L2): a workgroup-scope store completes in that
// L2; otherwise a device-scope store writes through to memory.
__device__ __forceinline__ void put_word(u64 *p, uint32_t payload, uint32_t tag, bool local) {
  const u64 v = ((u64)tag << 32) | payload;
  if (local) __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  else __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Two consecutive words (p 16-byte aligned).  Within one XCD a single 16-byte store carries both:
// it lands in one L2 line, so each 8-byte word (tag with its payload) becomes visible whole.
__device__ __forceinline__ void put_words2(u64 *p, uint32_t pa, uint32_t pb, uint32_t tag, bool local) {
  if (local) {
    *(u32x4 *)p = u32x4{pa, tag, pb, tag};
  } else {
    put_word(p, pa, tag, false);
    put_word(p + 1, pb, tag, false);
  }
}
__device__ __forceinline__ uint32_t xcd_id() {
  return __builtin_amdgcn_s_getreg((3 << 11) | (0 << 6) | 20) & 15;  // HW_REG_XCC_ID, bits 3:0
}
__device__ __forceinline__ u64 get_word(const u64 *p) {
  return __hip_atomic_load((u64 *)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t get_flag(const uint32_t *p) {
  return __hip_atomic_load((uint32_t *)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// A wait ran out: end every other wait of the launch, and leave a sticky mark for the host.  `mark`
// identifies the launch (families that zero the region before every launch use 1).
__device__ __forceinline__ void raise_abort(uint32_t *abort_word, uint32_t *sticky, uint32_t mark = 1u) {
  __hip_atomic_store(abort_word, mark, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(sticky, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Load the N tagged words p[e STRIDE] until every tag equals `tag` (or the abort word holds this
// launch's `mark`).
// Per lane.  Every wait of a tile uses STRIDE = the number of lanes polling it, so that each load
// instruction reads consecutive words: a poll whose lanes each take a run of consecutive words
// touches a cache line per lane and instruction, and those requests (not the L2's latency) made
// the tile gathers 2-3x slower.
template <int N, int STRIDE = 1>
__device__ __forceinline__ void wait_words(const u64 *p, uint32_t tag, uint32_t (&out)[N], uint32_t *abort_word,
                                           uint32_t *sticky, uint32_t mark = 1u) {
  u64 v[N];
  for (int it = 0;; ++it) {
#pragma unroll
    for (int e = 0; e < N; ++e) v[e] = get_word(p + e * STRIDE);
    bool ok = true;
#pragma unroll
    for (int e = 0; e < N; ++e) ok = ok && (uint32_t)(v[e] >> 32) == tag;
    if (ok) break;
    // the abort word every 16 polls: a stale poll then costs one round trip, not two
    if ((it & 15) == 15) {
      if (get_flag(abort_word) == mark) break;
      if (it >= kSpinMax) {
        raise_abort(abort_word, sticky, mark);
        break;
      }
    }
  }
#pragma unroll
  for (int e = 0; e < N; ++e) out[e] = (uint32_t)v[e];
}

}  // namespace xg
}  // namespace fwg
