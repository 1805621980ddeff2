// General step-kernel family (fwg_kernels.hip): packed-weight layout, layer table and LDS layout.
#pragma once

#include "fwg_internal.h"

namespace fwg {

// Packed-weight layout of the VALU family: W^T blocked by 16 bytes along K,
// Wp[kb][n][kb_elems], with W^T[k][n] the weight from input k to output n.
inline int valu_kb_elems(int dtype) { return dtype == 1 ? 8 : 4; }

// The layer fields the general step kernel reads in its loop, copied to LDS at launch.
struct ValuLayer {
  const void *block;    // the layer's weight + bias block
  long long ring_off;   // element offset of the layer's queue
  int dil, depth;
  int pad_[2];
};
static_assert(sizeof(ValuLayer) == 32, "eight floats per layer in the LDS table");

// LDS layout (in floats) of the VALU step kernel for rows-per-block `rpw`: two buffers of popped
// states and, when a layer's weights are staged (wfloats > 0), two weight buffers.
struct ValuLds {
  int xf, xo, vo, vo2, ao, zo, so, ho, h2, lg, partA, partB, wb0, wb1, ltab, slots, ins, total_floats;
};
constexpr int kValuPrefPops = 8;   // popped elements per thread and layer held in registers
// Weight staging: a layer's block, at most kValuStagePieces 16-byte pieces per thread (64 KB).
constexpr int kValuStagePieces = 16;
__host__ __device__ inline int valu_part_cols(int N) { return N >= 256 ? N : 256; }
__host__ __device__ inline ValuLds valu_lds_layout(int kind, int C, int S, int H, int Q, int L, int rpw, int w,
                                                   int wfloats) {
  ValuLds o;
  int p = 0;
  auto take = [&](int n) { int at = p; p += (n + 3) & ~3; return at; };
  const int Co = kind == 2 ? 2 * C : C;
  o.xf = take(rpw * C);
  o.xo = take(rpw * C);
  o.vo = take(rpw * (w - 1) * C);  // the w - 1 popped states per stream, oldest first
  o.vo2 = take(rpw * (w - 1) * C);
  o.ao = take(rpw * Co);
  o.zo = take(kind == 2 ? rpw * C : 0);
  o.so = take(kind == 2 ? rpw * S : 0);
  o.ho = take(kind == 2 ? rpw * S : 0);
  o.h2 = take(kind == 2 ? rpw * H : 0);
  o.lg = take(rpw * Q);
  int partN = valu_part_cols(Co);
  if (kind == 2) {
    partN = partN > valu_part_cols(S) ? partN : valu_part_cols(S);
    partN = partN > valu_part_cols(H) ? partN : valu_part_cols(H);
  }
  partN = partN > valu_part_cols(Q) ? partN : valu_part_cols(Q);
  o.partA = take(rpw * partN);
  o.partB = take(kind == 2 ? rpw * valu_part_cols(C) : 0);
  o.wb0 = take(wfloats);
  o.wb1 = take(wfloats);
  o.ltab = take(8 * L);  // per layer: weight block address, queue offset, dilation, depth (ValuLayer)
  o.slots = take(L);   // int
  o.ins = take(rpw);   // int
  o.total_floats = p;
  return o;
}

hipError_t launch_valu_step(const StepArgs &a, int rpw, size_t lds_bytes, hipStream_t s);
hipError_t set_valu_lds_limit(size_t bytes);

}  // namespace fwg
