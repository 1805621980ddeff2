// Time-parallel evaluation of the dilated stack over a whole input sequence (gfx950).
//
// With every input known in advance (teacher forcing, online prediction over an
// observed stretch, priming the queues from a prefix), the stack need not run one
// step at a time: each layer is a width-2 dilated causal convolution over the
// whole sequence, the training-time view of the network (paper Section 1), and
// its products become dense GEMMs with one row per (stream, time) pair.
//
// A call is cut into chunks of Tc steps.  Rows of a chunk are stream-major,
// m = b * Tc + j for time t0 + j.  Layer l reads x^{l-1} at t and at t - d_l; the
// second comes from the chunk's own rows when t - d_l lies in the chunk, and from
// the layer's convolution queue otherwise (the queue holds exactly the states
// x^{l-1}_{t0-d_l} ... x^{l-1}_{t0-1}, slot = time mod d_l, Section 2.1).  After the
// layer, the chunk's newest d_l states replace the queue contents, so the queues
// leave the call in the state the step-by-step pop/push loop (Section 2.2) would
// have left them, and a later generation call continues from there.
//
// Kernels:
//   par_gemm_kernel   C[m][n] = A[m][:] . W[n][:] with a row-gathering prologue
//                     (plain rows, or the two taps of the dilated convolution)
//                     and an epilogue per layer kind (relu, relu + residual,
//                     gate, residual add, logits).  64 x 64 or 128 x 128 tiles,
//                     4 waves, operands staged through LDS in 128-byte k-tiles,
//                     MFMA 16x16x32 bf16 or 16x16x4 f32 with fp32 accumulation.
//   par_embed_kernel  x^0 rows: the 1x1 convolution of the one-hot input (a row
//                     gather), from the forced sequence or the pending input.
//   par_ring_kernel   the queue refresh after each layer.
//
// The same GEMM kernel also evaluates the naive generator's tree (paper Fig. 1): per
// sample, every distinct (layer, time) node the output depends on, from the last
// receptive-field inputs, with nothing cached between samples (rows gathered through
// per-layer node tables; par_sample_kernel draws the sample and extends the input history).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fwg_bf16.h"
#include "fwg_internal.h"
#include "fwg_par.h"
#include "fwg_sample.h"

namespace fwg {
namespace par {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int NT = 256;
constexpr int KT_BYTES = 128;            // bytes of one row inside a k-tile
constexpr int ROWB = KT_BYTES + 16;      // LDS row stride (padding spreads the rows over banks)

// Operand types: float (f32 models) or uint16_t (bf16 bit patterns).
template <typename OT> struct Op;
template <> struct Op<float> {
  static constexpr int KT = KT_BYTES / 4;  // k per tile
  __device__ static __forceinline__ float get(const void *p, long long i) { return ((const float *)p)[i]; }
  __device__ static __forceinline__ void put(void *p, long long i, float v) { ((float *)p)[i] = v; }
  __device__ static __forceinline__ float opnd(float v) { return v; }
  // one 16-byte chunk of A and of B per lane and half-tile: 4 MFMAs of k = 4, element j of lane
  // group g standing for k = 4g + j on both sides
  __device__ static __forceinline__ f32x4 mma(const uint4 &a, const uint4 &b, f32x4 c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
    return c;
  }
};
template <> struct Op<uint16_t> {
  static constexpr int KT = KT_BYTES / 2;
  __device__ static __forceinline__ float get(const void *p, long long i) {
    return __uint_as_float(((uint32_t)((const uint16_t *)p)[i]) << 16);
  }
  __device__ static __forceinline__ void put(void *p, long long i, float v) { ((uint16_t *)p)[i] = bf16_bits(v); }
  __device__ static __forceinline__ float opnd(float v) { return round_bf16(v); }
  // lane group g holds k = 8g .. 8g + 7 of both operands
  __device__ static __forceinline__ f32x4 mma(const uint4 &a, const uint4 &b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                  0, 0, 0);
  }
};

__device__ __forceinline__ float sigmoid(float g) { return 1.f / (1.f + __expf(-g)); }

// Row sources of the A operand.
constexpr int A_PLAIN = PAR_A_PLAIN, A_CONV = PAR_A_CONV, A_TREE = PAR_A_TREE;
// Epilogues:
//   E_RELU      out = opnd(relu(acc + b))
//   E_RELU_RES  x = x_in + relu(acc + b): fp32 x and its operand copy
//   E_RES_ADD   x = x_in + acc + b:       fp32 x and its operand copy
//   E_GATE      z = tanh(.) * sigmoid(.) over interleaved column pairs -> operand z
//   E_LOGITS    logits[b][s0 + j][n] = acc + b
constexpr int E_RELU = PAR_E_RELU, E_RELU_RES = PAR_E_RELU_RES, E_RES_ADD = PAR_E_RES_ADD, E_GATE = PAR_E_GATE,
              E_LOGITS = PAR_E_LOGITS;

template <typename OT, int AM>
__device__ __forceinline__ uint4 load_a(const ParGemm &g, int m, int k) {
  if (m >= g.M) return make_uint4(0, 0, 0, 0);
  if (AM == A_PLAIN) return *(const uint4 *)((const OT *)g.A + (long long)m * g.lda + k);
  // tap k / C of the width-w dilated product reads the state (w - 1 - tap) d steps back
  const int tap = k / g.C, kc = k - tap * g.C;
  const int shift = (g.w - 1 - tap) * g.dil;
  const int b = m / g.Tcur, j = m - b * g.Tcur;
  if (AM == A_TREE) {
    if (g.tnow + g.toff[j] - shift < 0) return make_uint4(0, 0, 0, 0);  // zero padding before time 0
    const long long row = (long long)b * g.nprev + g.tsrc[tap * g.Tcur + j];
    return *(const uint4 *)((const OT *)g.A + row * g.C + kc);
  }
  // dilated convolution over the chunk: the row `shift` steps back, or, before the chunk, the queue
  // slot of that time (depth = (w - 1) d slots, slot = time mod depth)
  const OT *src;
  if (j >= shift) {
    src = (const OT *)g.A + (long long)(m - shift) * g.C + kc;
  } else {
    const long long tau = g.t0 + j - shift;  // >= -depth: before time 0 the slot holds zeros
    const long long slot = tau >= 0 ? tau % g.depth : tau + g.depth;
    src = (const OT *)g.ring + (slot * g.brows + b) * (long long)g.C + kc;
  }
  return *(const uint4 *)src;
}

template <typename OT>
__device__ __forceinline__ uint4 load_w(const ParGemm &g, int n, int k) {
  if (n >= g.N) return make_uint4(0, 0, 0, 0);
  return *(const uint4 *)((const OT *)g.W + (long long)n * g.K + k);
}

// Tile (64 TM) x (64 TM): 4 waves in 2 x 2, each (32 TM) x (32 TM) = (2 TM) x (2 TM) MFMA tiles.
// TM = 2 for outputs at least 128 wide (more MFMAs per staged byte), else 1.
template <typename OT, int AM, int EM, int TM>
__global__ void __launch_bounds__(NT) par_gemm_kernel(ParGemm g) {
  constexpr int TB = 64 * TM, TW = 32 * TM, MT = 2 * TM;
  __shared__ __attribute__((aligned(16))) unsigned char lds_a[TB * ROWB];
  __shared__ __attribute__((aligned(16))) unsigned char lds_b[TB * ROWB];
  constexpr int KT = Op<OT>::KT;
  constexpr int EPC = 16 / sizeof(OT);  // elements per 16-byte chunk
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = w & 1, wn = w >> 1;
  const int m0 = blockIdx.x * TB, n0 = blockIdx.y * TB;
  // staging: thread -> (row sr + 32 i, 16-byte chunk sq)
  const int sr = tid >> 3, sq = tid & 7;

  f32x4 acc[MT][MT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < MT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = g.K / KT;
  uint4 ra[MT], rb[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    ra[i] = load_a<OT, AM>(g, m0 + sr + 32 * i, sq * EPC);
    rb[i] = load_w<OT>(g, n0 + sr + 32 * i, sq * EPC);
  }
  const int lr = lane & 15, lg = lane >> 4;
  for (int kt = 0; kt < nk; ++kt) {
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      *(uint4 *)(lds_a + (sr + 32 * i) * ROWB + sq * 16) = ra[i];
      *(uint4 *)(lds_b + (sr + 32 * i) * ROWB + sq * 16) = rb[i];
    }
    __syncthreads();
    if (kt + 1 < nk) {
      const int k = (kt + 1) * KT + sq * EPC;
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        ra[i] = load_a<OT, AM>(g, m0 + sr + 32 * i, k);
        rb[i] = load_w<OT>(g, n0 + sr + 32 * i, k);
      }
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      uint4 av[MT], bv[MT];
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        av[i] = *(const uint4 *)(lds_a + (TW * wm + 16 * i + lr) * ROWB + kk * 64 + lg * 16);
        bv[i] = *(const uint4 *)(lds_b + (TW * wn + 16 * i + lr) * ROWB + kk * 64 + lg * 16);
      }
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < MT; ++j) acc[i][j] = Op<OT>::mma(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }

  // epilogue: acc[i][j][e] is row TW wm + 16 i + 4 lg + e, column TW wn + 16 j + lr of the tile
  if (EM == E_GATE) {
    // columns come in groups of 32: 16 tanh columns, then the 16 sigmoid columns of the same
    // channels; the wave's TM groups are its MFMA column tiles (2 q, 2 q + 1)
#pragma unroll
    for (int q = 0; q < TM; ++q) {
      const int grp = (n0 + TW * wn) / 32 + q;
      if (32 * grp >= g.N) continue;
      const int ch = 16 * grp + lr;
      const float bt = g.bias[32 * grp + lr], bs = g.bias[32 * grp + 16 + lr];
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int m = m0 + TW * wm + 16 * i + 4 * lg + e;
          if (m < g.M) {
            const float z = tanhf(acc[i][2 * q][e] + bt) * sigmoid(acc[i][2 * q + 1][e] + bs);
            Op<OT>::put(g.oout, (long long)m * g.ldo + g.zoff + ch, z);
            if (AM == A_TREE && g.ztop) {
              const int b = m / g.Tcur;
              if (m - b * g.Tcur == g.Tcur - 1) Op<OT>::put(g.ztop, (long long)b * g.ldo + g.zoff + ch, z);
            }
          }
        }
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < MT; ++j) {
    const int n = n0 + TW * wn + 16 * j + lr;
    if (n >= g.N) continue;
    const float bn = g.bias[n];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int m = m0 + TW * wm + 16 * i + 4 * lg + e;
        if (m >= g.M) continue;
        const float v = acc[i][j][e] + bn;
        if (EM == E_RELU) {
          Op<OT>::put(g.oout, (long long)m * g.ldo + n, fmaxf(v, 0.f));
        } else if (EM == E_RELU_RES || EM == E_RES_ADD) {
          const long long at = (long long)m * g.ldo + n;
          long long xr = at;
          if (g.tsrc1) {  // naive tree: x_in is the same-time node of the level below
            const int b = m / g.Tcur;
            xr = ((long long)b * g.nprev + g.tsrc1[m - b * g.Tcur]) * g.ldo + n;
          }
          const float x = g.xres[xr] + (EM == E_RELU_RES ? fmaxf(v, 0.f) : v);
          g.xout[at] = x;
          if (g.oout) Op<OT>::put(g.oout, at, x);
        } else {  // E_LOGITS
          const int b = m / g.Tcur, jj = m - b * g.Tcur;
          g.logits[((long long)b * g.n_steps + g.s0 + jj) * g.N + n] = v;
        }
      }
  }
}

template <typename OT, int AM, int TM>
static hipError_t launch_em_t(const ParGemm &g, int em, dim3 grid, hipStream_t s) {
  switch (em) {
    case E_RELU: hipLaunchKernelGGL((par_gemm_kernel<OT, AM, E_RELU, TM>), grid, dim3(NT), 0, s, g); break;
    case E_RELU_RES: hipLaunchKernelGGL((par_gemm_kernel<OT, AM, E_RELU_RES, TM>), grid, dim3(NT), 0, s, g); break;
    case E_RES_ADD: hipLaunchKernelGGL((par_gemm_kernel<OT, AM, E_RES_ADD, TM>), grid, dim3(NT), 0, s, g); break;
    case E_GATE: hipLaunchKernelGGL((par_gemm_kernel<OT, AM, E_GATE, TM>), grid, dim3(NT), 0, s, g); break;
    case E_LOGITS: hipLaunchKernelGGL((par_gemm_kernel<OT, AM, E_LOGITS, TM>), grid, dim3(NT), 0, s, g); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// 128-wide tiles for outputs at least 128 wide over at least 4096 rows, else 64-wide tiles
template <typename OT, int AM>
static hipError_t launch_em(const ParGemm &g, int em, hipStream_t s) {
  if (g.N >= 128 && g.M >= 4096) {
    const dim3 grid((g.M + 127) / 128, (g.N + 127) / 128);
    return launch_em_t<OT, AM, 2>(g, em, grid, s);
  }
  const dim3 grid((g.M + 63) / 64, (g.N + 63) / 64);
  return launch_em_t<OT, AM, 1>(g, em, grid, s);
}

// ---------------------------------------------------------------------------
// One gated layer over a block of 64 rows: conv (all 2R outputs, interleaved tanh / sigmoid
// groups), gate, residual 1x1 from LDS, add.  Every global access is a 16-byte-per-lane row
// access: the residual input rows are loaded during the conv, and the z, x and operand-x rows are
// assembled in LDS and stored whole.
template <typename OT, int RT>
__global__ void __launch_bounds__(NT) par_gated_layer_kernel(ParGemm g) {
  constexpr int R = 16 * RT, CO = 2 * R;
  constexpr int XROW = R * 4 + 16;  // LDS stride of a float32 x row
  // after the conv, the z rows take the A staging area and the x rows the W staging area (37 KB in
  // all for R = 64: four blocks per CU)
  constexpr int WX_BYTES = CO * ROWB > 64 * XROW ? CO * ROWB : 64 * XROW;
  __shared__ __attribute__((aligned(16))) unsigned char lds_a[64 * ROWB];
  __shared__ __attribute__((aligned(16))) unsigned char lds_b[WX_BYTES];
  __shared__ __attribute__((aligned(16))) unsigned char lds_r[R * ROWB];
  unsigned char *const lds_z = lds_a, *const lds_x = lds_b;
  constexpr int KT = Op<OT>::KT;
  constexpr int EPC = 16 / sizeof(OT);
  constexpr int ZB = R * (int)sizeof(OT);  // bytes of a z row (<= 128)
  constexpr int XC = R * 4 / 16;           // 16-byte chunks of a float32 x row
  constexpr int XPT = 64 * XC / NT;        // x chunks per thread
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int wm = w & 1, wn = w >> 1;
  const int m0 = blockIdx.x * 64;
  const int sr = tid >> 3, sq = tid & 7;
  const int lr = lane & 15, lg = lane >> 4;

  // residual weights [R][R] (one k-tile): rows sr + 32 i
#pragma unroll
  for (int i = 0; i < (R + 31) / 32; ++i) {
    const int n = sr + 32 * i;
    if (n < R) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (sq * 16 < ZB) v = *(const uint4 *)((const OT *)g.W2 + (long long)n * R + sq * EPC);
      *(uint4 *)(lds_r + n * ROWB + sq * 16) = v;
    }
  }
  // the residual input rows, in flight during the conv: chunk c of the tile = row c / XC, piece c % XC
  uint4 xin[XPT];
#pragma unroll
  for (int i = 0; i < XPT; ++i) {
    const int c = tid + NT * i, r = c / XC, q = c % XC, m = m0 + r;
    xin[i] = m < g.M ? *(const uint4 *)(g.xres + (long long)m * g.ldo + 4 * q) : make_uint4(0, 0, 0, 0);
  }

  // the previous layer's queue refresh: its input rows of this block that are among the chunk's
  // last qdepth steps, each to the slot of its time
  if (g.qring) {
    constexpr int RC = ZB / 16;  // 16-byte pieces of an operand row of C = R channels
    for (int c = tid; c < 64 * RC; c += NT) {
      const int r = c / RC, q = c % RC, m = m0 + r;
      if (m >= g.M) break;
      const int b = m / g.Tcur, j = m - b * g.Tcur;
      if (j < g.Tcur - g.qdepth) continue;
      const long long slot = (g.t0 + j) % g.qdepth;
      *(uint4 *)((char *)g.qring + (slot * g.brows + b) * (long long)ZB + 16 * q) =
          *(const uint4 *)((const char *)g.qsrc + (long long)m * ZB + 16 * q);
    }
  }

  // ---- dilated product: 64 rows x CO columns; wave (wm, wn): rows 32 wm.., columns (CO / 2) wn..
  f32x4 acc[2][RT];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < RT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int nk = g.K / KT;
  constexpr int WR = CO / 32;  // W staging rows per thread
  uint4 ra[2], rb[WR];
#pragma unroll
  for (int i = 0; i < 2; ++i) ra[i] = load_a<OT, A_CONV>(g, m0 + sr + 32 * i, sq * EPC);
#pragma unroll
  for (int i = 0; i < WR; ++i) rb[i] = load_w<OT>(g, sr + 32 * i, sq * EPC);
  for (int kt = 0; kt < nk; ++kt) {
#pragma unroll
    for (int i = 0; i < 2; ++i) *(uint4 *)(lds_a + (sr + 32 * i) * ROWB + sq * 16) = ra[i];
#pragma unroll
    for (int i = 0; i < WR; ++i) *(uint4 *)(lds_b + (sr + 32 * i) * ROWB + sq * 16) = rb[i];
    __syncthreads();
    if (kt + 1 < nk) {
      const int k = (kt + 1) * KT + sq * EPC;
#pragma unroll
      for (int i = 0; i < 2; ++i) ra[i] = load_a<OT, A_CONV>(g, m0 + sr + 32 * i, k);
#pragma unroll
      for (int i = 0; i < WR; ++i) rb[i] = load_w<OT>(g, sr + 32 * i, k);
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      uint4 av[2], bv[RT];
#pragma unroll
      for (int i = 0; i < 2; ++i) av[i] = *(const uint4 *)(lds_a + (32 * wm + 16 * i + lr) * ROWB + kk * 64 + lg * 16);
#pragma unroll
      for (int j = 0; j < RT; ++j)
        bv[j] = *(const uint4 *)(lds_b + ((CO / 2) * wn + 16 * j + lr) * ROWB + kk * 64 + lg * 16);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < RT; ++j) acc[i][j] = Op<OT>::mma(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }

  // ---- gate: the wave's column tiles (2 q, 2 q + 1) are the tanh and sigmoid halves of 16 channels;
  // the residual input rows land in the staging area (free after the conv)
#pragma unroll
  for (int q = 0; q < RT / 2; ++q) {
    const int grp = ((CO / 2) * wn) / 32 + q;
    const int ch = 16 * grp + lr;
    const float bt = g.bias[32 * grp + lr], bs = g.bias[32 * grp + 16 + lr];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 32 * wm + 16 * i + 4 * lg + e;
        const float z = tanhf(acc[i][2 * q][e] + bt) * sigmoid(acc[i][2 * q + 1][e] + bs);
        Op<OT>::put(lds_z + r * ROWB, ch, z);
      }
  }
#pragma unroll
  for (int i = 0; i < XPT; ++i) {
    const int c = tid + NT * i, r = c / XC, q = c % XC;
    *(uint4 *)(lds_x + r * XROW + 16 * q) = xin[i];
  }
  // zero the padding of the z rows beyond R (read by the second half-tile when R operands < 128 B)
  if (ZB < KT_BYTES)
    for (int i = tid; i < 64 * ((KT_BYTES - ZB) / 16); i += NT) {
      const int r = i / ((KT_BYTES - ZB) / 16), c = i % ((KT_BYTES - ZB) / 16);
      *(uint4 *)(lds_z + r * ROWB + ZB + c * 16) = make_uint4(0, 0, 0, 0);
    }
  __syncthreads();

  // ---- residual 1x1 from LDS: 64 rows x R; wave (wm, wn): rows 32 wm.., columns (R / 2) wn..
  constexpr int RJ = RT / 2;
  f32x4 res[2][RJ];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < RJ; ++j) res[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    uint4 av[2], bv[RJ];
#pragma unroll
    for (int i = 0; i < 2; ++i) av[i] = *(const uint4 *)(lds_z + (32 * wm + 16 * i + lr) * ROWB + kk * 64 + lg * 16);
#pragma unroll
    for (int j = 0; j < RJ; ++j)
      bv[j] = *(const uint4 *)(lds_r + ((R / 2) * wn + 16 * j + lr) * ROWB + kk * 64 + lg * 16);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < RJ; ++j) res[i][j] = Op<OT>::mma(av[i], bv[j], res[i][j]);
  }
  // x += W_res z + b_res in the LDS rows (each element has one owner lane)
#pragma unroll
  for (int j = 0; j < RJ; ++j) {
    const int n = (R / 2) * wn + 16 * j + lr;
    const float bn = g.bias2[n];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float *px = (float *)(lds_x + (32 * wm + 16 * i + 4 * lg + e) * XROW) + n;
        *px += res[i][j][e] + bn;
      }
  }
  __syncthreads();

  // ---- row stores: z rows (operand), x rows (float32) and their operand copies
  constexpr int ZC = ZB / 16;
  for (int c = tid; c < 64 * ZC; c += NT) {
    const int r = c / ZC, q = c % ZC, m = m0 + r;
    if (m < g.M) *(uint4 *)((OT *)g.zout + (long long)m * g.ldz + g.zoff + q * EPC) = *(const uint4 *)(lds_z + r * ROWB + 16 * q);
  }
#pragma unroll
  for (int i = 0; i < XPT; ++i) {
    const int c = tid + NT * i, r = c / XC, q = c % XC, m = m0 + r;
    if (m >= g.M) continue;
    const float4 v = *(const float4 *)(lds_x + r * XROW + 16 * q);
    *(float4 *)(g.xout + (long long)m * g.ldo + 4 * q) = v;
    if (g.oout) {
      OT *o = (OT *)g.oout + (long long)m * g.ldo + 4 * q;
      Op<OT>::put(o, 0, v.x);
      Op<OT>::put(o, 1, v.y);
      Op<OT>::put(o, 2, v.z);
      Op<OT>::put(o, 3, v.w);
    }
  }
}

// ---------------------------------------------------------------------------
// x^0 rows: E[token] + b, fp32 stream and operand copy.  Tokens: the forced sequence
// (teacher forcing) or, in online prediction, the pending input followed by the
// observed samples.
template <typename OT>
__global__ void par_embed_kernel(ParEmbed e) {
  const long long total = (long long)e.M * e.C;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (long long)gridDim.x * blockDim.x) {
    const int m = (int)(i / e.C), c = (int)(i - (long long)m * e.C);
    const int b = m / e.Tcur, j = m - b * e.Tcur;
    const long long st = e.s0 + j;  // step index inside the call
    int tok;
    if (e.hist) {
      const long long tau = e.tnow + e.toff[j];
      tok = tau >= 0 ? e.hist[(long long)b * (e.hmask + 1) + (tau & e.hmask)] : 0;
    } else if (e.mode == MODE_TEACHER) {
      tok = e.inputs[(long long)b * e.n_steps + st];
    } else {
      tok = st == 0 ? e.last[b] : e.inputs[(long long)b * e.n_steps + st - 1];
    }
    const float v = Op<OT>::get(e.embed, (long long)tok * e.C + c) + e.embed_b[c];
    if (e.xout) e.xout[i] = v;
    Op<OT>::put(e.oout, i, v);
  }
}

// Queue refresh after layer l: slot k takes the newest state of this chunk whose time is
// k mod depth (if the chunk reaches that slot); the operand rows of the layer's input are copied
// in 16-byte pieces.
__global__ void par_ring_kernel(ParRing r) {
  const int pieces = r.row_bytes / 16;
  const long long total = (long long)r.batch * r.depth * pieces;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (long long)gridDim.x * blockDim.x) {
    const int q = (int)(i % pieces);
    const long long bk = i / pieces;
    const int k = (int)(bk % r.depth), b = (int)(bk / r.depth);
    const long long last_t = r.t0 + r.Tcur - 1;
    long long back = (last_t - k) % r.depth;                 // last_t may be below k: keep it non-negative
    if (back < 0) back += r.depth;
    const long long tnew = last_t - back;                    // newest time <= last_t with slot k
    if (tnew < r.t0) continue;                               // the chunk is shorter than d: slot kept
    const long long m = (long long)b * r.Tcur + (tnew - r.t0);
    const uint4 v = *(const uint4 *)((const char *)r.src + m * r.row_bytes + q * 16);
    *(uint4 *)((char *)r.ring + ((long long)k * r.brows + b) * r.row_bytes + q * 16) = v;
  }
}

// One wavefront per stream: inverse-CDF sample of its logits row, stored and appended to the history.
__global__ void par_sample_kernel(const float *logits, const float *uniforms, int32_t *samples, int32_t *hist,
                                  int hmask, long long tnext, int batch, int n_steps, int s) {
  const int b = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (b >= batch) return;
  const int k = sample_row_256(logits + (long long)b * 256, uniforms[(long long)b * n_steps + s]);
  if ((threadIdx.x & 63) == 0) {
    samples[(long long)b * n_steps + s] = k;
    hist[(long long)b * (hmask + 1) + (tnext & hmask)] = k;
  }
}

__global__ void par_set_last_kernel(const int32_t *inputs, int32_t *last, int batch, int n_steps) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < batch) last[b] = inputs[(long long)b * n_steps + n_steps - 1];
}

// ---------------------------------------------------------------------------
// Weight repacks (at create) into plain [N][K] operand rows.
template <typename T>
__global__ void par_repack_kernel(const T *__restrict__ src, T *__restrict__ dst, int mode, int N, int K, int C,
                                  int interleave, long long ldd, long long doff) {
  const long long total = (long long)N * K;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (long long)gridDim.x * blockDim.x) {
    const int n = (int)(i / K), k = (int)(i - (long long)n * K);
    if (mode == PAR_REPACK_CONV) {
      // dst row n holds conv output channel o(n): [tap 0 over C | ... | tap w - 1 over C], K = w C
      int o = n;
      if (interleave) {
        const int grp = n >> 5, wi = n & 31, R = N / 2;
        o = wi < 16 ? 16 * grp + wi : R + 16 * grp + (wi - 16);
      }
      const int w = K / C, tap = k / C, c = k - tap * C;
      dst[i] = src[((long long)o * C + c) * w + tap];
    } else {  // PAR_REPACK_COPY: src [N][K] into dst rows of stride ldd at column offset doff
      dst[(long long)n * ldd + doff + k] = src[i];
    }
  }
}

__global__ void par_bias_kernel(const float *src, float *dst, int N, int interleave, int accumulate) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= N) return;
  int o = n;
  if (interleave) {
    const int grp = n >> 5, wi = n & 31, R = N / 2;
    o = wi < 16 ? 16 * grp + wi : R + 16 * grp + (wi - 16);
  }
  const float v = src ? src[o] : 0.f;
  dst[n] = accumulate ? dst[n] + v : v;
}

}  // namespace par

// ---------------------------------------------------------------------------
static int grid_for(long long total) {
  const long long b = (total + 255) / 256;
  return (int)(b < 8192 ? (b > 0 ? b : 1) : 8192);
}

hipError_t launch_par_gemm(const ParGemm &g, int dtype, int amode, int emode, hipStream_t s) {
  if (g.M <= 0) return hipSuccess;
  if (dtype == 1) {
    if (amode == par::A_CONV) return par::launch_em<uint16_t, par::A_CONV>(g, emode, s);
    if (amode == par::A_TREE) return par::launch_em<uint16_t, par::A_TREE>(g, emode, s);
    return par::launch_em<uint16_t, par::A_PLAIN>(g, emode, s);
  }
  if (amode == par::A_CONV) return par::launch_em<float, par::A_CONV>(g, emode, s);
  if (amode == par::A_TREE) return par::launch_em<float, par::A_TREE>(g, emode, s);
  return par::launch_em<float, par::A_PLAIN>(g, emode, s);
}

bool par_gated_layer_ok(int R, int dtype) {
  const int es = dtype == 1 ? 2 : 4;
  return (R == 32 || R == 64) && R * es <= par::KT_BYTES;
}

hipError_t launch_par_gated_layer(const ParGemm &g, int dtype, hipStream_t s) {
  if (g.M <= 0) return hipSuccess;
  const dim3 grid((g.M + 63) / 64);
  if (dtype == 1) {
    if (g.C == 64) hipLaunchKernelGGL((par::par_gated_layer_kernel<uint16_t, 4>), grid, dim3(par::NT), 0, s, g);
    else hipLaunchKernelGGL((par::par_gated_layer_kernel<uint16_t, 2>), grid, dim3(par::NT), 0, s, g);
  } else {
    hipLaunchKernelGGL((par::par_gated_layer_kernel<float, 2>), grid, dim3(par::NT), 0, s, g);
  }
  return hipGetLastError();
}

hipError_t launch_par_embed(const ParEmbed &e, int dtype, hipStream_t s) {
  const int grid = grid_for((long long)e.M * e.C);
  if (dtype == 1) hipLaunchKernelGGL(par::par_embed_kernel<uint16_t>, dim3(grid), dim3(256), 0, s, e);
  else hipLaunchKernelGGL(par::par_embed_kernel<float>, dim3(grid), dim3(256), 0, s, e);
  return hipGetLastError();
}

hipError_t launch_par_ring(const ParRing &r, hipStream_t s) {
  const int grid = grid_for((long long)r.batch * r.depth * (r.row_bytes / 16));
  hipLaunchKernelGGL(par::par_ring_kernel, dim3(grid), dim3(256), 0, s, r);
  return hipGetLastError();
}

hipError_t launch_par_sample(const float *logits, const float *uniforms, int32_t *samples, int32_t *hist, int hmask,
                             long long tnext, int batch, int n_steps, int s, hipStream_t st) {
  hipLaunchKernelGGL(par::par_sample_kernel, dim3((batch + 3) / 4), dim3(256), 0, st, logits, uniforms, samples, hist,
                     hmask, tnext, batch, n_steps, s);
  return hipGetLastError();
}

hipError_t launch_par_set_last(const int32_t *inputs, int32_t *last, int batch, int n_steps, hipStream_t s) {
  hipLaunchKernelGGL(par::par_set_last_kernel, dim3((batch + 255) / 256), dim3(256), 0, s, inputs, last, batch,
                     n_steps);
  return hipGetLastError();
}

hipError_t launch_par_repack(const void *src, void *dst, int mode, int dtype, int N, int K, int C, int interleave,
                             long long ldd, long long doff, hipStream_t s) {
  const int grid = grid_for((long long)N * K);
  if (dtype == 1)
    hipLaunchKernelGGL(par::par_repack_kernel<uint16_t>, dim3(grid), dim3(256), 0, s, (const uint16_t *)src,
                       (uint16_t *)dst, mode, N, K, C, interleave, ldd, doff);
  else
    hipLaunchKernelGGL(par::par_repack_kernel<float>, dim3(grid), dim3(256), 0, s, (const float *)src, (float *)dst,
                       mode, N, K, C, interleave, ldd, doff);
  return hipGetLastError();
}

hipError_t launch_par_bias(const float *src, float *dst, int N, int interleave, int accumulate, hipStream_t s) {
  hipLaunchKernelGGL(par::par_bias_kernel, dim3((N + 255) / 256), dim3(256), 0, s, src, dst, N, interleave,
                     accumulate);
  return hipGetLastError();
}

}  // namespace fwg
