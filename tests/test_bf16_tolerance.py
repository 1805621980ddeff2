"""Where the bf16 logit bar (2e-2 per row) sits against a correct float32 implementation, on the CPU.

Under the bf16 reading every operand of a weight product is rounded to bf16, while accumulators,
biases, nonlinearities, the residual stream and the skip sum stay at full precision.  A correct
float32 implementation differs from the float64 oracle not only by float32 summation error but by
the operands that error pushes across a bf16 rounding boundary (2^-8 relative), and those flips
compound over the layers.  This test evaluates the benchmark model with float32 arithmetic, BLAS
summation order and exactly the oracle's rounding points (plain numpy, time-parallel form: each
layer over the whole sequence with zero history, Section 2.2) and measures its distance to the
float64 oracle: ~1.4e-2 on the 30-layer stack, the spread the GPU kernels show too (~1.7e-2 at full
size), below the 2e-2 bar; deeper stacks spread further (~2.2e-2 at 48 layers), so the GPU tests scale
the bar with depth beyond 30 layers.  The bar does not tell the rounding points apart: the same float32
evaluation with no bf16 rounding at all lands ~1.2e-2 from the oracle as well (printed, not
asserted); the bf16 rounding function itself is pinned by the golden vectors.
"""
import numpy as np

import workloads as W

TOL_BF16 = 2e-2


def _bf(x):
    return W.bf16_bits_to_f32(W.f32_to_bf16_bits(np.ascontiguousarray(x, np.float32))).reshape(x.shape)


def _float32_teacher_forced(w, inputs, operands_bf16=True):
    cfg = w.cfg
    B, T = inputs.shape
    R = cfg.channels
    rnd = _bf if operands_bf16 else (lambda v: v)
    x = (w.embed[:, inputs].transpose(1, 2, 0) + w.embed_b).astype(np.float32)  # [B][T][R]
    s = np.zeros((B, T, cfg.skip_channels), np.float32)
    for l, d in enumerate(cfg.dilations):
        xo = rnd(x)
        ro = np.zeros_like(xo)
        ro[:, d:] = xo[:, :T - d]  # the state d steps back (zeros before time 0)
        a = ro @ w.conv[l][:, :, 0].T + xo @ w.conv[l][:, :, 1].T + w.conv_b[l]
        z = rnd(np.tanh(a[..., :R]) * (np.float32(1) / (np.float32(1) + np.exp(-a[..., R:]))))
        x = x + z @ w.res[l].T + w.res_b[l]
        s = s + z @ w.skip[l].T + w.skip_b[l]
    rs = rnd(np.maximum(s, 0))
    h = rnd(np.maximum(rs @ w.head.T + w.head_b, 0))
    return h @ w.out.T + w.out_b


def _row_rel_err(a, b):
    return np.abs(a - b).max(-1) / np.maximum(np.abs(b).max(-1), 1e-6)


def test_float32_accumulation_spread_of_the_bf16_reading(oracle_lib):
    wl = W.WORKLOADS["gated_r64_s512_l30_b256_bf16"]
    w = W.make_weights(wl.model, wl.weight_seed)
    x = W.sequences(wl.uniform_seed, 2, 1000)
    o = oracle_lib.Oracle(w).teacher_forced(x)
    e = _row_rel_err(_float32_teacher_forced(w, x), o)
    print(f"float32 with the oracle's bf16 rounding points vs the float64 oracle: max {e.max():.3e}, "
          f"p99.9 {np.quantile(e, 0.999):.3e}, median {np.median(e):.3e} over {e.size} rows")
    # a correct float32 implementation of the reading fits the bar, with a visible spread
    assert 3e-3 < e.max() < TOL_BF16
    e_plain = _row_rel_err(_float32_teacher_forced(w, x, operands_bf16=False), o)
    print(f"float32 with no bf16 rounding at all vs the float64 oracle: max {e_plain.max():.3e}")


def test_float32_spread_grows_with_depth(oracle_lib):
    """The same float32 evaluation on the 48-layer split-kernel test stack (dilations 1..32 eight
    times, the GPU tests' weights and inputs): past the benchmark's 30 layers the spread of a correct
    float32 implementation exceeds 2e-2, and stays within the depth-scaled bar the GPU tests use
    (2e-2 x L / 30)."""
    cfg = W.ModelConfig(W.GATED, W.BF16, 64, (1, 2, 4, 8, 16, 32) * 8, 512, 512)
    w = W.make_weights(cfg, 100, bias_scale=0.1)
    x = W.sequences(3, 11, cfg.queue_total + 60)
    o = oracle_lib.Oracle(w).teacher_forced(x)
    e = _row_rel_err(_float32_teacher_forced(w, x), o)
    print(f"48 layers: float32 with the oracle's bf16 rounding points vs the float64 oracle: max "
          f"{e.max():.3e}, p99.9 {np.quantile(e, 0.999):.3e}")
    assert TOL_BF16 < e.max() < TOL_BF16 * cfg.n_layers / 30
