"""Test helper: a gated bf16 model whose logits have a closed form that depends on where bf16 rounding
happens (the bf16 reading: every operand of a weight product is rounded, sums stay full precision).

Every conv weight is zero, so the gate of layer l sees only its bias: z^l = tanh(b_t) * sigmoid(b_s)
(Section 2.2's layer step with nothing popped or current contributing).  Layers 0 and 1 have
nonzero biases, deeper layers zero ones (z = tanh(0) sigmoid(0) = 0); W_skip of layers 0 and 1 maps
channel c to skip channel c, the first head 1x1 is the identity and the output 1x1 selects hidden
channel q for class q < 64.  So for q < 64

    logit_q = bf16(relu(bf16(z^0_q) + bf16(z^1_q)))      (z rounded as the skip product's operand)

and 0 for the other classes; without the rounding of z it would be bf16(relu(z^0_q + z^1_q)).  The
biases are drawn so that every z^l_q lies at least 1e-4 (relative) from a bf16 rounding boundary
(float32 transcendentals cannot move it across one) and the two forms differ for every q < 64.
"""
import numpy as np

import workloads as W

R = 64


def bf16_round(x):
    """Round float64 values to 8 significant bits, nearest, ties to even."""
    x = np.asarray(x, np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.rint(m * 256.0), e - 8)


def _margin(v):
    # relative distance to the nearest bf16 rounding boundary (a midpoint between neighbours)
    m, _ = np.frexp(np.asarray(v, np.float64))
    f = m * 256.0
    return np.abs(f - np.floor(f) - 0.5) / np.abs(f)


def _z(bt, bs):
    return np.tanh(bt) / (1.0 + np.exp(-bs))


def gate_biases(seed: int = 7):
    """bt, bs [2][R] float32: the tanh-half and sigmoid-half biases of layers 0 and 1."""
    rng = np.random.default_rng(seed)
    bt = np.zeros((2, R), np.float32)
    bs = np.zeros((2, R), np.float32)
    for c in range(R):
        cand_t = rng.uniform(0.2, 2.0, (4096, 2)).astype(np.float32)
        cand_s = rng.uniform(-1.0, 2.0, (4096, 2)).astype(np.float32)
        z = _z(cand_t.astype(np.float64), cand_s.astype(np.float64))
        ok = (z > 0).all(1) & (_margin(z).min(1) > 1e-4) & (_margin(z.sum(1)) > 1e-4)
        ok &= bf16_round(bf16_round(z[:, 0]) + bf16_round(z[:, 1])) != bf16_round(z.sum(1))
        i = int(np.argmax(ok))
        assert ok[i], c
        bt[:, c], bs[:, c] = cand_t[i], cand_s[i]
    return bt, bs


def make_model(n_layers: int, seed: int = 7):
    dil = tuple(2 ** (l % 6) for l in range(n_layers))
    cfg = W.ModelConfig(W.GATED, W.BF16, R, dil, skip_channels=512, head_channels=512)
    w = W.make_weights(cfg, 0)
    bt, bs = gate_biases(seed)
    w.embed[:] = 0
    w.embed_b[:] = 0
    for l in range(n_layers):
        w.conv[l][:] = 0
        w.conv_b[l][:] = 0
        w.res[l][:] = 0
        w.res_b[l][:] = 0
        w.skip[l][:] = 0
        w.skip_b[l][:] = 0
        if l < 2:
            w.conv_b[l][:R] = bt[l]
            w.conv_b[l][R:] = bs[l]
            w.skip[l][np.arange(R), np.arange(R)] = 1.0
    w.head[:] = np.eye(512, dtype=np.float32)
    w.head_b[:] = 0
    w.out[:] = 0
    w.out[np.arange(R), np.arange(R)] = 1.0
    w.out_b[:] = 0
    return cfg, w


def closed_form(seed: int = 7):
    """(logits with z rounded, logits without): [256] float64 each."""
    bt, bs = gate_biases(seed)
    z = _z(bt.astype(np.float64), bs.astype(np.float64))
    want = np.zeros(256)
    alt = np.zeros(256)
    want[:R] = bf16_round(np.maximum(bf16_round(z[0]) + bf16_round(z[1]), 0.0))
    alt[:R] = bf16_round(np.maximum(z[0] + z[1], 0.0))
    return want, alt
