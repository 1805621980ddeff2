"""Test helper: a gated bf16 model whose logits have a closed form that depends on where bf16 rounding
happens (the bf16 reading: every operand of a weight product is rounded to bf16 -- the current
input, the popped states, z, relu(s), the hidden layer -- while accumulators, biases, the residual
stream and the skip sum stay full precision).

Per channel c < 64 (R = 64), with the embedding zero and its bias bE (so x0 = bE at every step),
b() = bf16 rounding:

  layer 0 (current tap = identity into both gate halves, recurrent tap zero):
      z0 = tanh(b(x0) + bt0) * sigmoid(b(x0) + bs0)
  residual 0 (W_res = identity, bias br0):   x1 = x0 + b(z0) + br0       (the stream: not rounded)
  layer 1 (current and recurrent taps = identity into both halves, dilation D1): the popped state
  is x1 from D1 steps back, zero for the first D1 steps (Section 2.2's zero queues):
      z1 = tanh(b(x1) [+ b(x1)] + bt1) * sigmoid(b(x1) [+ b(x1)] + bs1)   ([..] from step D1 on)
  residual 1 (identity, bias br1):           x2 = x1 + b(z1) + br1
  layer 2 (current tap identity):            z2 = tanh(b(x2) + bt2) * sigmoid(b(x2) + bs2)
  deeper layers: zero weights and biases (z = 0, the stream unchanged)
  skip (layers 0-2: identity into channel c), first head 1x1 the identity, output 1x1 selects
  hidden channel q for class q < 64:
      logit_q = b(relu(b(z0) + b(z1) + b(z2)))           (0 for classes >= 64)

The parameters are drawn so that every rounded intermediate lies at least 1e-4 (relative) from a
bf16 rounding boundary (float32 sums and transcendentals cannot move it across one), and so that
moving any one rounding point (z not rounded; the layer inputs not rounded; the stream rounded)
changes the logits of a third of the channels at every step (the final rounding of the logit to 8
bits hides most single moves, so each third is drawn for one of them).
"""
import functools

import numpy as np

import workloads as W

R = 64
D1 = 2  # dilation of layer 1


def bf16_round(x):
    """Round float64 values to 8 significant bits, nearest, ties to even."""
    x = np.asarray(x, np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.rint(m * 256.0), e - 8)


def _margin(v):
    # relative distance to the nearest bf16 rounding boundary (a midpoint between neighbours)
    m, _ = np.frexp(np.asarray(v, np.float64))
    f = m * 256.0
    return np.abs(f - np.floor(f) - 0.5) / np.maximum(np.abs(f), 1e-300)


def _gate(a_t, a_s):
    return np.tanh(a_t) / (1.0 + np.exp(-a_s))


def forms(p, popped, rz=True, rx=True, rstream=False):
    """Logit of one channel for parameter rows p [..., 9] = (bE, bt0, bs0, br0, bt1, bs1, br1, bt2,
    bs2); popped: whether layer 1's recurrent tap sees x1 (steps >= D1) or zeros.  rz / rx / rstream:
    whether z, the layer inputs (current and popped) and the residual stream are rounded.  Returns
    the logit and the rounded intermediates."""
    b = bf16_round
    ident = lambda v: v
    bz, bx, bs_ = (b if rz else ident), (b if rx else ident), (b if rstream else ident)
    bE, bt0, bs0, br0, bt1, bs1, br1, bt2, bs2 = (p[..., i] for i in range(9))
    x0 = bs_(bE)
    z0 = _gate(bx(x0) + bt0, bx(x0) + bs0)
    x1 = bs_(x0 + bz(z0) + br0)
    cur = bx(x1) + (bx(x1) if popped else 0.0)
    z1 = _gate(cur + bt1, cur + bs1)
    x2 = bs_(x1 + bz(z1) + br1)
    z2 = _gate(bx(x2) + bt2, bx(x2) + bs2)
    s = bz(z0) + bz(z1) + bz(z2)
    return b(np.maximum(s, 0.0)), (z0, x1, z1, x2, z2), s


ALTS = (dict(rz=False), dict(rx=False), dict(rstream=True))
ALT_NAMES = ("z not rounded", "inputs not rounded", "stream rounded")


def parameters(seed: int = 7):
    return _parameters(seed).copy()


@functools.lru_cache(maxsize=None)
def _parameters(seed: int):
    """[R][9] float32: (bE, bt0, bs0, br0, bt1, bs1, br1, bt2, bs2) per channel.  Channel c is
    drawn so that moving rounding point 3 c // R (ALTS) changes its logit at every step."""
    rng = np.random.default_rng(seed)
    out = np.zeros((R, 9), np.float32)
    lo = np.array([0.05, 0.2, -1.0, -0.5, 0.2, -1.0, -0.5, 0.2, -1.0])
    hi = np.array([0.6, 1.5, 2.0, 0.5, 1.5, 2.0, 0.5, 1.5, 2.0])
    for c in range(R):
        cand = rng.uniform(lo, hi, (65536, 9)).astype(np.float32).astype(np.float64)
        ok = np.ones(len(cand), bool)
        for popped in (False, True):
            want, inter, s = forms(cand, popped)
            for v in inter:
                ok &= _margin(v) > 1e-4
            ok &= s > 0.05
            ok &= forms(cand, popped, **ALTS[3 * c // R])[0] != want
        i = int(np.argmax(ok))
        assert ok[i], c
        out[c] = cand[i]
    return out


def make_model(n_layers: int, seed: int = 7):
    assert n_layers >= 3
    dil = tuple(D1 if l == 1 else 2 ** (l % 6) for l in range(n_layers))
    cfg = W.ModelConfig(W.GATED, W.BF16, R, dil, skip_channels=512, head_channels=512)
    w = W.make_weights(cfg, 0)
    p = parameters(seed)
    ch = np.arange(R)
    w.embed[:] = 0
    w.embed_b[:] = p[:, 0]
    for l in range(n_layers):
        for a in (w.conv[l], w.conv_b[l], w.res[l], w.res_b[l], w.skip[l], w.skip_b[l]):
            a[:] = 0
    # layer 0: current tap (tap 1) identity into both gate halves
    w.conv[0][ch, ch, 1] = 1.0
    w.conv[0][R + ch, ch, 1] = 1.0
    w.conv_b[0][:R], w.conv_b[0][R:] = p[:, 1], p[:, 2]
    w.res[0][ch, ch] = 1.0
    w.res_b[0][:] = p[:, 3]
    # layer 1: current and recurrent taps identity into both halves
    for tap in (0, 1):
        w.conv[1][ch, ch, tap] = 1.0
        w.conv[1][R + ch, ch, tap] = 1.0
    w.conv_b[1][:R], w.conv_b[1][R:] = p[:, 4], p[:, 5]
    w.res[1][ch, ch] = 1.0
    w.res_b[1][:] = p[:, 6]
    # layer 2: current tap identity into both halves
    w.conv[2][ch, ch, 1] = 1.0
    w.conv[2][R + ch, ch, 1] = 1.0
    w.conv_b[2][:R], w.conv_b[2][R:] = p[:, 7], p[:, 8]
    for l in range(3):
        w.skip[l][ch, ch] = 1.0
    w.head[:] = np.eye(512, dtype=np.float32)
    w.head_b[:] = 0
    w.out[:] = 0
    w.out[ch, ch] = 1.0
    w.out_b[:] = 0
    return cfg, w


def closed_form(T: int, seed: int = 7):
    """Logits [T][256] float64 of every row (the first D1 steps pop zeros for layer 1), and the
    same under each moved rounding point, as a dict name -> [T][256]."""
    p = parameters(seed).astype(np.float64)

    def rows(**kw):
        out = np.zeros((T, 256))
        for t in range(T):
            out[t, :R] = forms(p, t >= D1, **kw)[0]
        return out

    return rows(), {name: rows(**alt) for name, alt in zip(ALT_NAMES, ALTS)}
