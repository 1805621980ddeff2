"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

Each test is chosen so that a plausible slip in the oracle (a dropped term, a
wrong tap, an off-by-one queue, a swapped gate half, a transposed matrix, a
wrong rounding) fails at least one of them.  None of them re-runs the oracle's
own formula: they use closed forms, brute force, an independent library
routine (torch conv1d in float64) and values stored under tests/golden/.
"""
import math
import os

import numpy as np
import pytest
import torch

import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
KINDS = [W.RELU, W.RELU_RESIDUAL, W.GATED]


def _read_pairs(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                rows.append(line.split())
    return rows


def _identity_delay_model(dilations, C=3, Q=16, w_r=1.0, w_e=0.0):
    """ReLU stack with W_r = w_r I, W_e = w_e I, zero biases, embedding e[c][q] = q + 10c (>= 0),
    output layer copying x^L into logits[0:C]."""
    cfg = W.ModelConfig(W.RELU, W.F32, C, tuple(dilations), n_classes=Q)
    w = W.make_weights(cfg, 0)
    w.embed[:] = np.array([[q + 10 * c for q in range(Q)] for c in range(C)], np.float32)
    for l in range(cfg.n_layers):
        w.conv[l][:] = 0
        for c in range(C):
            w.conv[l][c, c, 0] = w_r
            w.conv[l][c, c, 1] = w_e
    w.out[:] = 0
    for c in range(C):
        w.out[c, c] = 1.0
    return cfg, w


# ---------------------------------------------------------------- P5 / Fig. 3
def test_queue_sizes_match_paper_example(oracle_lib):
    """Section 2.1 / Fig. 3: the queue feeding a layer holds as many states as its dilation.
    A single layer of dilation d is a pure delay of d steps iff its queue has depth d."""
    rows = _read_pairs("queue_example.txt")
    pairs = [(int(a), int(b)) for a, b in rows if a != "total"]
    total = [int(b) for a, b in rows if a == "total"][0]
    dil = tuple(d for d, _ in pairs)
    assert W.ModelConfig(W.RELU, W.F32, 4, dil).queue_total == total == sum(s for _, s in pairs)
    # caption: the queue under the l-th hidden layer holds 2^l states
    assert [s for _, s in pairs] == [2 ** l for l in range(len(pairs))]
    x = W.sequences(11, 1, 40, n_classes=16)
    for d, size in pairs:
        cfg, w = _identity_delay_model((d,))
        lg = oracle_lib.Oracle(w).teacher_forced(x)[0]
        for t in range(40):
            want = [w.embed[c, x[0, t - size]] if t - size >= 0 else 0.0 for c in range(3)]
            assert list(lg[t, :3]) == want


# ---------------------------------------------------------------- P3 delay line
@pytest.mark.parametrize("dilations", [(1, 2, 4, 8), (3, 1, 5), (512,), (1, 2, 4, 8, 16, 32, 64, 128, 256, 512)])
def test_delay_line_closed_form(oracle_lib, dilations):
    """W_e = 0, W_r = I, ReLU, zero biases, non-negative embeddings: x^L_t = x^0_{t - sum d}.
    Pins pop order (pop before push), queue depth and wrap-around at every dilation."""
    cfg, w = _identity_delay_model(dilations)
    D = sum(dilations)
    T = D + 40
    x = W.sequences(3, 2, T, n_classes=16)
    lg = oracle_lib.Oracle(w).teacher_forced(x)
    for b in range(2):
        for t in range(T):
            want = [w.embed[c, x[b, t - D]] if t >= D else 0.0 for c in range(3)]
            assert list(lg[b, t, :3]) == want, (b, t)


# ---------------------------------------------------------------- P4 window sums
@pytest.mark.parametrize("w_r,L", [(1.0, 4), (2.0, 4), (1.0, 6)])
def test_window_sum_closed_form(oracle_lib, w_r, L):
    """W_r = w_r I, W_e = I, dilations 1..2^(L-1): the binary tree of Fig. 1 in closed form,
    x^L_t = sum_{j=0}^{2^L-1} w_r^popcount(j) x^0_{t-j} (exact for small integers)."""
    dil = tuple(2 ** i for i in range(L))
    cfg, w = _identity_delay_model(dil, w_r=w_r, w_e=1.0)
    T = 2 ** L + 20
    x = W.sequences(5, 1, T, n_classes=16)
    lg = oracle_lib.Oracle(w).teacher_forced(x)[0]
    for t in range(T):
        for c in range(3):
            want = sum(w_r ** bin(j).count("1") * w.embed[c, x[0, t - j]]
                       for j in range(2 ** L) if t - j >= 0)
            assert lg[t, c] == want


# ---------------------------------------------------------------- P1 brute force
def _tiny(kind, dtype, dil, seed, C=4):
    cfg = W.tiny_model(kind, dtype, channels=C, dilations=dil, skip=6, head=5)
    return cfg, W.make_weights(cfg, seed, bias_scale=0.3)


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("dil", [(1, 2, 4), (1, 2, 4, 8, 1, 2), (2, 2, 3, 1)])
def test_cached_equals_naive_tree(oracle_lib, kind, dtype, dil):
    """Fig. 1 vs Fig. 2: the cached generation model equals the uncached recursive tree."""
    cfg, w = _tiny(kind, dtype, dil, seed=17 + kind)
    o = oracle_lib.Oracle(w)
    T = 48
    x = W.sequences(9, 2, T)
    fast = o.teacher_forced(x)
    for b in range(2):
        for t in range(T):
            naive = o.naive(x[b], t)
            np.testing.assert_allclose(fast[b, t], naive, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- P2 parallel / torch
def _torch_reference(w, inputs):
    """Independent evaluation with torch.nn.functional.conv1d in float64: every layer over the
    whole sequence, dilation d, left zero padding d (tap 0 of a PyTorch [Cout][Cin][2] kernel
    meets x_{t-d}).  bf16 models round weight-product operands with torch's bf16 cast."""
    cfg = w.cfg
    f64 = torch.float64
    q = (lambda t: t.to(torch.bfloat16).to(f64)) if cfg.dtype == W.BF16 else (lambda t: t)
    x = torch.as_tensor(inputs, dtype=torch.long)
    B, T = x.shape
    E = torch.as_tensor(w.embed, dtype=f64)
    h = E[:, x].permute(1, 0, 2) + torch.as_tensor(w.embed_b, dtype=f64)[None, :, None]  # [B][C][T]
    s = None
    for l, d in enumerate(cfg.dilations):
        wt = torch.as_tensor(w.conv[l], dtype=f64)
        pad = (cfg.filter_width - 1) * d  # causal: every tap at or before t
        a = torch.nn.functional.conv1d(torch.nn.functional.pad(q(h), (pad, 0)), wt,
                                       torch.as_tensor(w.conv_b[l], dtype=f64), dilation=d)
        if cfg.kind == W.RELU:
            h = torch.relu(a)
        elif cfg.kind == W.RELU_RESIDUAL:
            h = h + torch.relu(a)
        else:
            R = cfg.channels
            z = q(torch.tanh(a[:, :R]) * torch.sigmoid(a[:, R:]))
            res = torch.nn.functional.conv1d(z, torch.as_tensor(w.res[l], dtype=f64)[:, :, None],
                                             torch.as_tensor(w.res_b[l], dtype=f64))
            sk = torch.nn.functional.conv1d(z, torch.as_tensor(w.skip[l], dtype=f64)[:, :, None],
                                            torch.as_tensor(w.skip_b[l], dtype=f64))
            h = h + res
            s = sk if s is None else s + sk
    if cfg.kind == W.GATED:
        hh = torch.nn.functional.conv1d(q(torch.relu(s)), torch.as_tensor(w.head, dtype=f64)[:, :, None],
                                        torch.as_tensor(w.head_b, dtype=f64))
        top = q(torch.relu(hh))
    else:
        top = q(h)
    lg = torch.nn.functional.conv1d(top, torch.as_tensor(w.out, dtype=f64)[:, :, None],
                                    torch.as_tensor(w.out_b, dtype=f64))
    return lg.permute(0, 2, 1).numpy()


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_cached_equals_parallel_and_torch_conv1d(oracle_lib, kind, dtype):
    """Teacher-forced cached generation equals the full-sequence dilated convolution
    (the training-time parallel evaluation), checked against the oracle's parallel form and
    against torch conv1d."""
    dil = (1, 2, 4, 8, 16, 1, 2, 4, 8, 16)
    cfg, w = _tiny(kind, dtype, dil, seed=40 + kind, C=8)
    o = oracle_lib.Oracle(w)
    x = W.sequences(21, 3, 120)
    fast = o.teacher_forced(x)
    par = o.parallel(x)
    np.testing.assert_allclose(fast, par, rtol=1e-12, atol=1e-12)
    ref = _torch_reference(w, x)
    np.testing.assert_allclose(fast, ref, rtol=1e-10, atol=1e-10)


@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_benchmark_shapes_against_torch(oracle_lib, name):
    """The benchmark model shapes (random nonzero biases), a short sequence: oracle vs torch."""
    wl = W.WORKLOADS[name]
    w = W.make_weights(wl.model, wl.weight_seed, bias_scale=0.1)
    x = W.sequences(1, 1, 24)
    np.testing.assert_allclose(oracle_lib.Oracle(w).teacher_forced(x), _torch_reference(w, x),
                               rtol=1e-9, atol=1e-9)


# ---------------------------------------------------------------- gate split
def test_gate_halves_closed_form(oracle_lib):
    """Zero conv weights: z = tanh(b[0:R]) * sigmoid(b[R:2R]) for every t.  With W_res = I the
    first layer's output is x^0 + z + b_res; the halves are distinguishable (tanh(b_g)sigma(b_f)
    differs), so a swapped split fails."""
    R = 3
    cfg = W.ModelConfig(W.GATED, W.F32, R, (1,), skip_channels=R, head_channels=R, n_classes=16)
    w = W.make_weights(cfg, 1)
    bf = np.array([0.3, -1.1, 2.0], np.float32)
    bg = np.array([-0.7, 0.4, 1.5], np.float32)
    w.conv[0][:] = 0
    w.conv_b[0][:] = np.concatenate([bf, bg])
    w.res[0][:] = np.eye(R, dtype=np.float32)
    w.res_b[0][:] = 0
    w.skip[0][:] = np.eye(R, dtype=np.float32)
    w.skip_b[0][:] = np.array([0.25, 0.5, -3.0], np.float32)
    w.head[:] = np.eye(R, dtype=np.float32)
    w.head_b[:] = 0
    w.out[:] = 0
    w.out[:R, :R] = np.eye(R, dtype=np.float32)
    lg = oracle_lib.Oracle(w).teacher_forced(np.array([[5, 9, 2]]))[0]
    z = np.tanh(bf.astype(np.float64)) / (1 + np.exp(-bg.astype(np.float64)))
    s = z + w.skip_b[0]
    # logits[0:R] = relu(I relu(s)) = relu(s)
    for t in range(3):
        np.testing.assert_allclose(lg[t, :R], np.maximum(s, 0), rtol=1e-13)
    swapped = np.tanh(bg.astype(np.float64)) / (1 + np.exp(-bf.astype(np.float64)))
    assert np.abs(np.maximum(swapped + w.skip_b[0], 0) - lg[0, :R]).max() > 1e-3


# ---------------------------------------------------------------- P6 complexity
@pytest.mark.parametrize("L", [3, 5, 7])
def test_product_counts(oracle_lib, L):
    """Section 3.1: the cached method applies 2L conv-tap products per sample (O(L)); the
    naive tree applies 2(2^L - 1) (O(2^L)) once t is past the receptive field."""
    dil = tuple(2 ** i for i in range(L))
    cfg = W.ModelConfig(W.RELU, W.F32, 2, dil, n_classes=8)
    w = W.make_weights(cfg, 2)
    o = oracle_lib.Oracle(w, count_products=True)
    T = cfg.receptive_field + 3
    x = W.sequences(1, 1, T, n_classes=8)
    o.reset_products()
    o.teacher_forced(x)
    assert o.products == 2 * L * T
    o.reset_products()
    o.naive(x[0], T - 1)
    assert o.products == 2 * (2 ** L - 1)


# ---------------------------------------------------------------- P7 receptive field
@pytest.mark.parametrize("kind", KINDS)
def test_receptive_field(oracle_lib, kind):
    dil = (1, 2, 4, 3, 1)
    cfg, w = _tiny(kind, W.F32, dil, seed=3, C=8)
    rf = cfg.receptive_field
    assert rf == 1 + sum(dil)
    o = oracle_lib.Oracle(w)
    T = rf + 5
    x = W.sequences(4, 1, T)
    t = T - 1
    base = o.teacher_forced(x)[0, t]
    far = x.copy()
    far[0, t - rf] = (far[0, t - rf] + 77) % 256
    assert np.array_equal(o.teacher_forced(far)[0, t], base)
    # the oldest input inside the field reaches the output along a single path of recurrent
    # taps, which a ReLU can switch off for a given input: some perturbation must show through
    changed = False
    for delta in range(1, 256, 15):
        near = x.copy()
        near[0, t - rf + 1] = (near[0, t - rf + 1] + delta) % 256
        changed |= not np.array_equal(o.teacher_forced(near)[0, t], base)
    assert changed


# ---------------------------------------------------------------- P8 sampler
def test_sampler_uniform_logits_is_floor(oracle_lib):
    """All-equal logits: inverse CDF of the uniform distribution over 256 classes is floor(256u)."""
    us = np.concatenate([W.uniforms(0, 1, 2000)[0],
                         np.array([0.0, 0.5, 1 - 2 ** -24, 3 / 256, 3 / 256 - 2 ** -24, 255 / 256], np.float32)])
    lg = np.zeros(256, np.float32)
    for u in us:
        assert oracle_lib.sample(lg, float(u)) == math.floor(256 * float(u))


def test_sampler_dominant_shift_and_bounds(oracle_lib):
    rng = np.random.default_rng(0)
    for k in [0, 17, 255]:
        lg = np.zeros(256, np.float32)
        lg[k] = 200.0
        for u in [0.0, 0.3, 0.999]:
            assert oracle_lib.sample(lg, u) == k
    lg = (rng.integers(-8, 8, 256) / 4.0).astype(np.float32)
    for u in W.uniforms(1, 1, 200)[0]:
        assert oracle_lib.sample(lg, float(u)) == oracle_lib.sample(lg + 6.0, float(u))
    assert oracle_lib.sample(lg, 1.0) == 255
    assert oracle_lib.sample(lg, -0.5) == 0


def test_cdf_closed_form(oracle_lib):
    p = np.arange(1, 257, dtype=np.float64)
    p /= p.sum()
    np.testing.assert_allclose(oracle_lib.cdf(np.log(p) + 3.0), np.cumsum(p), rtol=1e-12)


# ---------------------------------------------------------------- P9 state invariants
def _gen_model():
    cfg = W.tiny_model(W.GATED, W.F32, channels=4, dilations=(1, 2, 4, 8, 1, 2, 4, 8), skip=8, head=8)
    return cfg, W.make_weights(cfg, 8, bias_scale=0.2)


def test_generation_continuation_and_reset(oracle_lib):
    cfg, w = _gen_model()
    o = oracle_lib.Oracle(w)
    u = W.uniforms(5, 3, 90)
    full = o.state(3).generate(u)
    st = o.state(3)
    part = np.concatenate([st.generate(u[:, :31]), st.generate(u[:, 31:])], axis=1)
    assert st.t == 90
    assert np.array_equal(full, part)
    st.reset()
    assert st.t == 0
    assert np.array_equal(st.generate(u), full)


def test_generation_streams_independent(oracle_lib):
    cfg, w = _gen_model()
    o = oracle_lib.Oracle(w)
    u = W.uniforms(6, 4, 70)
    together = o.state(4).generate(u)
    for b in range(4):
        alone = o.state(1).generate(u[b:b + 1])
        assert np.array_equal(alone[0], together[b])


def test_generation_is_teacher_forced_on_own_samples(oracle_lib):
    """Feeding back each prediction (Section 1): generation logits equal the teacher-forced
    logits on [seed_input, samples[:-1]], and each sample is drawn from its own logits."""
    cfg, w = _gen_model()
    o = oracle_lib.Oracle(w)
    u = W.uniforms(7, 2, 60)
    s, lg = o.state(2).generate(u, return_logits=True)
    seq = np.concatenate([np.full((2, 1), cfg.seed_input), s[:, :-1]], axis=1)
    np.testing.assert_array_equal(o.teacher_forced(seq), lg)
    for b in range(2):
        for t in range(60):
            assert s[b, t] == oracle_lib.sample(lg[b, t].astype(np.float32), float(u[b, t]))
            c = oracle_lib.cdf(lg[b, t])
            lo = c[s[b, t] - 1] if s[b, t] > 0 else 0.0
            assert lo - 1e-6 <= u[b, t] < c[s[b, t]] + 1e-6


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_online_prediction_continues_the_history(oracle_lib, dtype):
    """Online prediction (Sections 1 and 4): generate, then feed observed samples, then generate
    again from the same queues.  Every step's logits equal a full-sequence torch conv1d over the
    realised history [seed, generated, observed, generated[:-1]], and the observed samples become
    the inputs that follow them."""
    cfg = W.tiny_model(W.GATED, dtype, channels=4, dilations=(1, 2, 4, 8, 1, 2, 4, 8), skip=8, head=8)
    w = W.make_weights(cfg, 8, bias_scale=0.2)
    o = oracle_lib.Oracle(w)
    B, n1, n2, n3 = 2, 13, 29, 17
    u = W.uniforms(31, B, n1 + n3)
    obs = W.sequences(32, B, n2)
    st = o.state(B)
    g1, lg1 = st.generate(u[:, :n1], return_logits=True)
    lg2 = st.step_forced(obs)
    g3, lg3 = st.generate(u[:, n1:], return_logits=True)
    assert st.t == n1 + n2 + n3
    hist = np.concatenate([np.full((B, 1), cfg.seed_input), g1, obs, g3[:, :-1]], axis=1)
    ref = _torch_reference(w, hist)
    got = np.concatenate([lg1, lg2, lg3], axis=1)
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-10)
    # the tree of Fig. 1 at a few times of the observed stretch
    for t in (n1, n1 + 7, n1 + n2 - 1):
        np.testing.assert_allclose(got[1, t], o.naive(hist[1], t), rtol=1e-12, atol=1e-12)
    # from a reset, online prediction over x is the teacher-forced pass over [seed, x[:-1]]
    st.reset()
    lo = st.step_forced(obs)
    np.testing.assert_allclose(lo, _torch_reference(
        w, np.concatenate([np.full((B, 1), cfg.seed_input), obs[:, :-1]], axis=1)), rtol=1e-10, atol=1e-10)


# ---------------------------------------------------------------- P11 filter width w > 2
@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("fw", [3, 4])
def test_width_cached_equals_parallel_naive_and_torch(oracle_lib, kind, dtype, fw):
    """Section 3.1, general filter width: with queues of (w - 1) d_l states, the cached form equals
    the full-sequence dilated convolution of kernel size w (torch conv1d in float64 and the
    oracle's parallel form) and the uncached tree in which every node has w children."""
    dil = (1, 3, 2, 5, 1)
    cfg = W.tiny_model(kind, dtype, channels=4, dilations=dil, skip=6, head=5, filter_width=fw)
    w = W.make_weights(cfg, 50 + kind + fw, bias_scale=0.3)
    o = oracle_lib.Oracle(w)
    x = W.sequences(22, 2, 70)
    fast = o.teacher_forced(x)
    np.testing.assert_allclose(fast, o.parallel(x), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(fast, _torch_reference(w, x), rtol=1e-10, atol=1e-10)
    for t in (0, 5, 23, 40, 69):
        np.testing.assert_allclose(fast[1, t], o.naive(x[1], t), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("fw,r,L", [(3, 3, 3), (3, 4, 4), (4, 4, 3)])
def test_width_product_counts(oracle_lib, fw, r, L):
    """Section 3.1 with filter width w and dilations r^l (r >= w): the cached method applies w
    tap products per layer and sample (O(wL)); the naive tree has (w^L - 1) / (w - 1) nodes of w
    products each (O(w^L)); the queues hold (w - 1)(r^L - 1)/(r - 1) states (O((w - 1) r^L))."""
    dil = tuple(r ** i for i in range(L))
    cfg = W.ModelConfig(W.RELU, W.F32, 2, dil, n_classes=8, filter_width=fw)
    assert cfg.queue_total == (fw - 1) * (r ** L - 1) // (r - 1)
    w = W.make_weights(cfg, 2)
    o = oracle_lib.Oracle(w, count_products=True)
    T = cfg.receptive_field + 2
    x = W.sequences(1, 1, T, n_classes=8)
    o.reset_products()
    o.teacher_forced(x)
    assert o.products == fw * L * T
    o.reset_products()
    o.naive(x[0], T - 1)
    assert o.products == fw * (fw ** L - 1) // (fw - 1)


@pytest.mark.parametrize("fw,dilations", [(3, (1, 2, 4)), (4, (3, 1, 5)), (3, (64,))])
def test_width_delay_line_closed_form(oracle_lib, fw, dilations):
    """Only the oldest tap carries the identity (the others and W_e zero): every layer is a pure
    delay of (w - 1) d_l, so x^L_t = x^0_{t - (w - 1) sum d}.  Pins the queue depth (w - 1) d_l and
    the tap order for w > 2."""
    C, Q = 3, 16
    cfg = W.ModelConfig(W.RELU, W.F32, C, tuple(dilations), n_classes=Q, filter_width=fw)
    w = W.make_weights(cfg, 0)
    w.embed[:] = np.array([[q + 10 * c for q in range(Q)] for c in range(C)], np.float32)
    for l in range(cfg.n_layers):
        w.conv[l][:] = 0
        w.conv[l][np.arange(C), np.arange(C), 0] = 1.0
    w.out[:] = 0
    w.out[np.arange(C), np.arange(C)] = 1.0
    D = (fw - 1) * sum(dilations)
    T = D + 30
    x = W.sequences(3, 2, T, n_classes=Q)
    lg = oracle_lib.Oracle(w).teacher_forced(x)
    for b in range(2):
        for t in range(T):
            want = [w.embed[c, x[b, t - D]] if t >= D else 0.0 for c in range(C)]
            assert list(lg[b, t, :C]) == want, (b, t)


# ---------------------------------------------------------------- P10 bf16
def test_bf16_rounding_vectors(oracle_lib):
    for a, b in _read_pairs("bf16_rne.txt"):
        assert oracle_lib.bf16_round(float(a)) == float(b), a


def test_bf16_rounding_matches_torch_on_random_doubles(oracle_lib):
    """Library routine as an independent reference (torch rounds float32 values to bf16 RNE;
    inputs are float32 so no double rounding is involved)."""
    x = (np.random.default_rng(1).standard_normal(20000) * 10.0 ** np.random.default_rng(2).integers(-6, 6, 20000))
    x = x.astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = np.array([oracle_lib.bf16_round(float(v)) for v in x])
    np.testing.assert_array_equal(got, ref)


# ---------------------------------------------------------------- bf16 rounding points
def test_bf16_rounding_points_closed_form(oracle_lib):
    """The oracle rounds exactly the operands of the weight products to bf16 (the current input, the
    popped state, z, relu(s), the hidden layer) and keeps the residual stream and every sum at full
    precision: on the closed-form model of tests/rounding_model.py its logits equal the closed form
    in every row (the first rows pop zeros), and moving any one rounding point changes many logits."""
    import rounding_model as RM
    T = 7
    want, alts = RM.closed_form(T)
    for name, alt in alts.items():
        for t in (0, T - 1):  # both kinds of rows: layer 1 pops zeros, then x1
            assert (alt[t, :RM.R] != want[t, :RM.R]).sum() >= 16, name
    for n_layers in (3, 12):
        cfg, w = RM.make_model(n_layers)
        lg = oracle_lib.Oracle(w).teacher_forced(W.sequences(5, 3, T))
        assert np.array_equal(lg, np.broadcast_to(want, lg.shape)), n_layers
