"""The allocation-free generation entry point (fwg_generate_noalloc) against fwg_generate, through
the C ABI: the kernel families whose blocks exchange words (split, wide, gated chain pair), with those
words in the library's static device array, must draw exactly the samples the workspace-backed launch
draws (integer outputs: bit-exact), on two
calls in a row, the second with a smaller batch after a reset (fewer groups, so a smaller part of
the array), and with a continuation across calls."""
import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_1611_09482_amd import binding  # noqa: E402


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _pair(cfg, max_batch):
    w = W.make_weights(cfg, 31, bias_scale=0.1)
    a = binding.from_model(cfg, w, max_batch=max_batch)
    b = binding.from_model(cfg, w, max_batch=max_batch)
    return a, b


def test_noalloc_matches_generate_split():
    cfg = W.ModelConfig(W.GATED, W.BF16, 64, (1, 2, 4, 8, 16, 32) * 2, 512, 512)
    ref, na = _pair(cfg, 37)
    assert ref.regime == na.regime == "mfma_split_bf16_r64_s512"
    # call 1: 37 streams (three groups, the last one ragged), 150 steps
    u = W.uniforms(41, 37, 150)
    want = ref.generate(_dev(u)).cpu().numpy()
    out = torch.empty((37, 150), dtype=torch.int32, device="cuda")
    got = na.generate_noalloc(_dev(u), out).cpu().numpy()
    print(f"noalloc call 1: 37 x 150, equal {np.array_equal(got, want)}", flush=True)
    assert np.array_equal(got, want)
    # call 2: after a reset, 5 streams (one group), 90 steps, split over two calls
    ref.reset()
    na.reset()
    u2 = W.uniforms(42, 5, 90)
    want2 = ref.generate(_dev(u2)).cpu().numpy()
    o1 = torch.empty((5, 40), dtype=torch.int32, device="cuda")
    o2 = torch.empty((5, 50), dtype=torch.int32, device="cuda")
    g1 = na.generate_noalloc(_dev(u2[:, :40]), o1).cpu().numpy()
    g2 = na.generate_noalloc(_dev(u2[:, 40:]), o2).cpu().numpy()
    got2 = np.concatenate([g1, g2], axis=1)
    print(f"noalloc call 2: 5 x 90 in two calls, equal {np.array_equal(got2, want2)}", flush=True)
    assert np.array_equal(got2, want2)
    # the workspace-backed entry point continues from the state the noalloc calls left
    u3 = W.uniforms(43, 5, 30)
    a = ref.generate(_dev(u3)).cpu().numpy()
    b = na.generate(_dev(u3)).cpu().numpy()
    assert np.array_equal(a, b)


def test_noalloc_matches_generate_wide():
    """The wide kernels (512-channel float32 ReLU + residual stack, groups of 32 blocks exchanging the
    layer outputs as words): exchange words in the static array, three stream groups with a ragged last
    one, then one group after a reset."""
    cfg = W.ModelConfig(W.RELU_RESIDUAL, W.F32, 512, (1, 2, 4, 8, 16, 1, 2))
    ref, na = _pair(cfg, 11)
    assert ref.regime == na.regime == "wide_f32_c512"
    u = W.uniforms(45, 11, 70)
    want = ref.generate(_dev(u)).cpu().numpy()
    out = torch.empty((11, 70), dtype=torch.int32, device="cuda")
    got = na.generate_noalloc(_dev(u), out).cpu().numpy()
    print(f"noalloc wide call 1: 11 x 70, equal {np.array_equal(got, want)}", flush=True)
    assert np.array_equal(got, want)
    ref.reset()
    na.reset()
    u2 = W.uniforms(46, 3, 40)
    want2 = ref.generate(_dev(u2)).cpu().numpy()
    out2 = torch.empty((3, 40), dtype=torch.int32, device="cuda")
    got2 = na.generate_noalloc(_dev(u2), out2).cpu().numpy()
    print(f"noalloc wide call 2: 3 x 40, equal {np.array_equal(got2, want2)}", flush=True)
    assert np.array_equal(got2, want2)


def test_noalloc_matches_generate_chain_pair():
    """The gated chain kernels' pair variant (two blocks per stream exchanging z rows, skip halves,
    hidden halves and logits as words): exchange words in the static array, 9 streams (pairs on
    every XCD slot and one more), then 2 streams after a reset in two calls."""
    cfg = W.ModelConfig(W.GATED, W.F32, 32, (1, 2, 4, 8, 16), 256, 256)
    ref, na = _pair(cfg, 9)
    assert ref.regime == na.regime == "chain_pair_f32_r32"
    u = W.uniforms(47, 9, 80)
    want = ref.generate(_dev(u)).cpu().numpy()
    out = torch.empty((9, 80), dtype=torch.int32, device="cuda")
    got = na.generate_noalloc(_dev(u), out).cpu().numpy()
    print(f"noalloc pair call 1: 9 x 80, equal {np.array_equal(got, want)}", flush=True)
    assert np.array_equal(got, want)
    ref.reset()
    na.reset()
    u2 = W.uniforms(48, 2, 60)
    want2 = ref.generate(_dev(u2)).cpu().numpy()
    o1 = torch.empty((2, 25), dtype=torch.int32, device="cuda")
    o2 = torch.empty((2, 35), dtype=torch.int32, device="cuda")
    g1 = na.generate_noalloc(_dev(u2[:, :25]), o1).cpu().numpy()
    g2 = na.generate_noalloc(_dev(u2[:, 25:]), o2).cpu().numpy()
    got2 = np.concatenate([g1, g2], axis=1)
    print(f"noalloc pair call 2: 2 x 60 in two calls, equal {np.array_equal(got2, want2)}", flush=True)
    assert np.array_equal(got2, want2)
    na.device_status()


def test_noalloc_other_family_and_errors():
    """Kernel families without per-launch scratch run exactly as fwg_generate; host-side errors
    (batch binding, range) come before anything is enqueued."""
    cfg = W.ModelConfig(W.RELU, W.F32, 32, (1, 2, 4, 8))
    ref, na = _pair(cfg, 6)
    assert ref.regime == "chain_f32_c32"
    u = W.uniforms(44, 6, 70)
    want = ref.generate(_dev(u)).cpu().numpy()
    out = torch.empty((6, 70), dtype=torch.int32, device="cuda")
    assert np.array_equal(na.generate_noalloc(_dev(u), out).cpu().numpy(), want)
    with pytest.raises(binding.FwgError) as e:
        na.generate_noalloc(_dev(W.uniforms(1, 3, 5)), torch.empty((3, 5), dtype=torch.int32, device="cuda"))
    assert e.value.code == binding.FWG_ESTATE
    with pytest.raises(binding.FwgError) as e:
        na.generate_noalloc(_dev(W.uniforms(1, 7, 5)), torch.empty((7, 5), dtype=torch.int32, device="cuda"))
    assert e.value.code == binding.FWG_EINVAL
