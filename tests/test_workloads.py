"""The seeded input generators shared by both sides (no method arithmetic here)."""
import os

import numpy as np
import torch

import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_splitmix64_published_outputs():
    want = [int(l, 16) for l in open(os.path.join(GOLDEN, "splitmix64.txt")) if l.startswith("0x")]
    gamma = 0x9E3779B97F4A7C15
    states = np.array([(gamma * (i + 1)) % 2 ** 64 for i in range(len(want))], dtype=np.uint64)
    assert [int(v) for v in W.splitmix64_mix(states)] == want


def test_uniforms_counter_based():
    u = W.uniforms(3, 8, 100)
    assert u.dtype == np.float32 and u.shape == (8, 100)
    assert (u >= 0).all() and (u < 1).all()
    assert np.array_equal((u * 2 ** 24), np.floor(u * 2 ** 24))
    # entry (b, s) depends only on (seed, stream, step): windows agree with the full draw
    assert np.array_equal(W.uniforms(3, 3, 40, t0=55, stream0=2), u[2:5, 55:95])
    assert not np.array_equal(W.uniforms(4, 8, 100), u)
    assert abs(float(u.mean()) - 0.5) < 0.02


def test_sequences_cover_classes():
    x = W.sequences(1, 4, 5000)
    assert x.dtype == np.int32 and x.min() == 0 and x.max() == 255
    assert np.array_equal(W.sequences(1, 2, 100, stream0=1), x[1:3, :100])


def test_bf16_weight_conversion_matches_torch():
    a = np.random.default_rng(0).standard_normal(50000).astype(np.float32)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(W.f32_to_bf16_bits(a), ref)
    assert np.array_equal(W.bf16_bits_to_f32(ref), torch.from_numpy(a).to(torch.bfloat16).float().numpy())


def test_weight_shapes_and_scale():
    wl = W.WORKLOADS["gated_r64_s512_l30_b256_bf16"]
    cfg = wl.model
    assert cfg.param_count() == 2_028_992
    assert cfg.queue_total == 3069 and cfg.receptive_field == 3070
    assert cfg.flops_per_sample() == 3_981_312
    w = W.make_weights(cfg, wl.weight_seed)
    assert w.embed.shape == (64, 256) and w.conv[0].shape == (128, 64, 2)
    assert w.res[0].shape == (64, 64) and w.skip[0].shape == (512, 64)
    assert w.head.shape == (512, 512) and w.out.shape == (256, 512)
    # bf16 models hold exactly representable values
    assert np.array_equal(W.bf16_bits_to_f32(W.f32_to_bf16_bits(w.conv[3])).reshape(w.conv[3].shape), w.conv[3])
    # N(0, 1/fan_in): fan_in = 2C for the dilated conv
    assert abs(float(w.conv[0].std()) * np.sqrt(128) - 1) < 0.05
    assert all((b == 0).all() for b in w.conv_b)
    w2 = W.make_weights(cfg, wl.weight_seed)
    assert np.array_equal(w.out, w2.out)


def test_workload_table():
    t = W.WORKLOADS
    assert [w.model.queue_total for w in t.values()] == [31, 2046, 2046, 3069, 155, 4372, 4372]
    assert [w.model.flops_per_sample() for w in t.values()] == [36_864, 794_624, 794_624, 3_981_312, 26_476_544,
                                                                692_224, 2_506_752]
    assert W.BENCH_WORKLOAD in t
