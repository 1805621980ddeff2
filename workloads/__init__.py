"""Seeded synthetic inputs for Fast Wavenet generation: model shapes, weights,
uniform draws and teacher-forcing sequences.

This module is the only code shared by the GPU path's callers (tests, bench)
and the CPU oracle.  It holds none of the method's arithmetic: it only draws
numbers and lays them out.  The random numbers the method consumes (one
uniform per stream and step for inverse-CDF sampling) are produced here and
passed in to both sides as inputs.

Five workloads are defined: a toy ReLU stack, WaveNet-style gated stacks
(2 blocks x 10 layers in fp32, 3 blocks x 10 layers in bf16) and a
ByteNet-decoder-style ReLU+residual stack (the paper names ByteNet's decoder as
another user of the scheme, Section 1).  The paper (Section 2.2) fixes only the
structure: a generation model equal to one step of a multi-layer RNN, fed by
one FIFO queue per layer whose depth is that layer's dilation.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Sequence

import numpy as np

RELU = 0           # x^l = relu(W_r x^{l-1}_{t-d} + W_e x^{l-1}_t + b)
RELU_RESIDUAL = 1  # x^l = x^{l-1} + relu(...)
GATED = 2          # z = tanh(a[:R]) * sigmoid(a[R:]); x^l = x^{l-1} + W_res z; s += W_skip z
F32 = 0
BF16 = 1

KIND_NAMES = {RELU: "relu", RELU_RESIDUAL: "relu_residual", GATED: "gated"}


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    """Shape of one dilated causal stack with filter width 2."""
    kind: int
    dtype: int
    channels: int                 # C (relu kinds) or R (gated residual channels)
    dilations: tuple
    skip_channels: int = 0        # S (gated only)
    head_channels: int = 0        # H (gated only)
    n_classes: int = 256
    seed_input: int = 128         # first input after a reset
    filter_width: int = 2         # w: taps x_{t-(w-1)d}, ..., x_{t-d}, x_t (Section 3.1)

    @property
    def n_layers(self) -> int:
        return len(self.dilations)

    @property
    def conv_out(self) -> int:
        return 2 * self.channels if self.kind == GATED else self.channels

    @property
    def head_in(self) -> int:
        return self.head_channels if self.kind == GATED else self.channels

    @property
    def queue_total(self) -> int:
        """Sum of queue depths ((w - 1) d_l per layer): cached states per channel and stream."""
        return int((self.filter_width - 1) * sum(self.dilations))

    @property
    def receptive_field(self) -> int:
        return 1 + self.queue_total

    def param_count(self) -> int:
        C, Q = self.channels, self.n_classes
        n = C * Q + C  # embedding + bias
        for _ in self.dilations:
            n += self.conv_out * C * self.filter_width + self.conv_out
            if self.kind == GATED:
                n += C * C + C + self.skip_channels * C + self.skip_channels
        if self.kind == GATED:
            n += self.head_channels * self.skip_channels + self.head_channels
        n += Q * self.head_in + Q
        return n

    def macs_per_sample(self) -> int:
        """Multiply-accumulates of one generated sample (embedding gather excluded)."""
        C = self.channels
        per_layer = self.conv_out * self.filter_width * C
        if self.kind == GATED:
            per_layer += C * C + self.skip_channels * C
        n = per_layer * self.n_layers
        if self.kind == GATED:
            n += self.head_channels * self.skip_channels
        n += self.n_classes * self.head_in
        return n

    def flops_per_sample(self) -> int:
        return 2 * self.macs_per_sample()


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    model: ModelConfig
    batch: int
    n_steps: int
    weight_seed: int
    uniform_seed: int
    description: str


def _blocks(n_blocks: int, per_block: int) -> tuple:
    return tuple(2 ** i for i in range(per_block)) * n_blocks


WORKLOADS: Dict[str, Workload] = {
    w.name: w for w in [
        Workload("toy_relu_c32_l5_b1",
                 ModelConfig(RELU, F32, 32, (1, 2, 4, 8, 16)),
                 batch=1, n_steps=1000, weight_seed=0, uniform_seed=0,
                 description="toy ReLU stack, C=32, L=5, fp32, batch 1, 1,000 steps"),
        Workload("gated_r32_s256_l20_b1",
                 ModelConfig(GATED, F32, 32, _blocks(2, 10), skip_channels=256, head_channels=256),
                 batch=1, n_steps=16000, weight_seed=1, uniform_seed=1,
                 description="gated 2x10 layers, R=32, S=H=256, fp32, batch 1, 16,000 steps"),
        Workload("gated_r32_s256_l20_b64",
                 ModelConfig(GATED, F32, 32, _blocks(2, 10), skip_channels=256, head_channels=256),
                 batch=64, n_steps=16000, weight_seed=1, uniform_seed=1,
                 description="gated 2x10 layers, R=32, S=H=256, fp32, batch 64, 16,000 steps"),
        Workload("gated_r64_s512_l30_b256_bf16",
                 ModelConfig(GATED, BF16, 64, _blocks(3, 10), skip_channels=512, head_channels=512),
                 batch=256, n_steps=8000, weight_seed=2, uniform_seed=2,
                 description="gated 3x10 layers, R=64, S=H=512, bf16 operands / fp32 accumulation, "
                             "batch 256, 8,000 steps"),
        Workload("bytenet_relu_res_c512_l25_b32",
                 ModelConfig(RELU_RESIDUAL, F32, 512, _blocks(5, 5)),
                 batch=32, n_steps=4096, weight_seed=3, uniform_seed=3,
                 description="ByteNet-decoder-style ReLU+residual 5x5 layers, C=512, fp32, batch 32, 4,096 steps"),
        # filter width 3 with dilation rate r = w = 3 (Section 3.1: O(wL) work, O((w-1) r^L) queue space)
        Workload("gated_r32_s256_w3_l14_b64",
                 ModelConfig(GATED, F32, 32, tuple(3 ** i for i in range(7)) * 2, skip_channels=256,
                             head_channels=256, filter_width=3),
                 batch=64, n_steps=8000, weight_seed=4, uniform_seed=4,
                 description="gated 2x7 layers of filter width 3 (dilations 1..729 per block), R=32, S=H=256, "
                             "fp32, batch 64, 8,000 steps"),
        # the same width-3 layer pattern on the benchmark's layer shape (bf16 operands, R = 64)
        Workload("gated_r64_s512_w3_l14_b256_bf16",
                 ModelConfig(GATED, BF16, 64, tuple(3 ** i for i in range(7)) * 2, skip_channels=512,
                             head_channels=512, filter_width=3),
                 batch=256, n_steps=8000, weight_seed=5, uniform_seed=5,
                 description="gated 2x7 layers of filter width 3 (dilations 1..729 per block), R=64, S=H=512, "
                             "bf16 operands / fp32 accumulation, batch 256, 8,000 steps"),
    ]
}

BENCH_WORKLOAD = "gated_r64_s512_l30_b256_bf16"


# ---------------------------------------------------------------------------
# bf16 helpers (input preparation only: weights handed to both sides in bf16)
# ---------------------------------------------------------------------------
def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# ---------------------------------------------------------------------------
# Weights
# ---------------------------------------------------------------------------
@dataclasses.dataclass
class Weights:
    """Model weights in PyTorch layouts, float32 (for bf16 models: values already
    rounded to bf16, so float32 holds them exactly; `bits()` gives the uint16 form).

    embed   [C][Q]           1x1 conv over the one-hot input
    conv[l] [Cout][C][2]     tap 0 multiplies x_{t-d} (recurrent), tap 1 multiplies x_t
    res[l]  [R][R], skip[l] [S][R]             (gated only)
    head    [H][S]                              (gated only)
    out     [Q][C or H]
    biases: float32 vectors of the output width
    """
    cfg: ModelConfig
    embed: np.ndarray
    embed_b: np.ndarray
    conv: List[np.ndarray]
    conv_b: List[np.ndarray]
    res: List[np.ndarray]
    res_b: List[np.ndarray]
    skip: List[np.ndarray]
    skip_b: List[np.ndarray]
    head: Optional[np.ndarray]
    head_b: Optional[np.ndarray]
    out: np.ndarray
    out_b: np.ndarray

    def matrices(self) -> List[np.ndarray]:
        m = [self.embed]
        for l in range(self.cfg.n_layers):
            m.append(self.conv[l])
            if self.cfg.kind == GATED:
                m += [self.res[l], self.skip[l]]
        if self.cfg.kind == GATED:
            m.append(self.head)
        m.append(self.out)
        return m

    def nbytes(self) -> int:
        per = 2 if self.cfg.dtype == BF16 else 4
        return sum(m.size for m in self.matrices()) * per


def make_weights(cfg: ModelConfig, seed: int, bias_scale: float = 0.0,
                 bias_seed: Optional[int] = None) -> Weights:
    """Draw N(0, 1/fan_in) weights in a fixed order: embed, per layer (conv, [res, skip]),
    [head], out.  fan_in = input channels x kernel width (256 for the one-hot embedding).
    Biases are zero unless bias_scale > 0 (then N(0, bias_scale^2) from a separate stream)."""
    rng = np.random.default_rng(seed)
    C, Q, S, H = cfg.channels, cfg.n_classes, cfg.skip_channels, cfg.head_channels

    def draw(shape, fan_in):
        w = (rng.standard_normal(shape, dtype=np.float64) * fan_in ** -0.5).astype(np.float32)
        if cfg.dtype == BF16:
            w = bf16_bits_to_f32(f32_to_bf16_bits(w)).reshape(shape)
        return w

    embed = draw((C, Q), Q)
    conv, res, skip = [], [], []
    for _ in range(cfg.n_layers):
        conv.append(draw((cfg.conv_out, C, cfg.filter_width), cfg.filter_width * C))
        if cfg.kind == GATED:
            res.append(draw((C, C), C))
            skip.append(draw((S, C), C))
    head = draw((H, S), S) if cfg.kind == GATED else None
    out = draw((Q, cfg.head_in), cfg.head_in)

    brng = np.random.default_rng(seed + 1_000_003 if bias_seed is None else bias_seed)

    def bias(n):
        if bias_scale == 0.0:
            return np.zeros(n, np.float32)
        return (brng.standard_normal(n) * bias_scale).astype(np.float32)

    embed_b = bias(C)
    conv_b = [bias(cfg.conv_out) for _ in range(cfg.n_layers)]
    res_b = [bias(C) for _ in range(cfg.n_layers)] if cfg.kind == GATED else []
    skip_b = [bias(S) for _ in range(cfg.n_layers)] if cfg.kind == GATED else []
    head_b = bias(H) if cfg.kind == GATED else None
    out_b = bias(Q)
    return Weights(cfg, embed, embed_b, conv, conv_b, res, res_b, skip, skip_b, head, head_b, out, out_b)


# ---------------------------------------------------------------------------
# Counter-based uniforms and sequences (SplitMix64 finaliser over packed keys)
# ---------------------------------------------------------------------------
_GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)
DOMAIN_UNIFORM = 1
DOMAIN_SEQUENCE = 2


def splitmix64_mix(z: np.ndarray) -> np.ndarray:
    """Vigna's SplitMix64 output function applied to a uint64 array (wrapping arithmetic)."""
    z = np.asarray(z, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def _stream_keys(domain: int, seed: int, streams: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore"):
        k = splitmix64_mix(np.uint64(seed) * _GOLDEN + np.uint64(domain) + _GOLDEN)
        return splitmix64_mix((k ^ streams.astype(np.uint64)) + _GOLDEN)


def _raw(domain: int, seed: int, batch: int, n_steps: int, t0: int = 0,
         stream0: int = 0) -> np.ndarray:
    streams = np.arange(stream0, stream0 + batch, dtype=np.uint64)
    steps = np.arange(t0, t0 + n_steps, dtype=np.uint64)
    with np.errstate(over="ignore"):
        base = _stream_keys(domain, seed, streams)[:, None]
        return splitmix64_mix(base + (steps[None, :] + np.uint64(1)) * _GOLDEN)


def uniforms(seed: int, batch: int, n_steps: int, t0: int = 0, stream0: int = 0) -> np.ndarray:
    """[batch][n_steps] float32 in [0, 1): top 24 bits x 2^-24 (exact in float32).
    Entry (b, s) depends only on (seed, stream0 + b, t0 + s)."""
    r = _raw(DOMAIN_UNIFORM, seed, batch, n_steps, t0, stream0)
    return ((r >> np.uint64(40)).astype(np.float64) * 2.0 ** -24).astype(np.float32)


def sequences(seed: int, batch: int, length: int, n_classes: int = 256, stream0: int = 0) -> np.ndarray:
    """[batch][length] int32 class indices, uniform over n_classes (n_classes a power of 2 <= 256)."""
    r = _raw(DOMAIN_SEQUENCE, seed, batch, length, 0, stream0)
    return ((r >> np.uint64(56)) % np.uint64(n_classes)).astype(np.int32)


def tiny_model(kind: int, dtype: int = F32, channels: int = 4,
               dilations: Sequence[int] = (1, 2, 4), skip: int = 8, head: int = 8,
               n_classes: int = 256, seed_input: int = 128, filter_width: int = 2) -> ModelConfig:
    return ModelConfig(kind, dtype, channels, tuple(dilations),
                       skip_channels=skip if kind == GATED else 0,
                       head_channels=head if kind == GATED else 0,
                       n_classes=n_classes, seed_input=seed_input, filter_width=filter_width)
