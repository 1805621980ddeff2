"""Python wrapper of the Fast Wavenet CPU oracle (fwo.c).

TEST INFRASTRUCTURE ONLY: imported by tests/, by the smoke check and by the
benchmark's CPU-baseline leg.  The product package never imports it.

The oracle receives the same seeded arrays as the GPU path (from `workloads`)
and converts them to float64; bf16 models pass weights whose float32 values
are already bf16, so the conversion is exact.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = [os.path.join(_HERE, "fwo.c"), os.path.join(_HERE, "fwo.h")]
LIB_PATH = os.path.join(_HERE, "liboracle.so")

GCC_CMD = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-o", LIB_PATH,
           os.path.join(_HERE, "fwo.c"), "-lm"]


def build(force: bool = False) -> str:
    """Compile liboracle.so with gcc (plain -O2, no fast-math)."""
    stale = not os.path.exists(LIB_PATH) or any(
        os.path.getmtime(s) > os.path.getmtime(LIB_PATH) for s in _SRC)
    if force or stale:
        tmp = LIB_PATH + ".tmp"
        cmd = GCC_CMD[:-3] + [tmp] + GCC_CMD[-2:]
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(LIB_PATH)
        dp, ip, fp = ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_float)
        L.fwo_state_new.restype = ctypes.c_void_p
        L.fwo_state_new.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int]
        L.fwo_state_free.argtypes = [ctypes.c_void_p]
        L.fwo_state_reset.argtypes = [ctypes.c_void_p]
        L.fwo_state_t.restype = ctypes.c_longlong
        L.fwo_state_t.argtypes = [ctypes.c_void_p]
        L.fwo_generate.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, fp, ip, dp]
        L.fwo_step_forced.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ip, dp]
        L.fwo_teacher_forced.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ip, dp]
        L.fwo_parallel.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ip, dp]
        L.fwo_naive.argtypes = [ctypes.c_void_p, ip, ctypes.c_int, dp]
        L.fwo_sample.argtypes = [fp, ctypes.c_int, ctypes.c_float]
        L.fwo_sample.restype = ctypes.c_int
        L.fwo_cdf.argtypes = [dp, ctypes.c_int, dp]
        L.fwo_bf16_round.argtypes = [ctypes.c_double]
        L.fwo_bf16_round.restype = ctypes.c_double
        L.fwo_max_threads.restype = ctypes.c_int
        _lib = L
    return _lib


class _Model(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int), ("bf16", ctypes.c_int),
        ("Q", ctypes.c_int), ("C", ctypes.c_int), ("S", ctypes.c_int), ("H", ctypes.c_int), ("L", ctypes.c_int),
        ("dil", ctypes.POINTER(ctypes.c_int)),
        ("embed", ctypes.c_void_p), ("embed_b", ctypes.c_void_p),
        ("conv", ctypes.c_void_p), ("conv_b", ctypes.c_void_p),
        ("res", ctypes.c_void_p), ("res_b", ctypes.c_void_p),
        ("skip", ctypes.c_void_p), ("skip_b", ctypes.c_void_p),
        ("head", ctypes.c_void_p), ("head_b", ctypes.c_void_p),
        ("out", ctypes.c_void_p), ("out_b", ctypes.c_void_p),
        ("products", ctypes.POINTER(ctypes.c_longlong)),
        ("w", ctypes.c_int),
    ]


def _ptr(a: Optional[np.ndarray]) -> Optional[int]:
    return None if a is None else a.ctypes.data


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


class Oracle:
    """Oracle bound to one model's weights (a `workloads.Weights`)."""

    def __init__(self, weights, count_products: bool = False):
        cfg = weights.cfg
        self.cfg = cfg
        keep = []

        def d(a):
            if a is None:
                return None
            arr = np.ascontiguousarray(a, dtype=np.float64)
            keep.append(arr)
            return arr

        def table(lst):
            arrs = [d(a) for a in lst]
            t = (ctypes.c_void_p * max(1, len(arrs)))(*[_ptr(a) for a in arrs])
            keep.append(t)
            return ctypes.cast(t, ctypes.c_void_p).value

        self._dil = _i32(cfg.dilations)
        self._counter = ctypes.c_longlong(0)
        m = _Model()
        m.kind, m.bf16 = cfg.kind, int(cfg.dtype == 1)
        m.Q, m.C, m.S, m.H, m.L = cfg.n_classes, cfg.channels, cfg.skip_channels, cfg.head_channels, cfg.n_layers
        m.dil = self._dil.ctypes.data_as(ctypes.POINTER(ctypes.c_int))
        m.embed, m.embed_b = _ptr(d(weights.embed)), _ptr(d(weights.embed_b))
        m.conv, m.conv_b = table(weights.conv), table(weights.conv_b)
        if cfg.kind == 2:
            m.res, m.res_b = table(weights.res), table(weights.res_b)
            m.skip, m.skip_b = table(weights.skip), table(weights.skip_b)
            m.head, m.head_b = _ptr(d(weights.head)), _ptr(d(weights.head_b))
        m.out, m.out_b = _ptr(d(weights.out)), _ptr(d(weights.out_b))
        m.w = cfg.filter_width
        if count_products:
            m.products = ctypes.pointer(self._counter)
        self._keep = keep
        self._m = m
        self._mp = ctypes.cast(ctypes.pointer(m), ctypes.c_void_p)

    # -- counters
    @property
    def products(self) -> int:
        return self._counter.value

    def reset_products(self):
        self._counter.value = 0

    # -- evaluation forms
    def teacher_forced(self, inputs) -> np.ndarray:
        x = _i32(inputs)
        B, T = x.shape
        out = np.empty((B, T, self.cfg.n_classes), np.float64)
        rc = lib().fwo_teacher_forced(self._mp, B, T, x.ctypes.data_as(ctypes.POINTER(ctypes.c_int)),
                                      out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
        assert rc == 0
        return out

    def parallel(self, inputs) -> np.ndarray:
        x = _i32(inputs)
        B, T = x.shape
        out = np.empty((B, T, self.cfg.n_classes), np.float64)
        rc = lib().fwo_parallel(self._mp, B, T, x.ctypes.data_as(ctypes.POINTER(ctypes.c_int)),
                                out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
        assert rc == 0
        return out

    def naive(self, inputs, t: int) -> np.ndarray:
        x = _i32(inputs)
        out = np.empty(self.cfg.n_classes, np.float64)
        rc = lib().fwo_naive(self._mp, x.ctypes.data_as(ctypes.POINTER(ctypes.c_int)), int(t),
                             out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
        assert rc == 0
        return out

    def state(self, batch: int, seed_input: Optional[int] = None) -> "OracleState":
        return OracleState(self, batch, self.cfg.seed_input if seed_input is None else seed_input)


class OracleState:
    """Generation state: per-stream queues, step counter and last sample."""

    def __init__(self, oracle: Oracle, batch: int, seed_input: int):
        self.oracle = oracle
        self.batch = batch
        self._h = lib().fwo_state_new(oracle._mp, batch, seed_input)
        assert self._h

    def __del__(self):
        h = getattr(self, "_h", None)
        if h:
            lib().fwo_state_free(h)
            self._h = None

    def reset(self):
        lib().fwo_state_reset(self._h)

    @property
    def t(self) -> int:
        return lib().fwo_state_t(self._h)

    def generate(self, u, return_logits: bool = False):
        u = np.ascontiguousarray(u, dtype=np.float32)
        B, n = u.shape
        assert B == self.batch
        samples = np.empty((B, n), np.int32)
        logits = np.empty((B, n, self.oracle.cfg.n_classes), np.float64) if return_logits else None
        rc = lib().fwo_generate(self.oracle._mp, self._h, n,
                                u.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                                samples.ctypes.data_as(ctypes.POINTER(ctypes.c_int)),
                                None if logits is None else logits.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
        assert rc == 0
        return (samples, logits) if return_logits else samples

    def step_forced(self, inputs) -> np.ndarray:
        """Online prediction: logits[b][i] is the distribution of inputs[b][i] given everything before."""
        x = _i32(inputs)
        B, n = x.shape
        assert B == self.batch
        logits = np.empty((B, n, self.oracle.cfg.n_classes), np.float64)
        rc = lib().fwo_step_forced(self.oracle._mp, self._h, n, x.ctypes.data_as(ctypes.POINTER(ctypes.c_int)),
                                   logits.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
        assert rc == 0
        return logits


def sample(logits_row, u: float) -> int:
    lf = np.ascontiguousarray(logits_row, dtype=np.float32)
    return lib().fwo_sample(lf.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), lf.size, ctypes.c_float(u))


def cdf(logits_row) -> np.ndarray:
    lg = np.ascontiguousarray(logits_row, dtype=np.float64)
    out = np.empty_like(lg)
    lib().fwo_cdf(lg.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), lg.size,
                  out.ctypes.data_as(ctypes.POINTER(ctypes.c_double)))
    return out


def bf16_round(x: float) -> float:
    return lib().fwo_bf16_round(float(x))


def max_threads() -> int:
    return lib().fwo_max_threads()
