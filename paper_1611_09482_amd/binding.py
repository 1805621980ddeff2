"""ctypes binding of libfwg.so (include/fwg.h).  Argument marshalling only:
every step of the generation path runs in the library's HIP kernels."""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

FWG_OK, FWG_EINVAL, FWG_ENOSPACE, FWG_EHIP, FWG_ESTATE, FWG_EUNSUPPORTED, FWG_EDEVICE = 0, -1, -2, -3, -4, -5, -6
FWG_RELU, FWG_RELU_RESIDUAL, FWG_GATED = 0, 1, 2
FWG_F32, FWG_BF16 = 0, 1

_STATUS = {FWG_EINVAL: "EINVAL", FWG_ENOSPACE: "ENOSPACE", FWG_EHIP: "EHIP", FWG_ESTATE: "ESTATE",
           FWG_EUNSUPPORTED: "EUNSUPPORTED", FWG_EDEVICE: "EDEVICE"}

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfwg.so")

EXPORTED = ["fwg_workspace_size", "fwg_create", "fwg_reset_queues", "fwg_generate", "fwg_generate_noalloc",
            "fwg_teacher_forced",
            "fwg_step_forced", "fwg_teacher_forced_parallel", "fwg_prime", "fwg_generate_naive", "fwg_naive_nodes",
            "fwg_destroy", "fwg_last_error", "fwg_regime", "fwg_device_status"]


class FwgError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"fwg {_STATUS.get(code, code)}: {msg}")
        self.code = code


class fwg_desc(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("dtype", ctypes.c_int32), ("n_classes", ctypes.c_int32),
                ("channels", ctypes.c_int32), ("skip_channels", ctypes.c_int32),
                ("head_channels", ctypes.c_int32), ("n_layers", ctypes.c_int32), ("max_batch", ctypes.c_int32),
                ("seed_input", ctypes.c_int32), ("dilations", ctypes.POINTER(ctypes.c_int32)),
                ("filter_width", ctypes.c_int32)]


class fwg_weights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("embed_b", ctypes.c_void_p),
                ("conv", ctypes.c_void_p), ("conv_b", ctypes.c_void_p),
                ("res", ctypes.c_void_p), ("res_b", ctypes.c_void_p),
                ("skip", ctypes.c_void_p), ("skip_b", ctypes.c_void_p),
                ("head", ctypes.c_void_p), ("head_b", ctypes.c_void_p),
                ("out", ctypes.c_void_p), ("out_b", ctypes.c_void_p)]


_lib = None


def load_library(path: Optional[str] = None):
    """Load libfwg.so.  Raises if it is missing: there is no fallback path."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise FileNotFoundError(f"{p} is missing: build it with `python -c 'import __graft_entry__ as g; g.build()'`")
    L = ctypes.CDLL(p)
    vp, i32 = ctypes.c_void_p, ctypes.c_int32
    L.fwg_workspace_size.argtypes = [ctypes.POINTER(fwg_desc), ctypes.POINTER(ctypes.c_size_t)]
    L.fwg_create.argtypes = [ctypes.POINTER(fwg_desc), ctypes.POINTER(fwg_weights), vp, ctypes.c_size_t, vp,
                             ctypes.POINTER(vp)]
    L.fwg_reset_queues.argtypes = [vp]
    L.fwg_generate.argtypes = [vp, i32, i32, vp, vp]
    L.fwg_generate_noalloc.argtypes = [vp, i32, i32, vp, vp]
    L.fwg_teacher_forced.argtypes = [vp, i32, i32, vp, vp]
    L.fwg_step_forced.argtypes = [vp, i32, i32, vp, vp]
    L.fwg_teacher_forced_parallel.argtypes = [vp, i32, i32, vp, vp]
    L.fwg_prime.argtypes = [vp, i32, i32, vp, vp]
    L.fwg_generate_naive.argtypes = [vp, i32, i32, vp, vp]
    L.fwg_naive_nodes.argtypes = [ctypes.POINTER(fwg_desc), ctypes.POINTER(ctypes.c_int64)]
    L.fwg_destroy.argtypes = [vp]
    L.fwg_last_error.restype = ctypes.c_char_p
    L.fwg_regime.argtypes = [vp]
    L.fwg_regime.restype = ctypes.c_char_p
    L.fwg_device_status.argtypes = [vp]
    for name in ["fwg_workspace_size", "fwg_create", "fwg_reset_queues", "fwg_generate", "fwg_generate_noalloc",
                 "fwg_teacher_forced",
                 "fwg_step_forced", "fwg_teacher_forced_parallel", "fwg_prime", "fwg_generate_naive",
                 "fwg_naive_nodes", "fwg_destroy", "fwg_device_status"]:
        getattr(L, name).restype = ctypes.c_int
    if path is None:
        _lib = L
    return L


def _check(rc: int):
    if rc != FWG_OK:
        raise FwgError(rc, load_library().fwg_last_error().decode())


def make_desc(kind: int, dtype: int, channels: int, dilations: Sequence[int], max_batch: int,
              skip_channels: int = 0, head_channels: int = 0, n_classes: int = 256, seed_input: int = 128,
              filter_width: int = 2):
    dil = (ctypes.c_int32 * max(1, len(dilations)))(*[int(d) for d in dilations])
    d = fwg_desc(kind, dtype, n_classes, channels, skip_channels, head_channels, len(dilations), max_batch,
                 seed_input, ctypes.cast(dil, ctypes.POINTER(ctypes.c_int32)), filter_width)
    d._keep = dil
    return d


def workspace_size(desc: fwg_desc) -> int:
    n = ctypes.c_size_t(0)
    _check(load_library().fwg_workspace_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def naive_nodes(desc: fwg_desc) -> int:
    """Layer-node evaluations per sample of the naive generator (distinct nodes of the Fig. 1 tree)."""
    n = ctypes.c_int64(0)
    _check(load_library().fwg_naive_nodes(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


class FastWavenet:
    """One model on one device stream.

    weights: an object with the attributes of `fwg_weights` holding torch CUDA
    tensors in PyTorch layouts (per-layer attributes are lists), see
    include/fwg.h.  The library copies and repacks them at creation.
    workspace: optional caller-owned uint8 CUDA tensor of at least ws_bytes (default: allocated
    here); it must outlive the handle."""

    def __init__(self, kind: int, dtype: int, channels: int, dilations: Sequence[int], max_batch: int,
                 weights, skip_channels: int = 0, head_channels: int = 0, n_classes: int = 256,
                 seed_input: int = 128, stream=None, filter_width: int = 2, workspace=None):
        import torch
        self._torch = torch
        self.lib = load_library()
        self.n_classes = n_classes
        self.max_batch = max_batch
        self.desc = make_desc(kind, dtype, channels, dilations, max_batch, skip_channels, head_channels,
                              n_classes, seed_input, filter_width)
        self.ws_bytes = workspace_size(self.desc)
        self.device = torch.device("cuda", torch.cuda.current_device())
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        if workspace is None:
            workspace = torch.empty(self.ws_bytes, dtype=torch.uint8, device=self.device)
        assert workspace.dtype == torch.uint8 and workspace.is_cuda and workspace.is_contiguous()
        assert workspace.numel() >= self.ws_bytes
        self.workspace = workspace

        def ptr(t):
            return None if t is None else t.data_ptr()

        def table(lst):
            if lst is None:
                return None, None
            arr = (ctypes.c_void_p * max(1, len(lst)))(*[ptr(t) for t in lst])
            return arr, ctypes.cast(arr, ctypes.c_void_p).value

        keep = []
        fw = fwg_weights()
        fw.embed, fw.embed_b = ptr(weights.embed), ptr(weights.embed_b)
        for name in ["conv", "conv_b", "res", "res_b", "skip", "skip_b"]:
            arr, addr = table(getattr(weights, name, None))
            keep.append(arr)
            setattr(fw, name, addr)
        fw.head, fw.head_b = ptr(getattr(weights, "head", None)), ptr(getattr(weights, "head_b", None))
        fw.out, fw.out_b = ptr(weights.out), ptr(weights.out_b)
        h = ctypes.c_void_p(0)
        _check(self.lib.fwg_create(ctypes.byref(self.desc), ctypes.byref(fw), self.workspace.data_ptr(),
                                   self.ws_bytes, self.stream.cuda_stream, ctypes.byref(h)))
        self.handle = h
        # kernel families whose launches wait on each other's blocks: a wait that ran out leaves
        # invalid outputs and a sticky device mark, which the calls below check by default
        self._waits = self.regime.startswith(("mfma_split", "wide", "chain_pair"))

    def _after(self, check: bool):
        if check and self._waits:
            self.device_status()

    @property
    def regime(self) -> str:
        return self.lib.fwg_regime(self.handle).decode()

    def reset(self):
        _check(self.lib.fwg_reset_queues(self.handle))

    def device_status(self):
        """Synchronise the handle's stream and raise FwgError (EDEVICE) if a launch since the last
        reset ended without valid results."""
        _check(self.lib.fwg_device_status(self.handle))

    def generate(self, uniforms, out=None, check: bool = True):
        """uniforms: float32 CUDA tensor [batch][n_steps] -> int32 samples [batch][n_steps].
        check: for kernel families with cross-block waits, synchronise and raise FwgError (EDEVICE)
        if the launch ended without valid results (False: return right after the enqueue)."""
        torch = self._torch
        assert uniforms.dtype == torch.float32 and uniforms.is_cuda and uniforms.is_contiguous()
        B, n = uniforms.shape
        if out is None:
            out = torch.empty((B, n), dtype=torch.int32, device=uniforms.device)
        _check(self.lib.fwg_generate(self.handle, B, n, uniforms.data_ptr(), out.data_ptr()))
        self._after(check)
        return out

    def generate_noalloc(self, uniforms, out, check: bool = True):
        """fwg_generate_noalloc: generate() for callers that cannot allocate (the split family's
        exchange words in the library's static device array); `out` is required."""
        torch = self._torch
        assert uniforms.dtype == torch.float32 and uniforms.is_cuda and uniforms.is_contiguous()
        B, n = uniforms.shape
        assert out.dtype == torch.int32 and out.is_cuda and out.is_contiguous() and tuple(out.shape) == (B, n)
        _check(self.lib.fwg_generate_noalloc(self.handle, B, n, uniforms.data_ptr(), out.data_ptr()))
        self._after(check)
        return out

    def teacher_forced(self, inputs, out=None, check: bool = True):
        """inputs: int32 CUDA tensor [batch][T] -> float32 logits [batch][T][n_classes] (check as in
        generate)."""
        torch = self._torch
        assert inputs.dtype == torch.int32 and inputs.is_cuda and inputs.is_contiguous()
        B, T = inputs.shape
        if out is None:
            out = torch.empty((B, T, self.n_classes), dtype=torch.float32, device=inputs.device)
        _check(self.lib.fwg_teacher_forced(self.handle, B, T, inputs.data_ptr(), out.data_ptr()))
        self._after(check)
        return out

    def step_forced(self, inputs, out=None, check: bool = True):
        """Online prediction from the current state.  inputs: int32 CUDA tensor [batch][n_steps] of
        observed samples -> float32 logits [batch][n_steps][n_classes]; logits[b][s] is the
        distribution predicted for inputs[b][s] (check as in generate)."""
        torch = self._torch
        assert inputs.dtype == torch.int32 and inputs.is_cuda and inputs.is_contiguous()
        B, n = inputs.shape
        if out is None:
            out = torch.empty((B, n, self.n_classes), dtype=torch.float32, device=inputs.device)
        _check(self.lib.fwg_step_forced(self.handle, B, n, inputs.data_ptr(), out.data_ptr()))
        self._after(check)
        return out

    def generate_naive(self, uniforms, out=None):
        """The naive baseline generator (its own state): same contract as generate()."""
        torch = self._torch
        assert uniforms.dtype == torch.float32 and uniforms.is_cuda and uniforms.is_contiguous()
        B, n = uniforms.shape
        if out is None:
            out = torch.empty((B, n), dtype=torch.int32, device=uniforms.device)
        _check(self.lib.fwg_generate_naive(self.handle, B, n, uniforms.data_ptr(), out.data_ptr()))
        return out

    def teacher_forced_parallel(self, inputs, out=None):
        """Time-parallel teacher forcing (same contract as teacher_forced)."""
        torch = self._torch
        assert inputs.dtype == torch.int32 and inputs.is_cuda and inputs.is_contiguous()
        B, T = inputs.shape
        if out is None:
            out = torch.empty((B, T, self.n_classes), dtype=torch.float32, device=inputs.device)
        _check(self.lib.fwg_teacher_forced_parallel(self.handle, B, T, inputs.data_ptr(), out.data_ptr()))
        return out

    def prime(self, inputs, logits: bool = False):
        """Time-parallel online prediction / priming from the current state (fwg_prime): the state
        advances over the observed samples; returns the logits when asked for, else None."""
        torch = self._torch
        assert inputs.dtype == torch.int32 and inputs.is_cuda and inputs.is_contiguous()
        B, n = inputs.shape
        out = torch.empty((B, n, self.n_classes), dtype=torch.float32, device=inputs.device) if logits else None
        _check(self.lib.fwg_prime(self.handle, B, n, inputs.data_ptr(), None if out is None else out.data_ptr()))
        return out

    def close(self):
        if getattr(self, "handle", None):
            self.lib.fwg_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class DeviceWeights:
    """Weights as CUDA tensors (matrices in the model dtype, biases float32)."""


def upload_weights(w, dtype: int, device=None) -> DeviceWeights:
    """Copy host arrays with the `fwg_weights` attribute names (numpy, PyTorch layouts) to the
    device.  bf16 models: matrices are converted with torch's round-to-nearest-even cast."""
    import numpy as np
    import torch
    dev = device or torch.device("cuda", torch.cuda.current_device())
    mdt = torch.bfloat16 if dtype == FWG_BF16 else torch.float32

    def mat(a):
        return None if a is None else torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev).to(mdt).contiguous()

    def vec(a):
        return None if a is None else torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev)

    d = DeviceWeights()
    d.embed, d.embed_b = mat(w.embed), vec(w.embed_b)
    d.conv = [mat(a) for a in w.conv]
    d.conv_b = [vec(a) for a in w.conv_b]
    d.res = [mat(a) for a in w.res] or None
    d.res_b = [vec(a) for a in w.res_b] or None
    d.skip = [mat(a) for a in w.skip] or None
    d.skip_b = [vec(a) for a in w.skip_b] or None
    d.head, d.head_b = mat(getattr(w, "head", None)), vec(getattr(w, "head_b", None))
    d.out, d.out_b = mat(w.out), vec(w.out_b)
    return d


def from_model(cfg, weights, max_batch: int, stream=None, workspace=None) -> FastWavenet:
    """Build a FastWavenet from a model description with the fields kind, dtype, channels,
    dilations, skip_channels, head_channels, n_classes, seed_input and host weights (workspace: as
    for FastWavenet)."""
    dw = upload_weights(weights, cfg.dtype)
    return FastWavenet(cfg.kind, cfg.dtype, cfg.channels, cfg.dilations, max_batch, dw,
                       skip_channels=cfg.skip_channels, head_channels=cfg.head_channels,
                       n_classes=cfg.n_classes, seed_input=cfg.seed_input, stream=stream,
                       filter_width=getattr(cfg, "filter_width", 2), workspace=workspace)
