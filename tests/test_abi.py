"""The C-ABI library loads, exports what include/fwg.h declares, and rejects bad
arguments on the host before touching a device (runs without a GPU)."""
import ctypes
import os
import re

import pytest

from paper_1611_09482_amd import binding as B
import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    from paper_1611_09482_amd import build
    if build.is_stale():
        build.build()
    return B.load_library()


def declared_functions():
    text = open(os.path.join(ROOT, "include", "fwg.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fwg_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert set(names) == set(B.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n


def _desc(**kw):
    base = dict(kind=W.GATED, dtype=W.BF16, channels=64, dilations=(1, 2, 4), max_batch=8,
                skip_channels=512, head_channels=512)
    base.update(kw)
    return B.make_desc(**base)


def _rc_size(lib, d):
    n = ctypes.c_size_t(0)
    return lib.fwg_workspace_size(ctypes.byref(d), ctypes.byref(n)), n.value


def test_workspace_size_for_every_workload(lib):
    for name, wl in W.WORKLOADS.items():
        m = wl.model
        d = B.make_desc(m.kind, m.dtype, m.channels, m.dilations, wl.batch, m.skip_channels,
                        m.head_channels, m.n_classes, m.seed_input, filter_width=m.filter_width)
        rc, n = _rc_size(lib, d)
        assert rc == B.FWG_OK, (name, lib.fwg_last_error())
        es = 2 if m.dtype == W.BF16 else 4
        queues = m.queue_total * wl.batch * m.channels * es
        # two queue regions (generation, teacher-forced) plus weights
        assert n >= 2 * queues + W.make_weights(m, 0).nbytes()
        # twice the streams: the queue regions grow with the batch (the kernel family, and with it the
        # packed weight arrays, may change: the 512-channel family takes at most 32 streams)
        d2 = B.make_desc(m.kind, m.dtype, m.channels, m.dilations, 2 * wl.batch, m.skip_channels,
                         m.head_channels, m.n_classes, m.seed_input, filter_width=m.filter_width)
        rc2, n2 = _rc_size(lib, d2)
        assert rc2 == B.FWG_OK and n2 >= 4 * queues + W.make_weights(m, 0).nbytes()


@pytest.mark.parametrize("kw,code", [
    (dict(dilations=()), B.FWG_EINVAL),
    (dict(dilations=(1, 0, 2)), B.FWG_EINVAL),
    (dict(kind=7), B.FWG_EINVAL),
    (dict(dtype=5), B.FWG_EINVAL),
    (dict(max_batch=0), B.FWG_EINVAL),
    (dict(seed_input=256), B.FWG_EINVAL),
    (dict(seed_input=-1), B.FWG_EINVAL),
    (dict(channels=0), B.FWG_EINVAL),
    (dict(skip_channels=0), B.FWG_EINVAL),
    (dict(n_classes=100, seed_input=5), B.FWG_EUNSUPPORTED),
    (dict(channels=3), B.FWG_EUNSUPPORTED),
    (dict(kind=W.RELU, dtype=W.F32, channels=6), B.FWG_EUNSUPPORTED),
])
def test_invalid_descriptors(lib, kw, code):
    rc, _ = _rc_size(lib, _desc(**kw))
    assert rc == code
    assert lib.fwg_last_error().decode()


def test_null_arguments(lib):
    n = ctypes.c_size_t(0)
    assert lib.fwg_workspace_size(None, ctypes.byref(n)) == B.FWG_EINVAL
    d = _desc()
    assert lib.fwg_workspace_size(ctypes.byref(d), None) == B.FWG_EINVAL
    h = ctypes.c_void_p(0)
    w = B.fwg_weights()
    assert lib.fwg_create(ctypes.byref(d), ctypes.byref(w), None, 0, None, ctypes.byref(h)) == B.FWG_EINVAL
    assert lib.fwg_create(ctypes.byref(d), ctypes.byref(w), 1 << 20, 1 << 40, None, None) == B.FWG_EINVAL
    assert lib.fwg_reset_queues(None) == B.FWG_EINVAL
    assert lib.fwg_generate(None, 1, 1, None, None) == B.FWG_EINVAL
    assert lib.fwg_generate_noalloc(None, 1, 1, None, None) == B.FWG_EINVAL
    assert lib.fwg_teacher_forced(None, 1, 1, None, None) == B.FWG_EINVAL
    assert lib.fwg_step_forced(None, 1, 1, None, None) == B.FWG_EINVAL
    assert lib.fwg_generate_naive(None, 1, 1, None, None) == B.FWG_EINVAL
    assert lib.fwg_teacher_forced_parallel(None, 1, 1, None, None) == B.FWG_EINVAL
    assert lib.fwg_prime(None, 1, 1, None, None) == B.FWG_EINVAL
    assert lib.fwg_naive_nodes(ctypes.byref(d), None) == B.FWG_EINVAL
    assert lib.fwg_destroy(None) == B.FWG_OK
    assert lib.fwg_regime(None) == b""


def test_workspace_checks_precede_device_work(lib):
    """Too small or misaligned workspaces are rejected before any HIP call (no device here)."""
    d = _desc()
    rc, need = _rc_size(lib, d)
    assert rc == 0
    w = B.fwg_weights()
    h = ctypes.c_void_p(0)
    fake = 1 << 30  # never dereferenced: the checks fail first
    assert lib.fwg_create(ctypes.byref(d), ctypes.byref(w), fake, need - 1, None, ctypes.byref(h)) == B.FWG_ENOSPACE
    assert lib.fwg_create(ctypes.byref(d), ctypes.byref(w), fake + 16, need, None, ctypes.byref(h)) == B.FWG_ENOSPACE
    # missing weights with a large enough workspace: EINVAL, still before any HIP call
    assert lib.fwg_create(ctypes.byref(d), ctypes.byref(w), fake, need, None, ctypes.byref(h)) == B.FWG_EINVAL
    assert h.value is None


def test_binding_raises_on_missing_library(tmp_path):
    with pytest.raises(FileNotFoundError):
        B.load_library(str(tmp_path / "nope.so"))


@pytest.mark.parametrize("L", [1, 2, 3, 5, 8, 12])
def test_naive_tree_node_counts(lib, L):
    """Section 3.1: the naive generator evaluates the tree of Fig. 1.  One block of dilations
    1, 2, ..., 2^(L-1) has 2^L - 1 layer nodes (O(2^L); the cached method evaluates L).  Two such
    blocks (the timing experiment's model): the top block is again a binary tree of 2^L - 1 nodes
    whose leaves span 2^L consecutive times, and level l of the bottom block spans
    2^(L+1) - 2^l consecutive times, (L - 1) 2^(L+1) + 2 in all."""
    one = tuple(2 ** i for i in range(L))
    for dil, want in [(one, 2 ** L - 1), (one + one, (2 ** L - 1) + (L - 1) * 2 ** (L + 1) + 2)]:
        d = B.make_desc(W.GATED, W.F32, 32, dil, 1, 256, 256)
        n = ctypes.c_int64(0)
        assert lib.fwg_naive_nodes(ctypes.byref(d), ctypes.byref(n)) == B.FWG_OK
        assert n.value == want, (dil, n.value, want)


def test_naive_nodes_equal_depth_without_branching(lib):
    """A stack whose every dilation exceeds the sum of the dilations below it branches at every
    level and never merges: 2^L - 1 nodes; equal dilations merge maximally (level l spans
    L - l + 1 times)."""
    d = B.make_desc(W.RELU, W.F32, 32, (1, 3, 9, 27), 1)
    n = ctypes.c_int64(0)
    assert lib.fwg_naive_nodes(ctypes.byref(d), ctypes.byref(n)) == B.FWG_OK and n.value == 15
    d = B.make_desc(W.RELU, W.F32, 32, (2, 2, 2, 2, 2), 1)
    assert lib.fwg_naive_nodes(ctypes.byref(d), ctypes.byref(n)) == B.FWG_OK and n.value == 5 + 4 + 3 + 2 + 1


@pytest.mark.parametrize("fw,r,L", [(3, 3, 4), (3, 5, 3), (4, 4, 3), (5, 7, 2)])
def test_naive_tree_node_counts_width(lib, fw, r, L):
    """Section 3.1, filter width w and dilations r^l with r >= w: the tree has w children per node
    and no two branches meet, (w^L - 1) / (w - 1) layer nodes (O(w^L)); the queues hold
    (w - 1)(r^L - 1) / (r - 1) states per channel and stream."""
    dil = tuple(r ** i for i in range(L))
    d = B.make_desc(W.RELU, W.F32, 32, dil, 1, filter_width=fw)
    n = ctypes.c_int64(0)
    assert lib.fwg_naive_nodes(ctypes.byref(d), ctypes.byref(n)) == B.FWG_OK
    assert n.value == (fw ** L - 1) // (fw - 1)
    cfg = W.ModelConfig(W.RELU, W.F32, 32, dil, filter_width=fw)
    assert cfg.queue_total == (fw - 1) * (r ** L - 1) // (r - 1)
    # the workspace grows with the queues: (w - 1) d_l slots per layer in two queue regions
    d2 = B.make_desc(W.RELU, W.F32, 32, dil, 1, filter_width=2)
    assert _rc_size(lib, d)[1] - _rc_size(lib, d2)[1] >= 2 * (fw - 2) * sum(dil) * 32 * 4


def test_filter_width_validation(lib):
    assert _rc_size(lib, _desc(filter_width=1))[0] == B.FWG_EINVAL
    assert _rc_size(lib, _desc(filter_width=-3))[0] == B.FWG_EINVAL
    assert _rc_size(lib, _desc(filter_width=17))[0] == B.FWG_EUNSUPPORTED
    assert _rc_size(lib, _desc(filter_width=0))[1] == _rc_size(lib, _desc(filter_width=2))[1]
