#!/usr/bin/env python3
"""Throughput of Fast Wavenet cached generation on one MI355X.

One "step" is one generation step of the whole batch: every stream pops its
queues, runs all layers, the head, the softmax and the inverse-CDF sample, and
pushes its new states.  The timed region is one fwg_generate call of --steps
steps (a single persistent kernel launch), bracketed by device synchronisation
and HIP events recorded on the launch stream, with inputs resident in HBM.

--mode teacher_forced times one teacher-forced call over the same batch and number
of steps instead (a seeded random input sequence, logits for every step): the
time-parallel fwg_teacher_forced_parallel, or with --tf-path step the step kernels
(fwg_teacher_forced), against the oracle's teacher-forced pass.

--mode naive_vs_fast runs the paper's timing experiment (Section 3.2): models of
2 blocks of L layers (dilations 1 .. 2^(L-1) per block), L = 1 .. 12, one stream,
generation time per sample of the cached method (fwg_generate) and of the naive
tree recomputation (fwg_generate_naive), each averaged over --repeats calls of
--naive-samples samples.

Prints one JSON line (see the design doc for the field definitions).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "generated samples/sec (batch x steps/s) + % HBM/MFMA roofline per config"
PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}   # dense MFMA peaks
# fp32 vector peak: 256 CUs x 2.4 GHz x 256 flop/clk (4 SIMDs x 16 lanes x 2 FMA issue x 2 flop);
# the factor 2 of FMA issue needs packed fp32, which this library keeps off, so 78.6 TFLOP/s is the
# ceiling its vector kernels can reach
VALU_F32_PEAK_TFLOPS = 157.3
HBM_PEAK_GBS = 8000.0


# sources of the benchmark's step kernel: the kernel file and the structures it reads
KERNEL_SOURCES = ("fwg_split.hip", "fwg_mfma.hip", "fwg_mfma_dev.h", "fwg_internal.h", "fwg_xchg.h")


def kernel_source_digest() -> str:
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_1611_09482_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def stored_traffic(workload: str):
    """The committed traffic record of the workload's benchmark kernel (rocprofv3 counter passes
    over one long launch), if it was taken on the current kernel sources; else None."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("kernel_digest") != kernel_source_digest() or not rec.get("steps"):
        return None
    return rec


def traffic_for(rec, steps: int):
    """HBM bytes of a launch of `steps` steps from a traffic record: the record's bytes per step
    (its launch's bytes over its steps; the launch-fixed part, the weights each block reads once, is
    below 0.1% of an 8,000-step launch) times `steps`."""
    if rec is None:
        return None
    return rec["hbm_bytes_per_launch"] / rec["steps"] * steps


def _counter_rows(path: str, counter: str):
    """(dispatch id, kernel name, value) of every dispatch in a rocprofv3 --pmc CSV directory."""
    import csv
    import glob
    files = glob.glob(os.path.join(path, "**", "*counter_collection.csv"), recursive=True)
    if len(files) != 1:
        raise SystemExit(f"expected one counter_collection.csv under {path}, found {len(files)}")
    per = {}
    for r in csv.DictReader(open(files[0])):
        if r["Counter_Name"] == counter:
            key = int(r["Dispatch_Id"])
            name, val = per.get(key, (r["Kernel_Name"], 0.0))
            per[key] = (name, val + float(r["Counter_Value"]))
    return [(k, n, v) for k, (n, v) in sorted(per.items())]


def record_traffic(root: str, workload: str, steps: int, kernel: str = "split_step_kernel", out_path=None) -> dict:
    """Write profiles/traffic_<workload>.json from four rocprofv3 counter passes under `root`:
    FETCH_SIZE/ and WRITE_SIZE/ of `python bench.py --no-cpu-baseline` (the last dispatch of the
    step kernel is the timed launch) and copy_FETCH_SIZE/, copy_WRITE_SIZE/ of
    `python bench.py --copy-calibration` (a 256 MiB device copy: the factor that turns each counter
    into bytes moved)."""
    copy_bytes_kib = (256 << 20) / 1024.0
    rec = {"kernel": kernel, "kernel_digest": kernel_source_digest(), "workload": workload, "steps": steps}
    total = 0.0
    for counter, key in (("FETCH_SIZE", "fetch"), ("WRITE_SIZE", "write")):
        launches = [v for _, n, v in _counter_rows(os.path.join(root, counter), counter) if kernel in n]
        copies = [v for _, n, v in _counter_rows(os.path.join(root, "copy_" + counter), counter)
                  if "copyBuffer" in n and v > 0.25 * copy_bytes_kib]
        if not launches or not copies:
            raise SystemExit(f"{counter}: no {kernel} dispatch or no copy dispatch found under {root}")
        factor = copy_bytes_kib / (sum(copies) / len(copies))
        rec[f"{key}_size_kib"] = launches[-1]
        rec[f"{key}_factor"] = factor
        total += launches[-1] * 1024.0 * factor
    rec["hbm_bytes_per_launch"] = total
    rec["hbm_bytes_per_step"] = total / steps
    rec["command"] = ("rocprofv3 --pmc FETCH_SIZE (then WRITE_SIZE) --output-format csv -d <dir>/<COUNTER> -o <COUNTER> "
                      "-- python bench.py --no-cpu-baseline; copy factors: rocprofv3 --pmc <COUNTER> --output-format csv "
                      "-d <dir>/copy_<COUNTER> -o copy_<COUNTER> -- python bench.py --copy-calibration; then "
                      "python bench.py --record-traffic <dir>")
    path = out_path or os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    with open(path, "w") as f:
        json.dump(rec, f, indent=1)
    return rec


def _oracle_build_note() -> str:
    import oracle
    return "float64 CPU oracle (" + " ".join(oracle.GCC_CMD[:4]) + ", no BLAS)"


def cpu_baseline(wl, weights, target_seconds: float):
    """The oracle as it stands, on this host's cores, on a bounded sample of the workload: the first
    streams (one per thread) generate a few calibration steps, then as many further steps as fit the
    time budget.  It draws its own uniforms (the workload's seed, those streams and steps), so the
    steps it runs do not depend on the GPU run's length; the rate counts exactly the steps the
    oracle's state advanced over in the timed call."""
    import oracle
    import workloads as W
    threads = oracle.max_threads()
    streams = max(1, min(wl.batch, threads))
    o = oracle.Oracle(weights)
    calib = 4
    st = o.state(streams)
    t0 = time.perf_counter()
    st.generate(W.uniforms(wl.uniform_seed, streams, calib))
    per_step = (time.perf_counter() - t0) / calib
    steps = int(max(8, min(wl.n_steps - calib, target_seconds / max(per_step, 1e-9))))
    u = W.uniforms(wl.uniform_seed, streams, steps, t0=calib)
    t_before = st.t
    t0 = time.perf_counter()
    st.generate(u)
    dt = time.perf_counter() - t0
    ran = st.t - t_before
    assert ran == steps == u.shape[1], (ran, steps, u.shape)
    return {"value": streams * ran / dt, "unit": "samples/s", "cores": min(threads, streams),
            "kind": "oracle", "streams": streams, "steps_run": ran, "seconds": dt,
            "sample": f"{_oracle_build_note()} generating streams 0..{streams - 1} of the {wl.batch}-stream "
                      f"workload for steps {calib}..{calib + ran - 1} of {wl.n_steps} (per-step cost does not "
                      f"depend on t), OpenMP over streams, {streams} x {ran} samples in {dt:.1f} s wall"}


def cpu_baseline_tf(wl, weights, target_seconds: float):
    """The oracle's teacher-forced pass on a bounded sample: the first streams (one per thread) over
    as many leading steps of the workload's seeded sequence as fit the time budget."""
    import oracle
    import workloads as W
    threads = oracle.max_threads()
    streams = max(1, min(wl.batch, threads))
    o = oracle.Oracle(weights)
    calib = 8
    t0 = time.perf_counter()
    o.teacher_forced(W.sequences(wl.uniform_seed, streams, calib))
    per_step = (time.perf_counter() - t0) / calib
    steps = int(max(16, min(wl.n_steps, target_seconds / max(per_step, 1e-9))))
    x = W.sequences(wl.uniform_seed, streams, steps)
    t0 = time.perf_counter()
    lg = o.teacher_forced(x)
    dt = time.perf_counter() - t0
    assert lg.shape[:2] == (streams, steps), lg.shape
    return {"value": streams * steps / dt, "unit": "samples/s", "cores": min(threads, streams),
            "kind": "oracle", "streams": streams, "steps_run": steps, "seconds": dt,
            "sample": f"{_oracle_build_note()} teacher-forcing streams 0..{streams - 1} of the {wl.batch}-stream "
                      f"workload over steps 0..{steps - 1} of {wl.n_steps} (cached form, per-step cost constant), "
                      f"OpenMP over streams, {streams} x {steps} samples in {dt:.1f} s wall"}


def cpu_baseline_online(wl, weights, target_seconds: float):
    """The oracle's online prediction (fwo_step_forced) on a bounded sample: the first streams (one
    per thread) over as many leading steps of the workload's seeded observed sequence as fit the time
    budget."""
    import oracle
    import workloads as W
    threads = oracle.max_threads()
    streams = max(1, min(wl.batch, threads))
    o = oracle.Oracle(weights)
    calib = 8
    t0 = time.perf_counter()
    oracle.OracleState(o, streams, wl.model.seed_input).step_forced(W.sequences(wl.uniform_seed, streams, calib))
    per_step = (time.perf_counter() - t0) / calib
    steps = int(max(16, min(wl.n_steps, target_seconds / max(per_step, 1e-9))))
    x = W.sequences(wl.uniform_seed, streams, steps)
    st = oracle.OracleState(o, streams, wl.model.seed_input)
    t0 = time.perf_counter()
    lg = st.step_forced(x)
    dt = time.perf_counter() - t0
    assert lg.shape[:2] == (streams, steps), lg.shape
    return {"value": streams * steps / dt, "unit": "samples/s", "cores": min(threads, streams),
            "kind": "oracle", "streams": streams, "steps_run": steps, "seconds": dt,
            "sample": f"{_oracle_build_note()} online prediction over streams 0..{streams - 1} of the "
                      f"{wl.batch}-stream workload for steps 0..{steps - 1} of {wl.n_steps} (per-step cost "
                      f"constant), OpenMP over streams, {streams} x {steps} samples in {dt:.1f} s wall"}


def bench_online(args, wl, name, fw, weights, stream, K, Wu):
    """One fwg_step_forced call (online prediction: each step reports the logits that predict the
    next observed sample, then takes that sample as its input) over the workload's batch and steps,
    on the same step kernels as generation."""
    import numpy as np
    import torch
    import workloads as W
    cfg = wl.model
    B = wl.batch
    x_host = W.sequences(wl.uniform_seed, B, max(K, Wu, 1))
    x = torch.from_numpy(np.ascontiguousarray(x_host[:, :K])).cuda()
    logits = torch.empty((B, K, cfg.n_classes), dtype=torch.float32, device="cuda")
    if Wu > 0:
        fw.step_forced(torch.from_numpy(np.ascontiguousarray(x_host[:, :Wu])).cuda(), check=False)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    e0.record(stream)
    fw.step_forced(x, out=logits, check=False)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = e0.elapsed_time(e1)
    sec = ms / 1e3
    fw.device_status()  # raises if the launch ended without valid results
    dtype = "bf16" if cfg.dtype == W.BF16 else "f32"
    samples = B * K
    flops = float(cfg.flops_per_sample()) * samples
    achieved = flops / sec / 1e12 if sec > 0 else 0.0
    mfma = fw.regime.startswith("mfma")
    peak = PEAK_TFLOPS[dtype] if mfma else VALU_F32_PEAK_TFLOPS
    result = {
        "metric": "online-prediction samples/sec (batch x steps/s)",
        "value": samples / sec if sec > 0 else 0.0,
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": Wu,
        "ms_per_step": ms / max(K, 1),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic",
        "config": {"workload": name, "description": wl.description, "batch": B, "seq_len": K,
                   "mode": "online", "regime": fw.regime},
        "roofline": {"bound": "mfma" if mfma else "alu", "achieved": achieved, "peak": peak,
                     "unit": "TFLOP/s", "frac": achieved / peak, "traffic": None,
                     "algorithmic_flops_per_launch": flops, "launch_ms": ms},
        "wall_s": wall,
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline_online(wl, weights, args.cpu_seconds)
    print(json.dumps(result), flush=True)


def bench_teacher_forced(args, wl, name, fw, weights, stream, K, Wu):
    import numpy as np
    import torch
    import workloads as W
    cfg = wl.model
    B = wl.batch
    x_host = W.sequences(wl.uniform_seed, B, max(K, Wu, 1))
    x = torch.from_numpy(np.ascontiguousarray(x_host[:, :K])).cuda()
    logits = torch.empty((B, K, cfg.n_classes), dtype=torch.float32, device="cuda")
    call = fw.teacher_forced if args.tf_path == "step" else fw.teacher_forced_parallel
    if Wu > 0:
        call(torch.from_numpy(np.ascontiguousarray(x_host[:, :Wu])).cuda())
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    e0.record(stream)
    call(x, out=logits)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = e0.elapsed_time(e1)
    sec = ms / 1e3
    dtype = "bf16" if cfg.dtype == W.BF16 else "f32"
    samples = B * K
    flops = float(cfg.flops_per_sample()) * samples
    achieved = flops / sec / 1e12 if sec > 0 else 0.0
    peak = PEAK_TFLOPS[dtype]
    result = {
        "metric": "teacher-forced samples/sec (batch x steps/s)",
        "value": samples / sec if sec > 0 else 0.0,
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": Wu,
        "ms_per_step": ms / max(K, 1),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic",
        "config": {"workload": name, "description": wl.description, "batch": B, "seq_len": K,
                   "mode": "teacher_forced",
                   "path": "step kernels" if args.tf_path == "step" else "time-parallel"},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak, "traffic": None, "scope": "whole call (all kernels)",
                     "algorithmic_flops_per_call": flops, "call_ms": ms},
        "wall_s": wall,
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline_tf(wl, weights, args.cpu_seconds)
    print(json.dumps(result), flush=True)


def naive_vs_fast(args):
    import numpy as np
    import torch
    import workloads as W
    from paper_1611_09482_amd import binding
    stream = torch.cuda.current_stream()
    n = args.naive_samples
    rows = []
    for L in range(1, args.max_blocks_layers + 1):
        dil = tuple(2 ** i for i in range(L)) * 2
        cfg = W.ModelConfig(W.GATED, W.F32, 32, dil, 256, 256)
        w = W.make_weights(cfg, 1)
        fw = binding.from_model(cfg, w, max_batch=1, stream=stream)
        d = binding.make_desc(cfg.kind, cfg.dtype, cfg.channels, cfg.dilations, 1, cfg.skip_channels,
                              cfg.head_channels)
        nodes = binding.naive_nodes(d)
        u = torch.from_numpy(W.uniforms(L, 1, n)).cuda()
        out = torch.empty((1, n), dtype=torch.int32, device="cuda")
        res = {}
        # the status of launches whose blocks wait on each other is checked after the timed calls,
        # not inside them (it synchronises the stream)
        fast = lambda uu, out: fw.generate(uu, out=out, check=False)
        for name, fn in (("fast", fast), ("naive", fw.generate_naive)):
            fn(u, out=out)  # warm-up call
            torch.cuda.synchronize()
            ms = []
            for _ in range(args.repeats):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                fn(u, out=out)
                e1.record(stream)
                torch.cuda.synchronize()
                ms.append(e0.elapsed_time(e1))
            res[name] = float(np.mean(ms)) / n
        fw.device_status()
        R, S, H, Q = 32, 256, 256, 256
        head = 2 * (2 * L) * R * S + 2 * S * H + 2 * H * Q
        fast_flops = cfg.flops_per_sample()
        naive_flops = nodes * 2 * (2 * R) * (2 * R) + (nodes - 1) * 2 * R * R + head
        rows.append({"L": L, "layers": 2 * L, "receptive_field": cfg.receptive_field,
                     "naive_nodes_per_sample": nodes, "fast_nodes_per_sample": 2 * L,
                     "fast_ms_per_sample": res["fast"], "naive_ms_per_sample": res["naive"],
                     "speedup": res["naive"] / res["fast"],
                     "fast_tflops": fast_flops / (res["fast"] * 1e-3) / 1e12,
                     "naive_tflops": naive_flops / (res["naive"] * 1e-3) / 1e12})
        print(json.dumps(rows[-1]), file=sys.stderr, flush=True)
        fw.close()
    print(json.dumps({"metric": "generation time per sample, naive vs cached (2 blocks of L layers)",
                      "unit": "ms/sample", "higher_is_better": False, "n_gpus": 1, "dtype": "f32",
                      "data": "synthetic",
                      "config": {"workload": "gated_r32_s256_2xL_b1",
                                 "description": "gated, R=32, S=H=256, fp32, 2 blocks of L layers "
                                                "(dilations 1..2^(L-1) per block), batch 1",
                                 "samples_per_call": n, "repeats": args.repeats},
                      "results": rows}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="generation steps timed (default: the workload's)")
    ap.add_argument("--warmup", type=int, default=None, help="untimed warm-up steps (default: same as --steps)")
    ap.add_argument("--workload", default=None)
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="wall-time budget of the CPU baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--mode", choices=["generate", "teacher_forced", "online", "naive_vs_fast"], default="generate")
    ap.add_argument("--tf-path", choices=["parallel", "step"], default="parallel",
                    help="teacher_forced mode: time-parallel kernels or the step kernels")
    ap.add_argument("--naive-samples", type=int, default=50, help="samples per timed call (naive_vs_fast)")
    ap.add_argument("--repeats", type=int, default=100, help="timed calls averaged (naive_vs_fast)")
    ap.add_argument("--max-blocks-layers", type=int, default=12, help="largest L of the sweep (naive_vs_fast)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 256 MiB device copy (counter calibration for rocprofv3)")
    ap.add_argument("--record-traffic", metavar="DIR", default=None,
                    help="write the traffic record of the benchmark launch from rocprofv3 counter passes under DIR "
                         "(no GPU needed)")
    args = ap.parse_args()

    if args.record_traffic:
        import workloads as W
        name = args.workload or W.BENCH_WORKLOAD
        print(json.dumps(record_traffic(args.record_traffic, name, args.steps or W.WORKLOADS[name].n_steps), indent=1))
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU: streams are independent and the path uses no collectives, so "
              f"--gpus {args.gpus} (WORLD_SIZE={world}) is not supported; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import workloads as W
    from paper_1611_09482_amd import binding

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)

    if args.copy_calibration:
        n = 256 << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n, "launches": 3}))
        return

    if args.mode == "naive_vs_fast":
        naive_vs_fast(args)
        return

    name = args.workload or W.BENCH_WORKLOAD
    wl = W.WORKLOADS[name]
    cfg = wl.model
    K = args.steps if args.steps is not None else wl.n_steps
    Wu = args.warmup if args.warmup is not None else K
    B = wl.batch

    weights = W.make_weights(cfg, wl.weight_seed)
    if args.mode == "teacher_forced":
        stream = torch.cuda.current_stream()
        fw = binding.from_model(cfg, weights, max_batch=B, stream=stream)
        bench_teacher_forced(args, wl, name, fw, weights, stream, K, Wu)
        return
    if args.mode == "online":
        stream = torch.cuda.current_stream()
        fw = binding.from_model(cfg, weights, max_batch=B, stream=stream)
        bench_online(args, wl, name, fw, weights, stream, K, Wu)
        return
    u_host = W.uniforms(wl.uniform_seed, B, max(K, Wu, 1))
    u_timed = torch.from_numpy(np.ascontiguousarray(u_host[:, :K])).cuda()
    u_warm = torch.from_numpy(np.ascontiguousarray(u_host[:, :Wu])).cuda()
    stream = torch.cuda.current_stream()
    fw = binding.from_model(cfg, weights, max_batch=B, stream=stream)
    out = torch.empty((B, K), dtype=torch.int32, device="cuda")

    # the warm-up steps, then the timed steps continue the same generation (queues, t and the pending
    # inputs carry over, as when a caller generates in chunks); every step does the same work
    if Wu > 0:
        fw.generate(u_warm, check=False)
    torch.cuda.synchronize()

    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    e0.record(stream)
    fw.generate(u_timed, out=out, check=False)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = e0.elapsed_time(e1)
    sec = ms / 1e3
    fw.device_status()  # raises if the launch ended without valid results

    dtype = "bf16" if cfg.dtype == W.BF16 else "f32"
    samples = B * K
    flops = float(cfg.flops_per_sample()) * samples
    achieved = flops / sec / 1e12 if sec > 0 else 0.0
    # the MFMA step kernels are bound by matrix-core work, the other step kernels multiply on the
    # vector ALUs in fp32; one stream (batch 1) takes the decode-style HBM roofline instead: every
    # step reads all weights once, pops and pushes its queue rows, reads a uniform, writes a sample
    mfma = fw.regime.startswith("mfma")
    es = 2 if cfg.dtype == W.BF16 else 4
    decode_bytes = (weights.nbytes() + cfg.n_layers * cfg.filter_width * cfg.channels * es * B + 8 * B) * K
    if B == 1:
        bound, peak, unit = "hbm", HBM_PEAK_GBS, "GB/s"
        achieved = decode_bytes / sec / 1e9 if sec > 0 else 0.0
    else:
        bound = "mfma" if mfma else "alu"
        peak, unit = (PEAK_TFLOPS[dtype] if mfma else VALU_F32_PEAK_TFLOPS), "TFLOP/s"
    rec = stored_traffic(name)
    traffic = traffic_for(rec, K)

    result = {
        "metric": METRIC,
        "value": samples / sec if sec > 0 else 0.0,
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": Wu,
        "ms_per_step": ms / max(K, 1),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic",
        "config": {
            "workload": name,
            "description": wl.description,
            "batch": B,
            "steps_per_launch": K,
            "regime": fw.regime,
        },
        "roofline": {
            "bound": bound,
            "achieved": achieved,
            "peak": peak,
            "unit": unit,
            "frac": achieved / peak,
            "traffic": traffic,
            "traffic_gbs": traffic / sec / 1e9 if traffic is not None and sec > 0 else None,
            "traffic_basis": None if rec is None else
            f"rocprofv3 FETCH_SIZE + WRITE_SIZE of a {rec['steps']}-step launch (copy-calibrated), per step x {K}",
            "algorithmic_flops_per_launch": flops,
            "algorithmic_tflops": flops / sec / 1e12 if sec > 0 else 0.0,
            "decode_bytes_per_launch": decode_bytes,
            "launch_ms": ms,
        },
        "wall_s": wall,
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, weights, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
