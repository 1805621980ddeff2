"""CPU checks of bench.py's host-side tools (no GPU): the traffic record written from rocprofv3
counter passes."""
import csv
import json
import os

import bench

HEADER = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id", "Grid_Size",
          "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size", "Scratch_Size", "VGPR_Count",
          "Accum_VGPR_Count", "SGPR_Count", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _write(path, counter, rows):
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, f"{counter}_counter_collection.csv"), "w", newline="") as f:
        wr = csv.writer(f)
        wr.writerow(HEADER)
        for i, (name, value) in enumerate(rows, 1):
            wr.writerow([i, i, "Agent 1", 1, 1, 1, 64, 1, name, 256, 0, 0, 8, 0, 16, counter, value, 0, 1])


def test_record_traffic(tmp_path):
    """The timed launch is the last dispatch of the step kernel; each counter is scaled by what it
    reads for a 256 MiB device copy; other kernels and the copy's helper kernels are ignored."""
    kib = 256 * 1024  # the copy moves 256 MiB
    _write(tmp_path / "FETCH_SIZE", "FETCH_SIZE", [("fwg::sp::split_step_kernel(fwg::StepArgs)", 1000.0),
                                                   ("fwg::fill_zero_kernel", 5.0),
                                                   ("fwg::sp::split_step_kernel(fwg::StepArgs)", 3000.0)])
    _write(tmp_path / "WRITE_SIZE", "WRITE_SIZE", [("fwg::sp::split_step_kernel(fwg::StepArgs)", 2000.0),
                                                   ("fwg::sp::split_step_kernel(fwg::StepArgs)", 4000.0)])
    # the copy reads half of what it moves (the counter's unit), and writes it all
    _write(tmp_path / "copy_FETCH_SIZE", "FETCH_SIZE", [("vectorized_elementwise_kernel", 10.0)] +
           [("__amd_rocclr_copyBuffer", kib / 2)] * 3)
    _write(tmp_path / "copy_WRITE_SIZE", "WRITE_SIZE", [("__amd_rocclr_copyBuffer", float(kib))] * 3)
    out = tmp_path / "traffic.json"
    rec = bench.record_traffic(str(tmp_path), "w", 8000, out_path=str(out))
    assert rec["fetch_size_kib"] == 3000.0 and rec["write_size_kib"] == 4000.0
    assert abs(rec["fetch_factor"] - 2.0) < 1e-12 and abs(rec["write_factor"] - 1.0) < 1e-12
    assert abs(rec["hbm_bytes_per_launch"] - (3000.0 * 2 + 4000.0) * 1024) < 1e-6
    assert rec["kernel_digest"] == bench.kernel_source_digest()
    assert json.load(open(out))["hbm_bytes_per_launch"] == rec["hbm_bytes_per_launch"]


def test_stored_traffic_matches_sources():
    """The committed traffic record of the benchmark workload is reported only while it was taken on
    the current step-kernel sources, and scales per step to any launch length."""
    rec = json.load(open(os.path.join(bench.ROOT, "profiles", "traffic_gated_r64_s512_l30_b256_bf16.json")))
    v = bench.stored_traffic("gated_r64_s512_l30_b256_bf16")
    if rec["kernel_digest"] == bench.kernel_source_digest():
        assert v == rec
        assert bench.traffic_for(v, rec["steps"]) == rec["hbm_bytes_per_launch"]
        assert abs(bench.traffic_for(v, 20) - rec["hbm_bytes_per_launch"] * 20 / rec["steps"]) < 1.0
    else:
        assert v is None and bench.traffic_for(v, 20) is None


def test_cpu_baseline_counts_the_steps_it_runs():
    """The CPU baseline draws its own uniforms and divides by exactly the steps the oracle ran,
    whatever the GPU run's length (a 20-step GPU run once made it divide 16 steps' time by 7,996)."""
    import workloads as W
    wl = W.WORKLOADS["toy_relu_c32_l5_b1"]
    w = W.make_weights(wl.model, wl.weight_seed)
    for budget in (0.0, 0.05):
        r = bench.cpu_baseline(wl, w, budget)
        assert r["steps_run"] >= 8 and r["steps_run"] <= wl.n_steps - 4
        assert abs(r["value"] - r["streams"] * r["steps_run"] / r["seconds"]) <= 1e-9 * r["value"]
        assert f"{r['streams']} x {r['steps_run']} samples" in r["sample"]
    r = bench.cpu_baseline_tf(wl, w, 0.0)
    assert r["steps_run"] == 16
    assert abs(r["value"] - r["streams"] * 16 / r["seconds"]) <= 1e-9 * r["value"]
    r = bench.cpu_baseline_online(wl, w, 0.0)
    assert r["steps_run"] == 16
    assert abs(r["value"] - r["streams"] * 16 / r["seconds"]) <= 1e-9 * r["value"]
    assert f"{r['streams']} x 16 samples" in r["sample"]
