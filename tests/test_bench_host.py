"""CPU checks of the benchmark's host-side logic: the one-GPU guard, the HBM counter summary
(calibration against a 1 GiB copy) and the staleness rule for the committed summary."""
import csv
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def _write_counters(d, counter, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "pmc_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for i, (name, v) in enumerate(rows):
            w.writerow({"Dispatch_Id": i + 1, "Kernel_Name": name, "Counter_Name": counter,
                        "Counter_Value": v})


def test_counter_summary_scales_by_the_calibration_copy(tmp_path):
    gib_kib = float(1 << 20)
    # the counters read half the copy's fetched bytes and all of its written bytes; an input copy
    # of 4 GiB before the library's kernels is not a calibration copy
    fetch_rows = [("__amd_rocclr_copyBuffer", 2 * gib_kib),
                  ("ebd::evict_copy_kernel(ebd::EvictLaunch)", 1000.0),
                  ("ebd::evict_copy_kernel(ebd::EvictLaunch)", 3000.0),
                  ("void ebd::attend_split_kernel<7>(ebd::AttendLaunch, int)", 500.0),
                  ("__amd_rocclr_copyBuffer", gib_kib / 2), ("__amd_rocclr_copyBuffer", 4.0),
                  ("void at::native::reduce_kernel<512, 1>", gib_kib / 2)]
    write_rows = [("__amd_rocclr_copyBuffer", 4 * gib_kib),
                  ("ebd::evict_copy_kernel(ebd::EvictLaunch)", 2000.0),
                  ("ebd::evict_copy_kernel(ebd::EvictLaunch)", 2000.0),
                  ("void ebd::attend_split_kernel<7>(ebd::AttendLaunch, int)", 10.0),
                  ("__amd_rocclr_copyBuffer", gib_kib)]
    _write_counters(str(tmp_path / "f"), "FETCH_SIZE", fetch_rows)
    _write_counters(str(tmp_path / "w"), "WRITE_SIZE", write_rows)
    out = str(tmp_path / "out")
    assert bench.summarize_pmc(str(tmp_path / "f"), str(tmp_path / "w"), "unit_test", "cmd",
                               out_dir=out) == 0
    rec = json.load(open(os.path.join(out, "hbm_traffic_unit_test.json")))
    assert abs(rec["fetch_scale"] - 2.0) < 1e-12 and abs(rec["write_scale"] - 1.0) < 1e-12
    assert abs(rec["fetch_scale_read_only_sum"] - 2.0) < 1e-12
    k = rec["kernels"]["evict_copy"]
    assert k["fetch_bytes_per_launch"] == 2 * 2000 * 1024  # mean 2000 KiB, scaled by 2
    assert k["write_bytes_per_launch"] == 2000 * 1024
    assert k["launches_profiled"] == 2
    assert rec["kernels"]["attend_split"]["bytes_per_launch"] == (2 * 500 + 10) * 1024
    assert rec["kernel_sources_hash"] == bench.kernel_sources_hash()


def test_committed_traffic_is_used_only_while_the_sources_match():
    path = os.path.join(ROOT, "profiles", "hbm_traffic_llama8b_16k.json")
    rec = json.load(open(path))
    got = bench.load_traffic("llama8b_16k", "attend_split")
    if rec["kernel_sources_hash"] == bench.kernel_sources_hash():
        assert got == rec["kernels"]["attend_split"]["bytes_per_launch"]
    else:
        assert got is None
    assert bench.load_traffic("no_such_workload", "evict_copy") is None
