"""The one-line JSON report of bench.py: its keys, their units and the relations
between them, on a short run of the default workload (the ViT-B/16 512 px batch),
and the refusal of a multi-GPU run."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, BENCH, "--gpus", "2"], capture_output=True, text=True, timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr
    assert p.stdout.strip() == ""


@pytest.mark.gpu
def test_report_line():
    sys.path.insert(0, ROOT)
    import bench

    cmd = [sys.executable, BENCH, "--steps", "5", "--warmup", "2", "--cpu-seconds", "1", "--cpu-single-seconds",
           "0.5", "--cold-steps", "1", "--prewarm-seconds", "0.1"]
    print("bench report: " + " ".join(cmd[1:]), flush=True)
    p = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert p.returncode == 0, p.stderr[-3000:]
    lines = [ln for ln in p.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, p.stdout
    r = json.loads(lines[0])

    assert r["metric"] == bench.METRIC
    assert r["unit"] == "images/s" and r["higher_is_better"] is True
    assert (r["n_gpus"], r["steps"], r["warmup"]) == (1, 5, 2)
    assert r["scaling"] == "weak" and r["vs_baseline"] is None
    assert r["dtype"] == "bf16" and r["data"] == "synthetic"
    assert r["config"]["workload"].startswith("vit_b_512") and r["config"]["global_batch"] == 64
    assert r["ms_per_step"] > 0
    assert abs(r["value"] - 64 / (r["ms_per_step"] * 1e-3)) <= 0.01 * r["value"]  # rounding of ms_per_step

    rf = r["roofline"]
    assert (rf["bound"], rf["peak"], rf["unit"]) == ("mfma", bench.PEAK_BF16_TFLOPS, "TFLOP/s")
    assert rf["achieved"] > 0 and abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-3
    assert rf["schedule"] == "symmetric"
    assert 0 < rf["frac_issued"] < rf["frac"]  # the symmetric schedule issues less than the dense S
    if bench.TRAFFIC["source_sha256"] == bench.kernel_source_hash():
        assert rf["traffic"] == bench.TRAFFIC["bytes_per_launch"]["vit_b_512"]
    else:
        assert rf["traffic"] is None
    # The roofline's launch time is the back-to-back figure; the launch-bound events
    # read at least as long (they add idle time next to the launches).
    at = r["affinity_timing"]
    assert at["method"] == "back to back" and len(at["us"]) == 2 == len(at["launch_bound_events_us"])
    mean_us = sum(at["us"]) / 2
    flops = [k["gflop"] for k in r["kernels"] if k["name"].startswith("affinity")]
    assert abs(rf["achieved"] - sum(flops) / 2 * 1e9 / (mean_us * 1e-6) / 1e12) <= 0.01 * rf["achieved"]

    cb = r["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["unit"] == "images/s" and cb["value"] > 0 and cb["cores"] >= 1
    assert isinstance(cb["sample"], str) and cb["sample"]
    assert r["cpu_baseline_single_thread"]["cores"] == 1
    names = [k["name"] for k in r["kernels"]]
    assert names == ["affinity+compact1", "average1", "affinity+compact2", "average2", "compose+unmerge"]
