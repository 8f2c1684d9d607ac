"""The benchmark's output contract: one JSON line with the fields a driver
reads, consistent with itself (value = B*T / seconds per step, roofline
fraction = achieved / peak), the per-kernel flop accounting that the
roofline divides, the oracle baseline leg, and the refusal of more than one
GPU."""

import json
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2205_01435_amd import workloads as wl  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


@pytest.mark.parametrize("name", ["tiny_rollout", "medium_rollout", "large_rollout", "xlarge_rollout"])
def test_kernel_flops_add_up_to_the_transition(name):
    """The three kernel classes of a multi-launch step (gates, mixture head,
    controller with the reward and done heads) count every product of a
    transition once, and the persistent kernel counts B*T transitions."""
    w = wl.WORKLOADS[name]
    per_row = sum(bench.kernel_flops_per_launch(k, w, 1, 1) for k in ("gates", "mdn", "ctrl"))
    assert per_row == pytest.approx(bench.flops_per_transition(w), rel=1e-12)
    assert bench.kernel_flops_per_launch("persist", w, w.B, w.T) == pytest.approx(
        w.B * w.T * bench.flops_per_transition(w), rel=1e-12)
    # written out: 2 (4H(Z+H) + 3ZKH + A(Z+H) + 2H)
    Z, H, A, K = w.Z, w.H, w.A, w.K
    assert bench.flops_per_transition(w) == 2.0 * (4 * H * (Z + H) + 3 * Z * K * H + A * (Z + H) + 2 * H)


def test_weight_stream_bytes_of_the_tiny_rollout():
    """fp32: every matrix, min(B, A) gathered one-hot rows of 4H, fp32 biases."""
    w = wl.WORKLOADS["tiny_rollout"]
    Z, H, A, K = w.Z, w.H, w.A, w.K
    mats = 4 * H * (Z + H) + 3 * Z * K * H + 2 * H + A * (Z + H)
    expect = 4 * (mats + min(w.B, A) * 4 * H) + 4 * (4 * H + 3 * Z * K + 2 + A)
    assert bench.weight_stream_bytes_per_step(w) == expect


def test_cpu_baseline_leg():
    """The oracle timing on a bounded sample: a positive rate and the fields
    the JSON line carries."""
    w = wl.WORKLOADS["tiny_rollout"]
    out = bench.cpu_baseline(w, wl.make_rollout_inputs(w), budget_s=0.2)
    assert out["kind"] == "oracle" and out["unit"] == "transitions/s"
    assert out["value"] > 0 and out["cores"] >= 1
    assert "tiny_rollout" in out["sample"]


@pytest.mark.gpu
@pytest.mark.timeout(600)
def test_bench_json_line():
    """A short run of the benchmark (no oracle leg, no per-workload table):
    one JSON line whose fields agree with each other."""
    print("bench.py --steps 2 --warmup 1 --no-cpu-baseline --no-workloads", flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "2", "--warmup", "1",
                        "--no-cpu-baseline", "--no-workloads"],
                       capture_output=True, text=True, timeout=540)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
              "scaling", "vs_baseline", "dtype", "data", "config", "roofline"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 2 and d["warmup"] == 1
    assert d["higher_is_better"] is True and d["dtype"] == "bf16" and d["unit"] == "transitions/s"
    w = wl.WORKLOADS[bench.HEADLINE]
    assert d["config"]["B"] == w.B and d["config"]["T"] == w.T
    assert d["value"] == pytest.approx(w.B * w.T / (d["ms_per_step"] / 1e3), rel=1e-9)
    rf = d["roofline"]
    assert rf["bound"] == "mfma" and rf["unit"] == "TFLOP/s" and rf["peak"] == pytest.approx(2516.6)
    assert rf["frac"] == pytest.approx(rf["achieved"] / rf["peak"], rel=1e-9)
    assert 0.0 < rf["frac"] < 1.0
    assert rf["launches"] > 0 and rf["avg_launch_us"] > 0
    # achieved = flops per launch / average launch time
    assert rf["achieved"] * 1e12 == pytest.approx(rf["flops_per_launch"] / (rf["avg_launch_us"] * 1e-6), rel=1e-9)
    assert rf["traffic"] is None or rf["traffic"] > 0
    assert np.isfinite(d["value"]) and d["value"] > 0
