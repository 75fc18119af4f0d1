"""Host-side checks of bench.py: the one-GPU refusal, the source hash that
keys the committed traffic counters, and the arithmetic of those records."""

import glob
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_source_hash_ignores_comments_and_blank_lines(tmp_path):
    a = tmp_path / "a.hip"
    a.write_text("int f() {\n  return 1;  // one\n}\n")
    b = tmp_path / "b.hip"
    b.write_text("// header\n\nint f() {\n\n  return 1;\n}\n")
    c = tmp_path / "c.hip"
    c.write_text("int f() {\n  return 2;\n}\n")
    assert bench.kernel_code_sha256(a) == bench.kernel_code_sha256(b)
    assert bench.kernel_code_sha256(a) != bench.kernel_code_sha256(c)


@pytest.mark.parametrize("path", sorted(glob.glob(os.path.join(ROOT, "profiles", "k_step_traffic_*.json"))))
def test_committed_traffic_records_are_consistent(path):
    """Scaled traffic = raw counters x the calibration copy's scale; the scale
    maps the copy's counters to its 1 GiB; traffic within 1% of the
    algorithmic bytes (the kernel reads no unfinished row)."""
    rec = json.load(open(path))
    c = rec["calibration"]
    assert c["fetch_scale"] == pytest.approx((1 << 30) / (c["fetch_kib"] * 1024), rel=1e-12)
    assert c["write_scale"] == pytest.approx((1 << 30) / (c["write_kib"] * 1024), rel=1e-12)
    traffic = (rec["fetch_kib_per_dispatch_raw"] * c["fetch_scale"] +
               rec["write_kib_per_dispatch_raw"] * c["write_scale"]) * 1024
    assert rec["traffic_bytes_per_launch"] == pytest.approx(traffic, rel=1e-12)
    ratio = rec["traffic_bytes_per_launch"] / rec["alg_bytes_per_launch_same_dispatches"]
    assert rec["traffic_over_alg"] == pytest.approx(ratio, rel=1e-12)
    assert abs(ratio - 1.0) < 0.01
    assert rec["workload"] in os.path.basename(path)


def test_bench_imports_nothing_from_the_test_package():
    src = open(os.path.join(ROOT, "bench.py")).read()
    assert "tests." not in src and "from tests" not in src and "import tests" not in src


def test_cpu_baselines_run_on_the_oracle():
    """Both CPU-baseline legs on small workloads, with a tiny time budget:
    whole oracle iterations, the rate in the bench's units."""
    from synth import workloads

    r = bench.cpu_baseline(workloads.TINY, budget_s=0.2, cols=4096)
    assert r["kind"] == "oracle" and r["cores"] == 1 and r["value"] > 0
    assert "columns [0, 4096)" in r["sample"]
    from synth import mlp_data

    wl = workloads.MLP_TINY
    A = mlp_data.inputs(wl.seed, wl.n_samples, wl.d_in)
    y = mlp_data.teacher_labels(wl.seed, A, wl.hidden, wl.classes)
    x0 = mlp_data.student_init(wl.seed, wl.d_in, wl.hidden, wl.classes)
    r = bench.cpu_baseline_mlp(wl, A, y, x0, budget_s=0.2)
    assert r["unit"] == "samples/s" and r["value"] > 0 and "iterations 0.." in r["sample"]
