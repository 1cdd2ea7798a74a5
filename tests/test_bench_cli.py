"""bench.py's host-side contract (CPU only): the one-GPU rule, the guard
that attaches counter figures to the kernel source they were taken on, and
the bounded oracle baseline."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import workloads  # noqa: E402


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=300)


@pytest.mark.parametrize("n", ["2", "8"])
def test_more_than_one_gpu_is_refused(n):
    r = _run("--gpus", n)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr
    assert r.stdout == ""


def test_no_gpu_is_an_error_not_a_fallback():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is visible")
    r = _run("--steps", "1", "--warmup", "0", "--no-cpu-baseline")
    assert r.returncode == 1
    assert "no GPU visible" in r.stderr
    assert r.stdout == ""


def test_kernel_hash_ignores_comments_only(tmp_path, monkeypatch):
    src = tmp_path / "k.hip"
    src.write_text("// a comment\n__global__ void f() {\n  int x = 1; /* more */\n}\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "KERNEL_SOURCES", ["k.hip"])
    h0 = bench.kernel_hash()
    src.write_text("__global__ void f() {\n\n  int x = 1;   // changed comment\n}\n")
    assert bench.kernel_hash() == h0
    src.write_text("__global__ void f() {\n  int x = 2;\n}\n")
    assert bench.kernel_hash() != h0


def test_traffic_figure_only_for_its_kernel_and_workload(tmp_path, monkeypatch):
    f = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    f.write_text(json.dumps({"kernel_hash": bench.kernel_hash(), "workload": "w",
                             "hbm_bytes_per_launch": 123}))
    assert bench.measured_traffic("w") == 123
    assert bench.measured_traffic("other") is None
    f.write_text(json.dumps({"kernel_hash": "0" * 16, "workload": "w", "hbm_bytes_per_launch": 123}))
    assert bench.measured_traffic("w") is None
    f.write_text("not json")
    assert bench.measured_traffic("w") is None


def test_cpu_baseline_is_bounded_and_labelled():
    inst = workloads.make_config(1)
    r = bench.cpu_baseline(inst, 0.2)
    assert set(r) == {"value", "unit", "cores", "kind", "sample"}
    assert r["kind"] == "oracle" and r["unit"] == "TFLOP/s"
    assert 1 <= r["cores"] <= 16
    assert r["value"] > 0
