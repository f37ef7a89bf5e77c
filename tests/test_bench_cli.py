"""bench.py's command-line contract on the host: one GPU only (a request for several exits with a
message and a non-zero status before any GPU work), and the kernel-source hash that ties committed
counter summaries to the sources they were taken on."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("gpus", ["2", "8"])
def test_more_than_one_gpu_is_refused(gpus):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", gpus, "--steps", "1"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


def test_kernel_source_hash_is_stable_and_tracks_sources(tmp_path, monkeypatch):
    sys.path.insert(0, ROOT)
    import bench

    h = bench.kernel_source_hash()
    assert h == bench.kernel_source_hash() and len(h) == 16
    # a counter summary is used only when it was taken on the current sources
    (tmp_path / "profiles").mkdir()
    path = tmp_path / "profiles" / "epoch_w_traffic.json"
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: h)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("w") is None  # no summary
    path.write_text(json.dumps({"kernel_source_hash": h, "hbm_bytes_per_launch": 123.0}))
    assert bench.measured_traffic("w") == 123.0
    path.write_text(json.dumps({"kernel_source_hash": "0" * 16, "hbm_bytes_per_launch": 123.0}))
    assert bench.measured_traffic("w") is None


@pytest.mark.parametrize("form,nnz,C,expect_gb", [
    ("svm_dual", 1_950_000_000, 50_000_000, 32.4),         # click-log workload
    ("svm_dual", 1_295_000_000, 350_000, 20.7),            # text SVM
    ("ridge_primal", 1_295_000_000, 16_600_000, 26.2),     # text ridge by columns
    ("ridge_dual", 5_001_930, 100_000, 0.0824),
])
def test_algorithmic_bytes_per_epoch(form, nnz, C, expect_gb):
    # 16 B per stored entry + 24 B per coordinate for the duals, 20 + 20 for the ridge primal
    sys.path.insert(0, ROOT)
    import types

    import bench

    prob = types.SimpleNamespace(form=form, nnz=nnz, C=C)
    got = bench.algorithmic_bytes(prob) / 1e9
    assert abs(got - expect_gb) <= 0.005 * expect_gb, got


def test_default_workload_is_the_largest():
    sys.path.insert(0, ROOT)
    import bench

    src = open(os.path.join(ROOT, "bench.py")).read()
    assert 'default="click_svm"' in src and "click_svm" in bench.WORKLOADS
