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
