"""bench.py's host-side parts on a host without a GPU: the one-GPU contract and the
helpers that price the dominant kernel."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


@pytest.mark.parametrize("L,W", [(8, 501), (384, 6001), (2000, 601)])
def test_write_bytes_per_fill(L, W):
    # the finalize writes Opt for every span and ap for every span not ending at L-1
    spans = L * (L + 1) // 2
    assert bench.write_bytes_per_fill("k_finalize", L, W) == (spans + spans - L) * W * 4
    # the band product writes one partial row per span of every 32-span band after the first
    cells = sum(L - d for d in range(32, L))
    assert bench.write_bytes_per_fill("k_product", L, W) == cells * W * 4
    assert bench.write_bytes_per_fill("k_mid", L, W) is None


def test_measured_traffic_follows_the_kernel_source(tmp_path, monkeypatch):
    import json
    prof = {"kernels_source": "k.hip", "kernels_source_sha256": "", "kernels": {
        "k_product": {"hbm_bytes_per_dispatch": 123.0}}}
    (tmp_path / "k.hip").write_bytes(b"source")
    import hashlib
    prof["kernels_source_sha256"] = hashlib.sha256(b"source").hexdigest()
    (tmp_path / "profiles").mkdir()
    (tmp_path / "profiles" / "hbm_traffic_w.json").write_text(json.dumps(prof))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic("w", "k_product") == (123.0, None)
    assert bench.measured_traffic("w", "k_mid") == (None, None)
    assert bench.measured_traffic("other", "k_product") == (None, None)
    (tmp_path / "k.hip").write_bytes(b"changed source")
    assert bench.measured_traffic("w", "k_product") == (None, None)
