"""Host-side checks of bench.py: the one-GPU guard, the library hash that
keys recorded traffic, and the recorded-traffic lookup (no GPU needed)."""
import json
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
    assert "one GPU" in r.stderr


def test_library_hash_is_stable_and_keys_the_traffic_record():
    lib = os.path.join(ROOT, "paper_2609_11562_amd", "libentwine.so")
    if not os.path.exists(lib):
        pytest.skip("library not built")
    h = bench.library_hash(ROOT)
    assert h == bench.library_hash(ROOT) and len(h) == 16
    rec = json.load(open(os.path.join(ROOT, "paper_2609_11562_amd", "traffic.json")))
    entry = rec["llama7b_mlp_down_tp8"]
    cfg = entry["config"]
    got = bench.measured_traffic(ROOT, "llama7b_mlp_down_tp8", entry["kernel"], cfg)
    if entry["library_sha256_16"] == h:
        assert got is not None
        assert got["bytes"] == pytest.approx(entry["fetch_kib"] * 1024 * entry["fetch_scale"]
                                             + entry["write_kib"] * 1024 * entry["write_scale"], rel=1e-6)
    else:
        assert got is None
    # any other configuration or kernel has no recorded traffic
    assert bench.measured_traffic(ROOT, "llama7b_mlp_down_tp8", entry["kernel"], dict(cfg, reduce_wgs=16)) is None
    assert bench.measured_traffic(ROOT, "llama7b_mlp_down_tp8", "gemm_producer", cfg) is None
