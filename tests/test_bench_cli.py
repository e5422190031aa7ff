"""The benchmark's command-line contract, checked without a GPU: more than one
GPU is refused with a message, and the traffic summary is rebuilt from the
committed counter summary format."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr and r.stdout == ""


def test_committed_traffic_summary_matches_the_kernel_sources():
    sys.path.insert(0, ROOT)
    import bench
    with open(os.path.join(ROOT, "profiles", "traffic.json")) as f:
        t = json.load(f)
    if t["source_hash"] != bench.kernel_source_hash():
        pytest.skip("kernel sources changed since the counters were taken: bench.py reports traffic null")
    # the two passes of the benchmark's layer (projected pass 1, slice-state pass 2)
    for k in ("k_slice_accumulate_pcp", "k_deslice_sf"):
        assert t["kernels"][k]["points"] == 1_000_000
        assert bench.measured_traffic(k, 1_000_000) == t["kernels"][k]["hbm_bytes_per_launch"]
