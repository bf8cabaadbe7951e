"""Host logic of bench.py (no GPU): the busy-time union of scorer intervals,
the traffic records' source check, and the one-GPU contract of the command
line."""

import json
import os
import subprocess
import sys

import numpy as np

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_union_of_intervals():
    assert bench.union_ms(np.zeros((0, 2))) == 0.0
    assert bench.union_ms(np.array([[0.0, 1.0]])) == 1.0
    # overlapping, nested, touching and disjoint intervals, in any order
    iv = np.array([[5.0, 6.0], [0.0, 2.0], [1.0, 3.0], [1.5, 1.7], [3.0, 4.0], [10.0, 10.5]])
    assert abs(bench.union_ms(iv) - (4.0 + 1.0 + 0.5)) < 1e-12


def test_traffic_records_match_their_sources():
    """Every committed traffic record names the scorer sources of its model
    and is reported only while their hash matches; a record whose hash is off
    is reported as unknown."""
    recs = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    model_of = {"score:C2": 1, "score:C5": 2}
    for key, rec in recs.items():
        m = model_of[key]
        assert rec["kernel_sources"] == bench.SCORER_SOURCES[m]
        assert rec["bytes_per_launch"] == round(rec["fetch_kib_raw"] * 1024 * rec["fetch_scale"]
                                                + rec["write_kib_raw"] * 1024 * rec["write_scale"])
        if rec["sources_sha256"] == bench.sources_sha256(rec["kernel_sources"]):
            assert bench.traffic_for(m, key) == (rec["bytes_per_launch"], rec["bytes_per_launch_by_request_size"])
    # a stale hash reads as unknown
    orig = bench.sources_sha256
    try:
        bench.sources_sha256 = lambda files: "0" * 64
        assert bench.traffic_for(1, "score:C2") == (None, None)
    finally:
        bench.sources_sha256 = orig
    assert bench.traffic_for(1, "score:no-such-workload") == (None, None)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, cwd=ROOT, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""
