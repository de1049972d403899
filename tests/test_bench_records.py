"""The benchmark's kept records (CPU): the decode-attention traffic record
under profiles/ names the kernel sources it was measured on, and bench.py
attaches it only while they are unchanged; this checks that the record kept
with the repository matches the sources as they are, so that a change to the
kernels cannot go out with counters taken on other code."""
import json
import os
import sys
import types

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_traffic_record_matches_kernel_sources():
    for workload, name in bench.TRAFFIC.items():
        path = os.path.join(ROOT, "profiles", name)
        with open(path) as f:
            rec = json.load(f)
        assert rec["kernel_sources_sha256"] == bench.kernel_sources_sha256(), (
            f"{name} was measured on other decode-attention sources: re-take its FETCH_SIZE / WRITE_SIZE "
            "counters on the benchmark's command")
        assert 1.0 <= rec["traffic_over_algorithmic"] < 1.5


def test_traffic_record_is_attached_for_its_workload_only():
    args = types.SimpleNamespace(split=None, traffic_dir=os.path.join(ROOT, "profiles"))
    for workload in bench.TRAFFIC:
        rec = bench.traffic_record(args, types.SimpleNamespace(name=workload))
        assert rec is not None and rec["traffic_over_algorithmic"] >= 1.0
    assert bench.traffic_record(args, types.SimpleNamespace(name="b32-L2048")) is None
    args.split = 512   # another launch configuration than the one measured
    for workload in bench.TRAFFIC:
        assert bench.traffic_record(args, types.SimpleNamespace(name=workload)) is None
