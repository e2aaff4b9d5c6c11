"""Host-side checks of bench.py's bookkeeping (no GPU): recorded HBM traffic
(`traffic_record:` lines of profiles/*_pmc*.md) is used only for the
workload, call and GEMM sources it was measured on, and then lies between the
algorithmic bytes it states and a few times them."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402

KEYS = {"workload", "call", "gemm_source_hash", "traffic_bytes_per_call", "algorithmic_bytes_per_call"}


def test_traffic_records_parse_and_are_plausible():
    recs = bench.traffic_records()
    assert recs, "no PMC traffic record committed"
    for kv in recs:
        assert KEYS <= set(kv), kv
        t, alg = float(kv["traffic_bytes_per_call"]), float(kv["algorithmic_bytes_per_call"])
        assert alg <= t <= 4 * alg, kv
        got = bench.measured_traffic(kv["workload"], kv["call"])
        if kv["gemm_source_hash"] == bench.gemm_source_hash():
            assert got == t
        else:
            assert got is None


def test_traffic_record_ignored_for_other_workloads_and_calls():
    assert bench.measured_traffic("no_such_workload", "expert_ffn_fwd") is None
    for kv in bench.traffic_records():
        assert bench.measured_traffic(kv["workload"], "no_such_call") is None


def test_source_hash_covers_the_gemm_sources():
    assert all(os.path.isfile(os.path.join(ROOT, rel)) for rel in bench.GEMM_SOURCES)
    h = bench.gemm_source_hash()
    assert len(h) == 16 and int(h, 16) >= 0
