"""Host-side checks of bench.py's bookkeeping (no GPU): recorded HBM traffic
(profiles/*_pmc_traffic.md) is used only for the workload, call and GEMM
sources it was measured on, and then lies between the algorithmic bytes it
states and a few times them."""
import glob
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402

KEYS = {"workload", "call", "gemm_source_hash", "traffic_bytes_per_call", "algorithmic_bytes_per_call"}


def _records():
    out = []
    for path in sorted(glob.glob(os.path.join(bench.PROFILES, "*_pmc_traffic.md"))):
        kv = {}
        for line in open(path).read().splitlines():
            if ":" in line and line.split(":", 1)[0].strip() in KEYS:
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
        out.append((path, kv))
    return out


def test_traffic_records_parse_and_are_plausible():
    recs = _records()
    assert recs, "no PMC traffic summary committed"
    for path, kv in recs:
        assert KEYS <= set(kv), (path, kv)
        t, alg = float(kv["traffic_bytes_per_call"]), float(kv["algorithmic_bytes_per_call"])
        assert alg <= t <= 3 * alg, path
        got = bench.measured_traffic(kv["workload"], kv["call"])
        if kv["gemm_source_hash"] == bench.gemm_source_hash():
            assert got == t
        else:
            assert got is None


def test_traffic_record_ignored_for_other_workloads_and_calls():
    assert bench.measured_traffic("no_such_workload", "expert_ffn_fwd") is None
    for _, kv in _records():
        assert bench.measured_traffic(kv["workload"], "no_such_call") is None


def test_source_hash_covers_the_gemm_sources():
    assert all(os.path.isfile(os.path.join(ROOT, rel)) for rel in bench.GEMM_SOURCES)
    h = bench.gemm_source_hash()
    assert len(h) == 16 and int(h, 16) >= 0
