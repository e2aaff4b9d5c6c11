"""Host-side checks of bench.py's bookkeeping (no GPU): the recorded HBM
traffic of the expert FFN forward is only used for the GEMM sources it was
measured on, and then lies between the algorithmic bytes and a few times them."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402

WORKLOAD = "layer_bf16_T8192_d1024_f4096_E16"


def _algorithmic_bytes():
    # FWD1 reads X and W1 and writes H and act(H); FWD2 reads act(H) and W2 and writes O (bf16).
    n, d, f, e = 16384, 1024, 4096, 16
    return ((n * d + e * f * d) + 2 * n * f + (n * f + e * d * f) + n * d) * 2


def test_traffic_record_parses_and_is_plausible():
    text = open(bench.TRAFFIC_FILE).read()
    keys = {line.split(":", 1)[0].strip() for line in text.splitlines() if ":" in line}
    assert {"workload", "gemm_source_hash", "traffic_bytes_per_call"} <= keys
    t = bench.measured_traffic(WORKLOAD)
    if t is not None:   # recorded for the current sources
        alg = _algorithmic_bytes()
        assert alg <= t <= 3 * alg


def test_traffic_record_ignored_for_other_workloads():
    assert bench.measured_traffic("layer_bf16_T16384_d2048_f8192_E8") is None


def test_source_hash_covers_the_gemm_sources():
    assert all(os.path.isfile(os.path.join(ROOT, rel)) for rel in bench.GEMM_SOURCES)
    h = bench.gemm_source_hash()
    assert len(h) == 16 and int(h, 16) >= 0
