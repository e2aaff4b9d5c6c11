"""The library's weight-gradient schedule planner (moe_dw_schedule, host C++)
against the oracle of Sec. 4 / Alg. 1: identical assignments and orders on
random instances, argument validation, and the MoE-block backward instance
(two blocks under expert parallelism, measured kernel times, all-to-alls
costed by an xGMI model) with the greedy's gap to the integer program."""
import numpy as np
import pytest

from oracle import dw_schedule_oracle as D

L = pytest.importorskip("paper_2404_19429_amd.lancet_moe", reason="library not built")

A2A, DW, OTHER = D.A2A, D.DW, D.OTHER


def _random_instance(rng, n, p_edge):
    kinds = [int(rng.choice([OTHER, A2A, DW], p=[0.45, 0.2, 0.35])) for _ in range(n)]
    edges = [(i, j) for i in range(n) for j in range(i + 1, n) if rng.random() < p_edge]
    # integer-valued and fractional times, with repeats (ties in the greedy choice)
    times = [float(rng.integers(0, 12)) if rng.random() < 0.5 else float(rng.random() * 10) for _ in range(n)]
    return kinds, times, edges


@pytest.mark.parametrize("seed", range(40))
def test_planner_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 60)) if seed % 4 else int(rng.integers(100, 260))
    kinds, times, edges = _random_instance(rng, n, p_edge=float(rng.choice([0.02, 0.08, 0.2])))
    asg, order, ov = D.schedule(n, kinds, times, edges)
    a, o, v = L.moe_dw_schedule(kinds, times, edges)
    want = np.full(n, -1, np.int32)
    for j, x in asg.items():
        want[j] = x
    np.testing.assert_array_equal(a, want)
    np.testing.assert_array_equal(o, order)
    assert v == pytest.approx(ov, rel=1e-12, abs=1e-12)


def test_planner_empty_and_no_edges():
    a, o, v = L.moe_dw_schedule([], [], [])
    assert a.size == 0 and o.size == 0 and v == 0.0
    a, o, v = L.moe_dw_schedule([A2A, DW, DW], [5.0, 2.0, 2.0], [])
    assert list(a) == [-1, 0, 0] and list(o) == [0, 1, 2] and v == 4.0


@pytest.mark.parametrize("kinds,times,edges,msg", [
    ([0, 3], [1.0, 1.0], [], "kind"),
    ([0, 1], [1.0, -1.0], [], "time"),
    ([0, 1], [1.0, float("nan")], [], "time"),
    ([0, 1], [1.0, 1.0], [(1, 0)], "edge"),
    ([0, 1], [1.0, 1.0], [(0, 2)], "edge"),
    ([0, 1], [1.0, 1.0], [(1, 1)], "edge"),
])
def test_planner_rejects_invalid(kinds, times, edges, msg):
    with pytest.raises(L.MoeError) as e:
        L.moe_dw_schedule(kinds, times, edges)
    assert e.value.status == L.MOE_EINVAL and msg in str(e.value)


# --------------------------------------------------- the MoE-block backward
# Per-operation times (µs) of the pre-LN MoE block (8 x 2048 tokens, d_model
# 2048, 16 heads, 16 experts, d_ff 8192, top-2) from the committed kernel trace
# of this library on one MI355X; the two all-to-alls of each block are costed
# by an xGMI model: with 8 GPUs (2 experts each), a GPU sends 7/8 of its kept
# rows (16384 tokens x 2 choices x 2048 x 2 bytes) in 7 parallel point-to-point
# streams of 153 GB/s: 117 MB / 7 / 153 GB/s = 110 µs.
BLOCK_OPS = [   # (name, kind, µs, inputs among the block's earlier ops; "in" = the block's incoming gradient)
    ("combine_bwd", OTHER, 74.0, ["in"]),
    ("a2a_dO", A2A, 110.0, ["combine_bwd"]),
    ("experts_dA_dH", OTHER, 1252.0, ["a2a_dO"]),
    ("experts_dX", OTHER, 981.0, ["experts_dA_dH"]),
    ("dW2", DW, 1241.0, ["a2a_dO"]),
    ("dW1", DW, 1241.0, ["experts_dA_dH"]),
    ("a2a_dX", A2A, 110.0, ["experts_dX"]),
    ("dispatch_bwd", OTHER, 90.0, ["a2a_dX", "combine_bwd"]),
    ("dWg", DW, 50.0, ["combine_bwd"]),
    ("ln2_bwd", OTHER, 196.0, ["dispatch_bwd"]),
    ("dln2", DW, 154.0, ["dispatch_bwd"]),
    ("outproj_dX", OTHER, 243.0, ["ln2_bwd"]),
    ("dWo", DW, 612.0, ["ln2_bwd"]),
    ("attn_bwd", OTHER, 1947.0, ["outproj_dX"]),
    ("qkv_dX", OTHER, 767.0, ["attn_bwd"]),
    ("dWqkv", DW, 612.0, ["attn_bwd"]),
    ("ln1_bwd", OTHER, 196.0, ["qkv_dX"]),
    ("dln1", DW, 154.0, ["qkv_dX"]),
]


def block_backward_instance(n_blocks):
    """The backward of n_blocks stacked MoE blocks, top block first: the
    incoming gradient of block b is the LN1 backward output of block b - 1."""
    kinds, times, edges, names = [], [], [], []
    prev_out = None
    for b in range(n_blocks):
        base = len(kinds)
        ix = {name: base + i for i, (name, _, _, _) in enumerate(BLOCK_OPS)}
        for name, kind, t, ins in BLOCK_OPS:
            kinds.append(kind)
            times.append(t)
            names.append(f"{name}[{b}]")
            for s in ins:
                if s == "in":
                    if prev_out is not None:
                        edges.append((prev_out, ix[name]))
                else:
                    edges.append((ix[s], ix[name]))
        prev_out = ix["ln1_bwd"]
        # dx of the residual stream also flows from ln2_bwd and dispatch_bwd (pre-LN residuals)
        edges.append((ix["dispatch_bwd"], ix["ln1_bwd"]))
    return kinds, times, sorted(set(edges)), names


def test_block_backward_schedule():
    kinds, times, edges, names = block_backward_instance(2)
    n = len(kinds)
    asg, order, ov = D.schedule(n, kinds, times, edges)
    a, o, v = L.moe_dw_schedule(kinds, times, edges)
    np.testing.assert_array_equal(o, order)
    assert v == pytest.approx(ov)
    W = D.label(n, kinds, edges)
    best, _ = D.ip_optimum(kinds, times, W)
    a2a_total = sum(t for t, k in zip(times, kinds) if k == A2A)
    print(f"\n[dw schedule] 2 blocks: all-to-all time {a2a_total:.0f} us, greedy overlap {ov:.0f} us, "
          f"integer-program optimum {best:.0f} us; assigned: "
          + ", ".join(f"{names[j]}->{names[x]}" for j, x in sorted(asg.items())))
    assert ov <= best + 1e-9
    # every all-to-all of the lower block has weight gradients of the upper block to hide behind
    lower = [i for i in range(len(BLOCK_OPS), n) if kinds[i] == A2A]
    assert all(any(x == i for x in asg.values()) for i in lower)


# ------------------------------------------------ partition-range planner
from oracle import pipeline_oracle as PO  # noqa: E402


@pytest.mark.parametrize("seed", range(30))
def test_pipeline_planner_matches_oracle(seed):
    rng = np.random.default_rng(500 + seed)
    N = int(rng.integers(1, 40))
    K = int(rng.integers(1, 9))
    kinds = [int(rng.integers(0, 2)) for _ in range(N)]
    times = []
    for _ in range(N):
        t1 = float(rng.integers(1, 50)) if rng.random() < 0.5 else float(rng.random() * 40)
        row = [t1] + [t1 / k + float(rng.random()) for k in range(2, K + 1)]
        if rng.random() < 0.1 and K > 1:
            row[int(rng.integers(1, K))] = float("inf")
        times.append(row)
    join = [0.0] + [float(rng.random() * 3) for _ in range(K - 1)]
    G = int(rng.integers(0, N + 1))
    T, segs = PO.plan(kinds, times, join, G)
    t2, s2 = L.moe_pipeline_plan(kinds, times, join, G)
    assert t2 == T and s2 == segs
    i, n = sorted(int(v) for v in rng.integers(1, N + 1, 2))
    for k in range(1, K + 1):
        assert L.moe_pipeline_range_cost(kinds, times, join, i, n, k) == PO.range_cost(kinds, times, join, i, n, k)


def test_pipeline_planner_rejects_invalid():
    for kinds, times, join in [([2], [[1.0]], [0.0]), ([0], [[float("nan")]], [0.0]), ([0], [[float("inf")]], [0.0]),
                               ([0], [[1.0, 1.0]], [0.0, -1.0])]:
        with pytest.raises(L.MoeError):
            L.moe_pipeline_plan(kinds, times, join)


def test_planner_large_instance_is_fast():
    import time
    rng = np.random.default_rng(7)
    n = 6000
    kinds = [int(k) for k in rng.choice([OTHER, A2A, DW], size=n, p=[0.5, 0.1, 0.4])]
    times = [float(t) for t in rng.integers(1, 20, n)]
    edges = sorted({(int(j), int(i)) for i in range(1, n) for j in rng.integers(max(0, i - 50), i, 3)})
    t0 = time.perf_counter()
    a, o, v = L.moe_dw_schedule(kinds, times, edges)
    assert time.perf_counter() - t0 < 5.0
    pos = np.empty(n, np.int64)
    pos[o] = np.arange(n)
    assert all(pos[s] < pos[d] for s, d in edges)          # a valid execution order
    assert sorted(o.tolist()) == list(range(n))


# --------------------------------------------- the library's block schedule
# moe_block_dw_schedule's instance, written here from its description in
# include/lancet_moe.h: instruction i runs block op OPS[i] (None = an
# all-to-all), in reverse-mode emission order.
_BOP = {n: i for i, n in enumerate(L.BLOCK_OPS)}
_LIB_OPS = ["combine_bwd", None, "expert_dx", "dw_expert", None, "dispatch_bwd", "dwg", "ln2_bwd", "dln2", "dwo",
            "dattn", "attn_bwd", "dwqkv", "da", "ln1_bwd", "dln1"]
_LIB_EDGES = [(0, 1), (1, 2), (1, 3), (2, 3), (2, 4), (4, 5), (0, 5), (0, 6), (5, 7), (7, 8), (7, 9), (7, 10),
              (10, 11), (11, 12), (11, 13), (13, 14), (14, 15)]


def _lib_instance(op_ms, a2a_ms):
    kinds = [A2A if o is None else (DW if _BOP[o] >= L.MOE_BOP_DW_EXPERT else OTHER) for o in _LIB_OPS]
    times = [a2a_ms if o is None else float(op_ms[_BOP[o]]) for o in _LIB_OPS]
    return kinds, times


@pytest.mark.parametrize("seed", range(12))
def test_block_schedule_matches_oracle(seed):
    rng = np.random.default_rng(100 + seed)
    op_ms = rng.random(len(L.BLOCK_OPS)) * rng.choice([0.05, 1.0, 3.0])
    a2a_ms = float(rng.choice([0.0, 0.02, 0.11, 1.0, 9.4]))
    order, assign, ov = L.moe_block_dw_schedule(op_ms, a2a_ms)
    kinds, times = _lib_instance(op_ms, a2a_ms)
    asg, seq, ov_o = D.schedule(16, kinds, times, _LIB_EDGES)
    want_assign = np.full(16, -1, np.int32)
    for j, a in asg.items():
        want_assign[j] = a
    np.testing.assert_array_equal(assign, want_assign)
    np.testing.assert_array_equal(order, [_BOP[_LIB_OPS[i]] for i in seq if kinds[i] == DW])
    assert ov == pytest.approx(ov_o, rel=1e-12, abs=1e-15)
    assert sorted(order.tolist()) == list(range(L.MOE_BOP_DW_EXPERT, L.MOE_BOP_DW_EXPERT + 6))


def test_block_schedule_moves_the_gate_gradient_under_the_first_all_to_all():
    """With all-to-all time, dWg (which reads only the gate's gradient) is the
    one candidate of the exchange of dO and goes right after it; the expert dW
    overlaps the exchange of dXe; without all-to-all time the emission order
    (the default dw_order) stays."""
    op_ms = np.array([0.07, 2.2, 0.09, 0.2, 0.24, 1.9, 0.77, 0.2, 2.4, 0.05, 0.15, 0.6, 0.6, 0.15])
    order, assign, ov = L.moe_block_dw_schedule(op_ms, 0.11)
    assert order.tolist() == [L.MOE_BOP_DW_EXPERT + 1, L.MOE_BOP_DW_EXPERT, 10, 11, 12, 13]
    assert assign[6] == 1 and assign[3] == 4
    assert ov == pytest.approx(0.05 + 0.11)
    order0, assign0, ov0 = L.moe_block_dw_schedule(op_ms, 0.0)
    assert order0.tolist() == [8, 9, 10, 11, 12, 13] and (assign0 == -1).all() and ov0 == 0.0


def test_block_schedule_validation():
    with pytest.raises(L.MoeError):
        L.moe_block_dw_schedule(np.full(len(L.BLOCK_OPS), -1.0), 0.1)
    with pytest.raises(L.MoeError):
        L.moe_block_dw_schedule(np.ones(len(L.BLOCK_OPS)), float("nan"))
