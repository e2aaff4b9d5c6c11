"""Pins of the weight-gradient schedule oracle (Sec. 4, Alg. 1) against
facts fixed independently of its code: hand-worked instances, the integer
program of Sec. 4.2 solved by enumeration, path sets from a boolean
transitive closure, and the validity of every produced order."""
import numpy as np
import pytest

from oracle import dw_schedule_oracle as D

A2A, DW, OTHER = D.A2A, D.DW, D.OTHER


def _closure(n, edges):
    """Boolean transitive closure by repeated squaring (not a graph search)."""
    R = np.zeros((n, n), bool)
    for s, d in edges:
        R[s, d] = True
    for _ in range(max(1, int(np.ceil(np.log2(max(n, 2)))) + 1)):
        R = R | ((R.astype(np.int64) @ R.astype(np.int64)) > 0)
    return R


def _random_dag(rng, n, p_edge=0.15, p_a2a=0.2, p_dw=0.35):
    kinds = [int(rng.choice([OTHER, A2A, DW], p=[1 - p_a2a - p_dw, p_a2a, p_dw])) for _ in range(n)]
    edges = [(i, j) for i in range(n) for j in range(i + 1, n) if rng.random() < p_edge]
    times = [float(rng.integers(1, 20)) for _ in range(n)]
    return kinds, times, edges


def _valid_order(n, order, edges):
    pos = {v: i for i, v in enumerate(order)}
    return sorted(order) == list(range(n)) and all(pos[s] < pos[d] for s, d in edges)


def test_hand_worked_single_all_to_all():
    # one all-to-all of 10 after a producer, three independent DW ops of 4, 7, 3
    kinds = [OTHER, A2A, DW, DW, DW]
    times = [1.0, 10.0, 4.0, 7.0, 3.0]
    edges = [(0, 1)]
    asg, order, ov = D.schedule(5, kinds, times, edges)
    # t_u = 10: closest is 7 (|3|); t_u = 3: closest is 3 (|0|); t_u = 0: stop
    assert asg == {3: 1, 4: 1}
    assert ov == 10.0
    assert order == [0, 1, 3, 4, 2]
    assert D.ip_optimum(kinds, times, D.label(5, kinds, edges))[0] == 10.0


def test_greedy_is_a_heuristic_gap_instance():
    # a2a 0 (5) may take A (5) or B (3); a2a 1 (5) only A: the greedy gives A
    # to the first all-to-all (exact fit) and leaves the second bare
    kinds = [A2A, A2A, DW, DW]            # 2 = A, 3 = B
    times = [5.0, 5.0, 5.0, 3.0]
    edges = [(3, 1)]                       # B feeds a2a 1, so B is no candidate of it
    W = D.label(4, kinds, edges)
    assert W == {0: [2, 3], 1: [2]}
    asg = D.greedy_assign(kinds, times, W)
    assert asg == {2: 0}
    assert D.overlap(kinds, times, asg) == 5.0
    best, best_asg = D.ip_optimum(kinds, times, W)
    assert best == 8.0 and best_asg == {2: 1, 3: 0}


def test_all_candidates_fit():
    # every DW fits inside the one all-to-all: all assigned, overlap = their sum
    kinds = [A2A] + [DW] * 5
    times = [100.0, 10.0, 20.0, 5.0, 30.0, 1.0]
    asg, order, ov = D.schedule(6, kinds, times, [])
    assert set(asg) == {1, 2, 3, 4, 5} and ov == 66.0
    assert D.ip_optimum(kinds, times, D.label(6, kinds, []))[0] == 66.0


@pytest.mark.parametrize("seed", range(12))
def test_labelling_matches_transitive_closure(seed):
    rng = np.random.default_rng(seed)
    n = 14
    kinds, times, edges = _random_dag(rng, n)
    R = _closure(n, edges)
    W = D.label(n, kinds, edges)
    for a in range(n):
        if kinds[a] != A2A:
            assert a not in W
            continue
        want = [j for j in range(n) if kinds[j] == DW and not R[a, j] and not R[j, a]]
        assert W[a] == want


@pytest.mark.parametrize("seed", range(25))
def test_schedule_constraints_bound_and_order(seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(6, 13))
    kinds, times, edges = _random_dag(rng, n)
    W = D.label(n, kinds, edges)
    asg, order, ov = D.schedule(n, kinds, times, edges)
    for j, a in asg.items():                      # constraints (1) and (2)
        assert kinds[j] == DW and kinds[a] == A2A and j in W[a]
    assert len(set(asg)) == len(asg)
    if sum(1 for k in kinds if k == DW) <= 8:
        assert ov <= D.ip_optimum(kinds, times, W)[0] + 1e-9
    assert _valid_order(n, order, edges)
    pos = {v: i for i, v in enumerate(order)}
    pred = {d: [s for s, dd in edges if dd == d] for d in range(n)}
    for j, a in asg.items():                      # right after its all-to-all or its last predecessor
        anchor = max([pos[a]] + [pos[p] for p in pred[j]])
        between = order[anchor + 1:pos[j]]
        assert all(v in asg for v in between), (j, a, between)


def test_equal_times_take_the_lower_index():
    # reading: equal |t_u - t_w| goes to the lower instruction index
    kinds = [A2A, DW, DW, DW]
    times = [3.0, 3.0, 3.0, 1.0]
    asg = D.greedy_assign(kinds, times, D.label(4, kinds, []))
    assert asg == {1: 0}
