"""Pins of the pipeline-cost / range-choice oracle (Sec. 5.1, 5.3) against
facts fixed independently of its code: the unsplit sum, the closed form of
a two-stage pipeline, a hand-worked three-stage timeline, and the dynamic
program against enumeration of every segmentation."""
import itertools
import math

import numpy as np
import pytest

from oracle import pipeline_oracle as P

COMP, COMM = P.COMP, P.COMM


def test_unsplit_range_is_the_sum():
    kinds = [COMP, COMM, COMP, COMM]
    times = [[3.0, 2.0], [1.0, 0.6], [2.0, 1.1], [4.0, 2.2]]
    assert P.range_cost(kinds, times, [0.0, 0.5], 1, 4, 1) == 10.0


@pytest.mark.parametrize("a,b,k", [(4.0, 3.0, 2), (3.0, 4.0, 2), (2.0, 2.0, 4), (1.0, 5.0, 8), (5.0, 1.0, 3)])
def test_two_stage_pipeline_closed_form(a, b, k):
    # compute then communication, k equal parts: a + b + (k - 1) max(a, b)
    assert P.simulate([(COMP, a), (COMM, b)], k) == a + b + (k - 1) * max(a, b)


def test_three_stage_hand_worked():
    # a = 4 (compute), b = 3 (communication), c = 2 (compute), two partitions:
    # compute p0 [0,4] p1 [4,8]; comm p0 [4,7] p1 [8,11];
    # second compute stage p0 [8,10] (after p1's first stage), p1 [11,13]
    assert P.simulate([(COMP, 4.0), (COMM, 3.0), (COMP, 2.0)], 2) == 13.0
    # merged runs: two compute instructions in a row form one stage
    assert P.stages([COMP, COMP, COMM, COMP], [1.0, 3.0, 3.0, 2.0]) == [(COMP, 4.0), (COMM, 3.0), (COMP, 2.0)]


def test_unsplittable_instruction_blocks_k():
    kinds = [COMP, COMM]
    times = [[2.0, math.inf], [2.0, 1.0]]
    assert P.range_cost(kinds, times, [0.0, 0.0], 1, 2, 2) == math.inf
    T, segs = P.plan(kinds, times, [0.0, 0.0])
    assert T == 4.0 and segs == [(1, 2, 1)]


def _brute(kinds, times, join, G):
    N, K = len(kinds), len(join)
    best = math.inf
    for cuts in itertools.product([0, 1], repeat=N - 1):
        bounds, s = [], 1
        for j, c in enumerate(cuts, start=1):
            if c:
                bounds.append((s, j))
                s = j + 1
        bounds.append((s, N))
        if any(n - i + 1 > G for i, n in bounds):
            continue
        tot = sum(min(P.range_cost(kinds, times, join, i, n, k) for k in range(1, K + 1)) for i, n in bounds)
        best = min(best, tot)
    return best


@pytest.mark.parametrize("seed", range(20))
def test_dp_equals_enumeration(seed):
    rng = np.random.default_rng(seed)
    N = int(rng.integers(1, 8))
    K = int(rng.integers(1, 4))
    kinds = [int(rng.integers(0, 2)) for _ in range(N)]
    times = []
    for _ in range(N):
        t1 = float(rng.integers(1, 10))
        row = [t1] + [t1 / k + float(rng.random()) for k in range(2, K + 1)]
        if rng.random() < 0.15 and K > 1:
            row[-1] = math.inf
        times.append(row)
    join = [0.0] + [float(rng.random() * 2) for _ in range(K - 1)]
    G = int(rng.integers(1, N + 1))
    T, segs = P.plan(kinds, times, join, G)
    assert T == pytest.approx(_brute(kinds, times, join, G))
    # the segments tile 1..N and reproduce T
    assert segs[0][0] == 1 and segs[-1][1] == N
    assert all(a[1] + 1 == b[0] for a, b in zip(segs, segs[1:]))
    assert sum(P.range_cost(kinds, times, join, i, n, k) for i, n, k in segs) == pytest.approx(T)


def test_split_range_pays_its_join_cost():
    # two stages a = 4 (compute), b = 3 (communication), split 2 ways, join 1.5:
    # a + b + (k - 1) max(a, b) + join = 4 + 3 + 4 + 1.5
    kinds = [COMP, COMM]
    times = [[8.0, 4.0], [6.0, 3.0]]
    assert P.range_cost(kinds, times, [0.0, 1.5], 1, 2, 2) == 12.5
    assert P.range_cost(kinds, times, [0.0, 1.5], 1, 2, 1) == 14.0   # unsplit: the sum, no join
