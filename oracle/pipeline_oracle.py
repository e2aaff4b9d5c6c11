"""CPU oracle for the operator-partition pass's cost model and range choice
(Sec. 5: partition range selection by dynamic programming, Sec. 5.1; the
pipeline scheduler's timeline simulation, Sec. 5.3).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this
module: only ``tests/`` use it.  It shares no code with the library's C++
planner.

An instance is a forward instruction sequence of N instructions, each COMP
(computation) or COMM (communication: the all-to-alls, or on one GPU the
dispatch/combine stream), with its execution time when the range holding it
is split into k parts, times[i][k - 1] for k = 1..K (one part's time; inf =
the instruction cannot be split k ways), and the cost of splitting a range's
inputs and joining its outputs, join[k - 1] (0 for k = 1).

Readings of points the paper leaves open:

* a stage is a maximal run of consecutive instructions of one kind in the
  range; a partition's stage depends on the same partition's previous stage
  only (partitions are independent of each other);
* the scheduled order of each kind is stage by stage, partition index within
  a stage (the schedule "by stages" of the paper's figure);
* P(i, n, k) = the simulated end time of the last stage plus join[k - 1];
  for k = 1 the range runs unsplit: the sum of its times;
* T(0) = 0 and T(n) = min over 0 <= i < n of T(i) + min over k of
  P(i + 1, n, k), ranges of at most G instructions; ties take the smaller i,
  then the smaller k.
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple

COMP, COMM = 0, 1
INF = math.inf


def stages(kinds: Sequence[int], times_k: Sequence[float]) -> List[Tuple[int, float]]:
    """Maximal runs of one kind: (kind, summed time of one partition)."""
    out: List[Tuple[int, float]] = []
    for kd, t in zip(kinds, times_k):
        if out and out[-1][0] == kd:
            out[-1] = (kd, out[-1][1] + t)
        else:
            out.append((kd, t))
    return out


def simulate(st: List[Tuple[int, float]], k: int) -> float:
    """Timeline of k partitions of the stages (Sec. 5.3): each stage of
    partition p starts at the later of (i) the end of p's previous stage and
    (ii) the end of the previous instruction of its kind in the scheduled
    order (stage by stage, partitions in index order).  Returns the end time
    of the last instruction."""
    end_prev_stage = [0.0] * k          # per partition: end of its latest stage
    free = {COMP: 0.0, COMM: 0.0}       # end of the last scheduled instruction of each kind
    last = 0.0
    for kd, t in st:
        for p in range(k):
            s = max(end_prev_stage[p], free[kd])
            e = s + t
            end_prev_stage[p] = e
            free[kd] = e
            last = max(last, e)
    return last


def range_cost(kinds, times, join, i: int, n: int, k: int) -> float:
    """P(i, n, k) for instructions i..n (1-based, inclusive)."""
    tk = [times[j][k - 1] for j in range(i - 1, n)]
    if any(math.isinf(t) for t in tk):
        return INF
    if k == 1:
        return float(sum(tk))
    return simulate(stages(kinds[i - 1:n], tk), k) + join[k - 1]


def plan(kinds, times, join, G: int = 0):
    """Sec. 5.1's dynamic program.  Returns (T(N), segments [(i, n, k)] in order)."""
    N = len(kinds)
    K = len(join)
    G = N if G <= 0 else G
    T = [0.0] + [INF] * N
    arg = [None] * (N + 1)
    for n in range(1, N + 1):
        for i in range(max(1, n - G + 1), n + 1):       # range i..n, preceded by T(i - 1)
            for k in range(1, K + 1):
                c = T[i - 1] + range_cost(kinds, times, join, i, n, k)
                if c < T[n]:
                    T[n], arg[n] = c, (i, k)
    segs, n = [], N
    while n > 0:
        i, k = arg[n]
        segs.append((i, n, k))
        n = i - 1
    return T[N], segs[::-1]
