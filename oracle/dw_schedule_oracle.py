"""CPU oracle for the weight-gradient computation schedule pass (Sec. 4,
"Weight Gradient Computation Schedule Pass": labelling, Sec. 4.1; greedy
scheduling, Sec. 4.2 and Alg. 1).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this
module: only ``tests/`` use it.  It shares no code with the library's C++
planner.

An instance is a sequence of n instructions (the order is a valid execution
order), each of kind OTHER, A2A (all-to-all) or DW (weight-gradient
computation), with an execution time, and dependency edges (src, dst):
dst consumes an output of src, and src precedes dst in the sequence.

Readings of points the paper leaves open:

* the candidates of an all-to-all are the DW instructions with no directed
  path to or from it (the labelling admits any instruction; only DW ones
  are ever assigned);
* equal |t_u - t_w| in the greedy choice: the lowest instruction index;
* the loop over an all-to-all stops once its unoverlapped time t_u is no
  longer positive or no unused candidate is left (t_u may end negative);
* reordering: the sequence without the assigned DW instructions, each
  assigned one emitted right after its all-to-all, or after its last
  predecessor if that comes later; an instruction that consumes an assigned
  DW instruction not yet emitted pulls it (and what it needs) in first, so
  the result is always a valid execution order.  Several DW instructions
  placed at one point keep their original order.
"""
from __future__ import annotations

import itertools
from typing import Dict, List, Sequence, Tuple

OTHER, A2A, DW = 0, 1, 2


def reachable(n: int, edges: Sequence[Tuple[int, int]]) -> List[set]:
    """reach[i] = every instruction with a directed path from i (breadth-first
    search from every node; Sec. 4.1 names depth- or breadth-first search)."""
    succ = [[] for _ in range(n)]
    for s, d in edges:
        succ[s].append(d)
    out = []
    for i in range(n):
        seen, frontier = set(), [i]
        while frontier:
            nxt = []
            for u in frontier:
                for v in succ[u]:
                    if v not in seen:
                        seen.add(v)
                        nxt.append(v)
            frontier = nxt
        out.append(seen)
    return out


def label(n: int, kinds: Sequence[int], edges) -> Dict[int, List[int]]:
    """W^{I_a} for every all-to-all a (Sec. 4.1): the DW instructions with no
    directed path between them and a, in sequence order."""
    reach = reachable(n, edges)
    W = {}
    for a in range(n):
        if kinds[a] != A2A:
            continue
        W[a] = [j for j in range(n) if j != a and kinds[j] == DW and j not in reach[a] and a not in reach[j]]
    return W


def greedy_assign(kinds: Sequence[int], times: Sequence[float], W: Dict[int, List[int]]) -> Dict[int, int]:
    """Alg. 1's scheduling loop: all-to-alls in sequence order; for each, while
    its unoverlapped time t_u is positive and an unused candidate is left,
    take the candidate whose time is closest to t_u (ties: lowest index),
    subtract its time from t_u and mark it used.  Returns {dw: a2a}."""
    used, asg = set(), {}
    for a in sorted(W):
        t_u = times[a]
        while t_u > 0:
            cand = [j for j in W[a] if j not in used]
            if not cand:
                break
            j_min = min(cand, key=lambda j: (abs(t_u - times[j]), j))
            t_u -= times[j_min]
            used.add(j_min)
            asg[j_min] = a
    return asg


def overlap(kinds, times, asg: Dict[int, int]) -> float:
    """The integer program's objective (Sec. 4.2): sum over all-to-alls of
    min(t_a, total time of the DW instructions assigned to it)."""
    tot = {a: 0.0 for a in range(len(kinds)) if kinds[a] == A2A}
    for j, a in asg.items():
        tot[a] += times[j]
    return sum(min(times[a], s) for a, s in tot.items())


def ip_optimum(kinds, times, W: Dict[int, List[int]]) -> Tuple[float, Dict[int, int]]:
    """The integer program of Sec. 4.2 solved by enumeration (each DW
    instruction: one all-to-all whose candidate set holds it, or none).
    Exponential: small instances only."""
    dws = sorted({j for js in W.values() for j in js})
    opts = [[None] + [a for a in sorted(W) if j in W[a]] for j in dws]
    best, best_asg = -1.0, {}
    for choice in itertools.product(*opts):
        asg = {j: a for j, a in zip(dws, choice) if a is not None}
        v = overlap(kinds, times, asg)
        if v > best + 1e-12:
            best, best_asg = v, asg
    return best, best_asg


def reorder(n: int, kinds, edges, asg: Dict[int, int]) -> List[int]:
    """ReorderInstrs of Alg. 1: every assigned DW instruction is placed right
    after its all-to-all (or after its last predecessor, if later)."""
    pred = [[] for _ in range(n)]
    for s, d in edges:
        pred[d].append(s)
    emitted, out = set(), []

    def emit(i):
        out.append(i)
        emitted.add(i)

    def pull(i):
        # emit the not-yet-emitted assigned DW instructions i needs, then i
        for p in sorted(pred[i]):
            if p not in emitted:
                pull(p)
        if i not in emitted:
            emit(i)

    def flush():
        # assigned DW instructions whose all-to-all and predecessors are out
        changed = True
        while changed:
            changed = False
            for j in sorted(asg):
                if j not in emitted and asg[j] in emitted and all(p in emitted for p in pred[j]):
                    emit(j)
                    changed = True

    for i in range(n):
        if i in asg or i in emitted:
            continue
        pull(i)
        flush()
    for j in sorted(asg):          # (every assigned instruction is out by now)
        if j not in emitted:
            pull(j)
    return out


def schedule(n: int, kinds, times, edges):
    """Alg. 1 end to end: (assignment {dw: a2a}, new sequence, overlap)."""
    W = label(n, kinds, edges)
    asg = greedy_assign(kinds, times, W)
    return asg, reorder(n, kinds, edges, asg), overlap(kinds, times, asg)
