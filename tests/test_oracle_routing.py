"""Pins for the oracle's gate, capacity rule and dispatch (CPU only).

Each test checks the oracle against something other than itself: a different
algorithm (repeated argmax instead of a sort, per-expert sorting instead of a
sequential walk), closed forms, the paper's worked example, or invariants.
"""
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import moe_oracle as O
from synth import routing_logits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------------- capacity
@pytest.mark.parametrize("T,E,k,num,den,expect", [
    (256, 4, 1, 5, 4, 80),        # tiny fp32 layer
    (8192, 16, 2, 5, 4, 1280),
    (16384, 8, 2, 5, 4, 5120),
    (32768, 64, 2, 2, 1, 2048),
    (16384, 16, 2, 5, 4, 2560),   # block MoE layer (unchunked token count)
    (10, 3, 1, 1, 1, 4),          # ceil(10/3)
    (0, 4, 2, 5, 4, 0),
])
def test_capacity_values(T, E, k, num, den, expect):
    assert O.capacity(T, E, k, num, den) == expect


def test_capacity_is_ceiling():
    for T in range(1, 60):
        for E in (1, 2, 3, 7):
            for k in (1, 2):
                C = O.capacity(T, E, k, 5, 4)
                exact = k * T * 5 / (4 * E)
                assert C - 1 < exact <= C


# -------------------------------------------------------------------------- top-k
def _topk_by_repeated_argmax(l, k):
    """Independent selection: take the maximum k times (np.argmax returns the
    first, i.e. lowest, index among equal maxima) and remove it."""
    l = l.astype(np.float64).copy()
    out = np.zeros((l.shape[0], k), np.int32)
    for r in range(k):
        j = np.argmax(l, axis=1)
        out[:, r] = j
        l[np.arange(l.shape[0]), j] = -np.inf
    return out


@pytest.mark.parametrize("E,k", [(4, 1), (16, 2), (8, 2), (64, 2), (5, 3)])
def test_topk_matches_repeated_argmax_with_ties(E, k):
    l = routing_logits(400, E, seed=7 + E, ties=0.3)
    np.testing.assert_array_equal(O.topk_route(l, k), _topk_by_repeated_argmax(l, k))


def test_topk_all_equal_picks_lowest_indices():
    l = np.full((5, 8), 0.25, np.float32)
    np.testing.assert_array_equal(O.topk_route(l, 3), np.tile([0, 1, 2], (5, 1)))


def test_topk_negative_zero_ties_positive_zero():
    l = np.array([[-0.0, 0.0, -1.0]], np.float32)
    np.testing.assert_array_equal(O.topk_route(l, 2), [[0, 1]])


def test_topk_rank_order_descending():
    l = routing_logits(200, 16, seed=3)
    idx = O.topk_route(l, 4)
    vals = np.take_along_axis(l, idx.astype(np.int64), 1)
    assert np.all(vals[:, :-1] >= vals[:, 1:])


# -------------------------------------------------------------------------- weights
def test_top1_weight_is_softmax_max_and_e2_sigmoid():
    l = routing_logits(300, 2, seed=11, scale=2.0)
    idx = O.topk_route(l, 1)
    p, w = O.gate_weights(l, idx, renorm=0)
    np.testing.assert_allclose(w[:, 0], p.max(axis=1), rtol=0, atol=0)
    gap = np.abs(l[:, 0].astype(np.float64) - l[:, 1])
    np.testing.assert_allclose(w[:, 0], 1.0 / (1.0 + np.exp(-gap)), rtol=1e-14)


def test_renorm_weights_sum_to_one_and_shift_invariant():
    l = routing_logits(300, 16, seed=12)
    idx = O.topk_route(l, 2)
    _, w = O.gate_weights(l, idx, renorm=1)
    np.testing.assert_allclose(w.sum(1), 1.0, rtol=1e-14)
    # k=2 renormalised weights are a sigmoid of the logit gap of the two choices
    l0 = np.take_along_axis(l, idx[:, :1].astype(np.int64), 1)[:, 0].astype(np.float64)
    l1 = np.take_along_axis(l, idx[:, 1:].astype(np.int64), 1)[:, 0].astype(np.float64)
    np.testing.assert_allclose(w[:, 0], 1.0 / (1.0 + np.exp(-(l0 - l1))), rtol=1e-13)
    _, w2 = O.gate_weights(l.astype(np.float64) + 3.0, idx, renorm=1)
    np.testing.assert_allclose(w, w2, rtol=1e-12)


def test_softmax_closed_form_uniform():
    p = O.softmax(np.zeros((3, 5)))
    np.testing.assert_allclose(p, 0.2, rtol=1e-15)


# ------------------------------------------------------------------ capacity rule
def _slots_by_sorting(idx, E, C, carry):
    """Different algorithm: list every (expert, token, rank) assignment, sort by
    expert then (token, rank), and give each expert's first C - carry_e entries
    consecutive rows starting at carry_e."""
    T, k = idx.shape
    ent = sorted((int(idx[t, r]), t, r) for t in range(T) for r in range(k))
    slot = np.full((T, k), -1, np.int32)
    pos = {}
    for e, t, r in ent:
        n = pos.get(e, 0)
        if carry[e] + n < C:
            slot[t, r] = carry[e] + n
        pos[e] = n + 1
    fill = np.array([min(C, carry[e] + pos.get(e, 0)) for e in range(E)])
    return slot, fill


@pytest.mark.parametrize("T,E,k,C", [(300, 4, 1, 60), (500, 16, 2, 40), (257, 8, 2, 70),
                                     (1000, 64, 2, 9)])
def test_slots_match_sort_based_bruteforce(T, E, k, C):
    rng = np.random.default_rng(T + E)
    l = routing_logits(T, E, seed=T * 3 + k)
    l[:, 0] += 1.5        # skew: expert 0 overflows
    idx = O.topk_route(l, k)
    carry = rng.integers(0, C // 2, size=E)
    slot, fill = O.assign_slots(idx, E, C, carry)
    s2, f2 = _slots_by_sorting(idx, E, C, carry)
    np.testing.assert_array_equal(slot, s2)
    np.testing.assert_array_equal(fill, f2)
    # invariants: slots unique per expert, in [carry, C), kept = min(demand, C - carry)
    for e in range(E):
        s = slot[idx == e]
        kept = s[s >= 0]
        assert len(np.unique(kept)) == len(kept)
        assert np.all((kept >= carry[e]) & (kept < C))
        demand = int((idx == e).sum())
        assert len(kept) == min(demand, C - carry[e])


def test_paper_worked_example_capacity_passing():
    g = json.load(open(os.path.join(GOLDEN, "capacity_passing_example.json")))
    C, E, n = g["C"], g["E"], g["tokens_per_microbatch"]
    idx = np.array(g["expert_of_token"], np.int32)[:, None]
    exp = g["expected"]

    def dropped(slot, idx_):
        return [int(((idx_[:, 0] == e) & (slot[:, 0] < 0)).sum()) for e in range(E)]

    slot_u, _ = O.assign_slots(idx, E, C)
    assert dropped(slot_u, idx) == exp["unpartitioned_dropped_per_expert"]

    assert C // 2 == exp["direct_microbatching_capacity"]
    slot_d = O.assign_slots_direct_microbatch(idx, E, C, 2)
    assert dropped(slot_d, idx) == exp["direct_microbatching_dropped_per_expert"]
    per_mb = [dropped(slot_d[i * n:(i + 1) * n], idx[i * n:(i + 1) * n]) for i in range(2)]
    assert per_mb == exp["direct_microbatching_dropped_in_microbatch"]

    s0, f0 = O.assign_slots(idx[:n], E, C)
    assert list(C - f0) == exp["capacity_passing_remaining_after_microbatch0"]
    s1, _ = O.assign_slots(idx[n:], E, C, carry=f0)
    slot_p = np.concatenate([s0, s1])
    assert dropped(slot_p, idx) == exp["capacity_passing_dropped_per_expert"]
    np.testing.assert_array_equal(slot_p, slot_u)


@settings(max_examples=60, deadline=None)
@given(T=st.integers(1, 120), E=st.integers(1, 9), k=st.integers(1, 3),
       C=st.integers(1, 40), seed=st.integers(0, 10_000), n_cuts=st.integers(0, 6))
def test_capacity_passing_equals_unpartitioned(T, E, k, C, seed, n_cuts):
    k = min(k, E)
    rng = np.random.default_rng(seed)
    idx = O.topk_route(rng.standard_normal((T, E)).astype(np.float32), k)
    cuts = sorted(set(rng.integers(0, T + 1, size=n_cuts).tolist()) | {0, T})
    slot_u, fill_u = O.assign_slots(idx, E, C)
    carry = np.zeros(E, np.int64)
    parts = []
    for a, b in zip(cuts[:-1], cuts[1:]):
        s, carry = O.assign_slots(idx[a:b], E, C, carry)
        parts.append(s)
    np.testing.assert_array_equal(np.concatenate(parts) if parts else slot_u, slot_u)
    np.testing.assert_array_equal(carry, fill_u)


# -------------------------------------------------------------------------- dispatch
def test_dispatch_is_exact_permutation_and_send_counts():
    T, E, k, C, d, G = 200, 8, 2, 30, 12, 4
    rng = np.random.default_rng(5)
    x = rng.standard_normal((T, d))
    idx = O.topk_route(rng.standard_normal((T, E)).astype(np.float32), k)
    slot, fill = O.assign_slots(idx, E, C)
    buf = O.dispatch(x, idx, slot, E, C)
    kept = slot >= 0
    assert int(kept.sum()) == int(fill.sum())
    for e in range(E):
        n = int(fill[e])
        assert not np.isnan(buf[e, :n]).any() and np.isnan(buf[e, n:]).all()
        src = [t for t in range(T) for r in range(k) if idx[t, r] == e and slot[t, r] >= 0]
        np.testing.assert_array_equal(buf[e, :n], x[src])       # bitwise rows, token order
    sc = O.send_counts(fill, G)
    assert sc.shape == (G,) and int(sc.sum()) == int(kept.sum())
    np.testing.assert_array_equal(sc, [fill[g * 2:(g + 1) * 2].sum() for g in range(G)])


# ------------------------------------------------------- batch-prioritized routing
def test_bpr_hand_worked_example():
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "bpr_small_example.json")))
    l = np.array(g["logits"], np.float32)
    idx = O.topk_route(l, g["k"])
    np.testing.assert_array_equal(idx, g["expected"]["idx"])
    imp = O.bpr_importance(l, idx)
    slot, fill, order = O.assign_slots_bpr(idx, g["E"], g["C"], imp)
    np.testing.assert_array_equal(order, g["expected"]["order"])
    np.testing.assert_array_equal(slot, g["expected"]["slot"])
    np.testing.assert_array_equal(fill, g["expected"]["fill"])
    s_tok, _ = O.assign_slots(idx, g["E"], g["C"])
    np.testing.assert_array_equal(s_tok, g["expected"]["token_order_slot"])


def test_bpr_importance_closed_forms():
    rng = np.random.default_rng(11)
    l = (rng.standard_normal((64, 6)) * 2).astype(np.float32)
    # top-1: the largest probability, 1 / sum_e exp(l_e - max)
    i1 = O.topk_route(l, 1)
    ld = l.astype(np.float64)
    want = 1.0 / np.exp(ld - ld.max(axis=1, keepdims=True)).sum(axis=1)
    np.testing.assert_array_equal(O.bpr_importance(l, i1), want.astype(np.float32))
    # every expert selected: the probabilities sum to one
    iE = O.topk_route(l, 6)
    np.testing.assert_array_equal(O.bpr_importance(l, iE), np.ones(64, np.float32))
    # E = 2, top-1: the logistic function of the logit gap
    l2 = l[:, :2]
    gap = np.abs(l2[:, 0].astype(np.float64) - l2[:, 1])
    np.testing.assert_allclose(O.bpr_importance(l2, O.topk_route(l2, 1)), 1 / (1 + np.exp(-gap)), rtol=1e-6)


@pytest.mark.parametrize("seed,T,E,k,C", [(0, 300, 8, 2, 40), (1, 257, 4, 1, 50), (2, 500, 16, 2, 30),
                                          (3, 100, 8, 3, 25)])
def test_bpr_kept_outrank_dropped(seed, T, E, k, C):
    rng = np.random.default_rng(seed)
    l = rng.standard_normal((T, E)).astype(np.float32)
    l[rng.random(T) < 0.1] = l[0]                    # equal-importance ties
    idx = O.topk_route(l, k)
    imp = O.bpr_importance(l, idx)
    slot, fill, order = O.assign_slots_bpr(idx, E, C, imp)
    assert sorted(order.tolist()) == list(range(T))
    demand = np.bincount(idx.ravel(), minlength=E)
    np.testing.assert_array_equal(fill, np.minimum(demand, C))      # order changes who, not how many
    pri = {int(t): i for i, t in enumerate(order)}                  # position in the visiting order
    for e in range(E):
        kept = [(t, int(slot[t, r])) for t in range(T) for r in range(k) if idx[t, r] == e and slot[t, r] >= 0]
        drop = [t for t in range(T) for r in range(k) if idx[t, r] == e and slot[t, r] < 0]
        assert sorted(s for _, s in kept) == list(range(len(kept)))
        # rows in priority order; every kept token is ahead of every dropped one:
        # higher importance, or equal importance and a lower token index
        ks = sorted(kept, key=lambda ts: ts[1])
        for (a, _), (b, _) in zip(ks, ks[1:]):
            assert imp[a] > imp[b] or (imp[a] == imp[b] and a < b)
        if kept and drop:
            a = ks[-1][0]
            for b in drop:
                assert imp[a] > imp[b] or (imp[a] == imp[b] and a < b)
                assert pri[a] < pri[b]


def test_bpr_equal_importance_is_token_order():
    # every row a permutation of one logit vector: one importance for all tokens
    rng = np.random.default_rng(4)
    base = rng.standard_normal(8).astype(np.float32)
    l = np.stack([rng.permutation(base) for _ in range(200)])
    idx = O.topk_route(l, 2)
    imp = O.bpr_importance(l, idx)
    assert np.unique(imp).size == 1
    slot, fill, order = O.assign_slots_bpr(idx, 8, 30, imp)
    s_tok, f_tok = O.assign_slots(idx, 8, 30)
    np.testing.assert_array_equal(order, np.arange(200))
    np.testing.assert_array_equal(slot, s_tok)
    np.testing.assert_array_equal(fill, f_tok)


def test_bpr_monotone_importance():
    # importance strictly decreasing in t: token order; increasing: reversed
    T, E, C = 120, 4, 20
    a = np.linspace(3.0, 0.5, T).astype(np.float32)
    l = np.zeros((T, E), np.float32)
    l[:, 0] = a
    l[np.arange(T) % 2 == 1] = np.roll(l[np.arange(T) % 2 == 1], 1, axis=1)   # half the tokens on expert 1
    idx = O.topk_route(l, 1)
    imp = O.bpr_importance(l, idx)
    assert np.all(np.diff(imp.astype(np.float64)) < 0)
    slot, _, order = O.assign_slots_bpr(idx, E, C, imp)
    np.testing.assert_array_equal(order, np.arange(T))
    np.testing.assert_array_equal(slot, O.assign_slots(idx, E, C)[0])
    lr, ir = l[::-1].copy(), idx[::-1].copy()
    slot_r, _, order_r = O.assign_slots_bpr(ir, E, C, O.bpr_importance(lr, ir))
    np.testing.assert_array_equal(order_r, np.arange(T)[::-1])
    np.testing.assert_array_equal(slot_r[::-1], O.assign_slots(idx, E, C)[0])
