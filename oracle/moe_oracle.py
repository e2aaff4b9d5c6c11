"""CPU oracle for the capacity-bounded top-k MoE layer and its exact gradient.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import this
module: only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline``
leg of ``bench.py`` use it.  It shares no code with the HIP library.

It is a plain, slow, float64 statement of what the paper's MoE layer computes
(Background, "Mixture of Experts": gate -> rearrangement into an E x C
capacity-bounded layout -> experts -> restoring the original token order).
The paper's transformations (batch partitioning with capacity passing, dX/dW
separation) are defined to leave the result unchanged (Introduction; Sec. 2.3
"Challenge 1"), so the oracle is the unpartitioned layer.

Readings of points the paper leaves open:

* capacity ``C = ceil(k*T*cf/E)`` in exact integer arithmetic, ``T`` the
  unpartitioned token count (the paper only states that each expert accepts at
  most C tokens per device);
* capacity is filled token-major: token t ascending, then rank r ascending --
  the order in which a single per-expert "remaining capacity" carried from one
  batch partition to the next reproduces the unpartitioned drops (Sec. 2.3,
  "Challenge 1");
* top-k orders experts by (logit descending, expert index ascending) on the
  float32 logits; the logits are the float64 dot product rounded once to
  float32, so the integer decision is taken in float32;
* weights: top-1 ``w = softmax(l)[e*]``; renormalised top-k
  ``w_r = p[e_r] / sum_sel p``, computed before the capacity rule;
* a dropped assignment contributes zero (a token with every choice dropped
  gets y = 0); rows of the E x C buffer past an expert's fill are unspecified
  (NaN here) and never read;
* no gradient flows through the top-k choice or the capacity rule, only
  through the weights; there is no auxiliary loss;
* the loss is ``L = sum_t <dy_t, y_t>`` for a given upstream gradient dy;
* Batch-prioritized Routing (named in Sec. 2.3 as a gate that decides over
  the whole batch): a token's importance is the sum of the softmax
  probabilities of its k selected experts (over all E, not renormalised),
  evaluated in float64 and rounded once to float32; tokens are visited by
  importance descending, equal importance in token order, each token's
  choices in rank order, under the same capacity rule.

Parity pins for every function live in tests/test_oracle_*.py (not gpu).
"""
from __future__ import annotations

import math

import numpy as np

__all__ = [
    "capacity", "gate_logits", "topk_route", "softmax", "gate_weights",
    "assign_slots", "assign_slots_direct_microbatch", "bpr_importance", "bpr_order",
    "assign_slots_bpr", "dispatch", "send_counts",
    "act", "act_grad", "expert_ffn", "combine",
    "combine_bwd", "expert_bwd_dx", "expert_bwd_dw", "dispatch_bwd", "gate_bwd",
    "layer_forward", "layer_backward", "expert_row_forward", "expert_row_backward",
    "expert_rows", "expert_dw1_row", "expert_dw2_col",
]

F64 = np.float64


# --------------------------------------------------------------------------- gate
def capacity(T: int, E: int, k: int, cf_num: int, cf_den: int) -> int:
    """Expert capacity C (Background, "Expert-parallelism"): the most tokens one
    expert accepts on one device.  Reading: ceil(k*T*cf/E), exact integers."""
    if T <= 0:
        return 0
    return -(-(k * T * cf_num) // (E * cf_den))


def gate_logits(x: np.ndarray, Wg: np.ndarray, bias=None, round_f32: bool = True) -> np.ndarray:
    """Gating scores from a trainable linear layer (Background, "Routing
    algorithms"): l[t][e] = <x_t, Wg_e> (+ b_e), in float64, rounded once to
    float32 (``round_f32=False`` keeps float64, for finite-difference checks)."""
    l = np.asarray(x, F64) @ np.asarray(Wg, F64).T
    if bias is not None:
        l = l + np.asarray(bias, F64)[None, :]
    return l.astype(np.float32) if round_f32 else l


def topk_route(logits32: np.ndarray, k: int) -> np.ndarray:
    """Top-k routing (Background, "Routing algorithms"): the k experts with the
    highest scores, in rank order; equal scores go to the lower expert index."""
    l = np.asarray(logits32).astype(F64)
    T, E = l.shape
    eidx = np.broadcast_to(np.arange(E), (T, E))
    order = np.lexsort((eidx, -l), axis=-1)       # primary: -logit, secondary: index
    return np.ascontiguousarray(order[:, :k]).astype(np.int32)


def softmax(l: np.ndarray) -> np.ndarray:
    l = np.asarray(l, F64)
    z = np.exp(l - l.max(axis=-1, keepdims=True))
    return z / z.sum(axis=-1, keepdims=True)


def gate_weights(logits32: np.ndarray, idx: np.ndarray, renorm: int):
    """Combine weights of the selected experts.  Returns (p, w): p the softmax
    over all experts, w [T][k].  Top-1 Switch-style gate (Sec. 2.3): w = p[e*];
    renormalised top-k: w_r = p[e_r] / sum of p over the selected experts."""
    p = softmax(np.asarray(logits32).astype(F64))
    sel = np.take_along_axis(p, idx.astype(np.int64), axis=1)
    w = sel / sel.sum(axis=1, keepdims=True) if renorm else sel
    return p, w


# ---------------------------------------------------------------- capacity / dispatch
def assign_slots(idx: np.ndarray, E: int, C: int, carry=None):
    """Capacity-bounded slot assignment (Background, "Expert-parallelism";
    Sec. 2.3 "Challenge 1", capacity passing between partitions).

    Starting from ``carry[e]`` tokens already placed in expert e by earlier
    partitions, walk tokens in order and each token's choices in rank order:
    the assignment takes the next free row of its expert if one is left below
    C, else it is dropped (slot -1).  Returns (slot [T][k] int32, fill [E]):
    ``fill`` is the carry handed to the next partition.
    """
    T, k = idx.shape
    fill = np.zeros(E, np.int64) if carry is None else np.asarray(carry, np.int64).copy()
    slot = np.full((T, k), -1, np.int32)
    for t in range(T):
        for r in range(k):
            e = int(idx[t, r])
            if fill[e] < C:
                slot[t, r] = fill[e]
                fill[e] += 1
    return slot, fill


def assign_slots_direct_microbatch(idx: np.ndarray, E: int, C: int, n_parts: int):
    """Negative control (Sec. 2.3, direct micro-batching): every partition gets
    capacity C // n_parts afresh, which drops extra tokens."""
    T = idx.shape[0]
    bounds = np.linspace(0, T, n_parts + 1).astype(int)
    slots = []
    for i in range(n_parts):
        s, _ = assign_slots(idx[bounds[i]:bounds[i + 1]], E, C // n_parts)
        slots.append(s)
    return np.concatenate(slots, axis=0)


def dispatch(x: np.ndarray, idx: np.ndarray, slot: np.ndarray, E: int, C: int) -> np.ndarray:
    """Re-arrange tokens by target expert into the fixed E x C x d buffer handed
    to the all-to-all (Sec. 2.3; Implementation, irregular all-to-all).  With G
    destination slices of E/G experts each, this [E][C][d] array is the same
    memory as [G][E/G][C][d].  Rows past an expert's fill are NaN (unspecified)."""
    T, d = x.shape
    buf = np.full((E, C, d), np.nan, F64)
    for t in range(T):
        for r in range(idx.shape[1]):
            s = int(slot[t, r])
            if s >= 0:
                buf[int(idx[t, r]), s] = x[t]
    return buf


# ------------------------------------------------------- batch-prioritized routing
def bpr_importance(logits32: np.ndarray, idx: np.ndarray) -> np.ndarray:
    """Importance score of each token for Batch-prioritized Routing (Sec. 2.3,
    "Opportunities and Challenges", the gating methods that decide over the
    whole batch): the sum of the token's k largest gating scores, i.e. of the
    softmax probabilities (over all E experts) of its selected experts, not
    renormalised.  Evaluated in float64 from the float32 logits and rounded
    once to float32: the ordering decision is taken on these float32 values."""
    p = softmax(np.asarray(logits32).astype(F64))
    sel = np.take_along_axis(p, np.asarray(idx, np.int64), axis=1)
    imp = np.zeros(sel.shape[0], F64)
    for r in range(sel.shape[1]):       # rank order
        imp = imp + sel[:, r]
    return imp.astype(np.float32)


def bpr_order(importance32: np.ndarray) -> np.ndarray:
    """Order in which Batch-prioritized Routing visits the tokens: importance
    descending; equal importance keeps token order (a stable sort)."""
    imp = np.asarray(importance32, np.float32).astype(F64)
    return np.argsort(-imp, kind="stable").astype(np.int32)


def assign_slots_bpr(idx: np.ndarray, E: int, C: int, importance32: np.ndarray):
    """Batch-prioritized capacity rule (Sec. 2.3): tokens are sorted by
    importance first and then assigned to experts, so the least important
    tokens are the ones dropped.  The capacity rule of ``assign_slots`` runs
    over the tokens in ``bpr_order`` (each token's choices in rank order), so
    an expert's rows hold its kept tokens by descending importance.  The whole
    batch decides the order, so there is no carry from earlier partitions.
    Returns (slot [T][k] in token order, fill [E], order [T])."""
    order = bpr_order(importance32)
    slot_sorted, fill = assign_slots(np.asarray(idx)[order], E, C)
    slot = np.empty_like(slot_sorted)
    slot[order] = slot_sorted
    return slot, fill, order


def send_counts(fill: np.ndarray, G: int) -> np.ndarray:
    """Rows to send to each destination slice: the payload of the first
    all-to-all of the irregular exchange (Implementation)."""
    f = np.asarray(fill, np.int64)
    return f.reshape(G, -1).sum(axis=1)


# -------------------------------------------------------------------------- experts
_GELU_C = math.sqrt(2.0 / math.pi)


def act(h: np.ndarray, kind: str) -> np.ndarray:
    h = np.asarray(h, F64)
    if kind == "relu":
        return np.maximum(h, 0.0)
    if kind == "gelu_tanh":
        return 0.5 * h * (1.0 + np.tanh(_GELU_C * (h + 0.044715 * h ** 3)))
    if kind == "gelu_erf":
        from scipy.special import erf
        return 0.5 * h * (1.0 + erf(h / math.sqrt(2.0)))
    if kind == "identity":
        return h.copy()
    raise ValueError(kind)


def act_grad(h: np.ndarray, kind: str) -> np.ndarray:
    """Derivative of ``act`` with respect to its input."""
    h = np.asarray(h, F64)
    if kind == "relu":
        return (h > 0).astype(F64)
    if kind == "gelu_tanh":
        u = _GELU_C * (h + 0.044715 * h ** 3)
        th = np.tanh(u)
        du = _GELU_C * (1.0 + 3 * 0.044715 * h ** 2)
        return 0.5 * (1.0 + th) + 0.5 * h * (1.0 - th ** 2) * du
    if kind == "gelu_erf":
        from scipy.special import erf
        return 0.5 * (1.0 + erf(h / math.sqrt(2.0))) + h * np.exp(-0.5 * h * h) / math.sqrt(2 * math.pi)
    if kind == "identity":
        return np.ones_like(h)
    raise ValueError(kind)


def expert_ffn(buf: np.ndarray, row_begin, row_end, W1: np.ndarray, W2: np.ndarray, kind: str):
    """Each expert runs its two-layer FFN on its own rows (Background, "Mixture
    of Experts"): H = X_e W1_e^T, A = act(H), O = A W2_e^T, rows
    [row_begin_e, row_end_e) only.  Returns H, A, O ([E][C][*], NaN elsewhere)."""
    E, C, d = buf.shape
    f = W1.shape[1]
    H = np.full((E, C, f), np.nan, F64)
    A = np.full((E, C, f), np.nan, F64)
    O = np.full((E, C, d), np.nan, F64)
    for e in range(E):
        b, n = int(row_begin[e]), int(row_end[e])
        if n <= b:
            continue
        X = buf[e, b:n]
        H[e, b:n] = X @ np.asarray(W1[e], F64).T
        A[e, b:n] = act(H[e, b:n], kind)
        O[e, b:n] = A[e, b:n] @ np.asarray(W2[e], F64).T
    return H, A, O


def combine(O: np.ndarray, idx: np.ndarray, slot: np.ndarray, w: np.ndarray) -> np.ndarray:
    """Gather expert outputs back into token order, weighted by the gate
    (Fig. "moe_and_sharding", Gather): y_t = sum over kept r of w[t,r] O[e_r, s_r].
    A token whose every choice was dropped gets y_t = 0."""
    T, k = idx.shape
    d = O.shape[2]
    y = np.zeros((T, d), F64)
    for t in range(T):
        for r in range(k):
            s = int(slot[t, r])
            if s >= 0:
                y[t] += w[t, r] * O[int(idx[t, r]), s]
    return y


# ------------------------------------------------------------------------- backward
def combine_bwd(dy: np.ndarray, O: np.ndarray, idx, slot, w, E: int, C: int):
    """Backward of the weighted gather.  dO[e][s] = w[t,r] dy_t for every kept
    (t,r); g[t,r] = <dy_t, O[e][s]> = dL/dw[t,r] (0 when dropped)."""
    T, k = idx.shape
    d = dy.shape[1]
    dO = np.full((E, C, d), np.nan, F64)
    g = np.zeros((T, k), F64)
    dy = np.asarray(dy, F64)
    for t in range(T):
        for r in range(k):
            s = int(slot[t, r])
            if s >= 0:
                e = int(idx[t, r])
                dO[e, s] = w[t, r] * dy[t]
                g[t, r] = float(dy[t] @ O[e, s])
    return dO, g


def expert_bwd_dx(dO, H, row_begin, row_end, W1, W2, kind: str):
    """Activation-gradient (dX) half of the experts' backward (Sec. 2.2, Fig.
    "example_dw": the dReLU / dX chain does not need dW):
    dA = dO W2_e, dH = dA * act'(H), dX_e = dH W1_e."""
    E, C, d = dO.shape
    f = H.shape[2]
    dH = np.full((E, C, f), np.nan, F64)
    dX = np.full((E, C, d), np.nan, F64)
    for e in range(E):
        b, n = int(row_begin[e]), int(row_end[e])
        if n <= b:
            continue
        dA = dO[e, b:n] @ np.asarray(W2[e], F64)
        dH[e, b:n] = dA * act_grad(H[e, b:n], kind)
        dX[e, b:n] = dH[e, b:n] @ np.asarray(W1[e], F64)
    return dH, dX


def expert_bwd_dw(dO, A, dH, buf, row_begin, row_end):
    """Weight-gradient (dW) half, independent of the dX chain (Sec. 2.3
    "Opportunity 1"): dW2_e = dO_e^T A_e, dW1_e = dH_e^T X_e over the expert's
    rows; an expert with no rows gets exact zeros."""
    E, C, d = dO.shape
    f = A.shape[2]
    dW1 = np.zeros((E, f, d), F64)
    dW2 = np.zeros((E, d, f), F64)
    for e in range(E):
        b, n = int(row_begin[e]), int(row_end[e])
        if n <= b:
            continue
        dW2[e] = dO[e, b:n].T @ A[e, b:n]
        dW1[e] = dH[e, b:n].T @ buf[e, b:n]
    return dW1, dW2


def dispatch_bwd(dX: np.ndarray, idx, slot, T: int) -> np.ndarray:
    """Backward of the re-arrangement: dx_t = sum over kept r of dX[e_r][s_r]."""
    k = idx.shape[1]
    d = dX.shape[2]
    dx = np.zeros((T, d), F64)
    for t in range(T):
        for r in range(k):
            s = int(slot[t, r])
            if s >= 0:
                dx[t] += dX[int(idx[t, r]), s]
    return dx


def gate_bwd(g: np.ndarray, p: np.ndarray, w: np.ndarray, idx: np.ndarray, renorm: int):
    """dL/dlogits through the combine weights only.

    Renormalised top-k: w_r is a softmax over the selected logits, so for a
    selected expert j = e_r, dl_j = w_r (g_r - sum_s w_s g_s), and 0 otherwise.
    Plain top-k (top-1 Switch gate): w_r = p[e_r] with p the softmax over all
    experts, so dl_j = sum_r g_r p[e_r] (delta(j, e_r) - p_j).
    """
    T, k = idx.shape
    E = p.shape[1]
    dl = np.zeros((T, E), F64)
    for t in range(T):
        if renorm:
            mean = float(np.dot(w[t], g[t]))
            for r in range(k):
                dl[t, idx[t, r]] += w[t, r] * (g[t, r] - mean)
        else:
            for r in range(k):
                e = int(idx[t, r])
                coef = g[t, r] * p[t, e]
                dl[t] -= coef * p[t]
                dl[t, e] += coef
    return dl


# ------------------------------------------------------------------------ composite
def layer_forward(spec, inp, carry=None, C=None, exact_logits: bool = False, routing: str = "token",
                  idx_override=None):
    """The whole MoE layer forward for a LayerSpec-like object ``spec`` (fields
    T, E, k, cf_num, cf_den, act, renorm) and inputs dict (x, Wg, bias, W1, W2).
    ``C`` defaults to the capacity of the unpartitioned T tokens.  ``routing``
    "bpr" fills capacity in batch-prioritized order (``assign_slots_bpr``; no
    carry).  ``idx_override`` [T][k] replaces the top-k choice (a test that has
    checked another computation's choice to be a valid top-k of these logits,
    differing only at near-ties, follows it from there on).  Returns every
    intermediate, so each stage can be compared on its own."""
    x = np.asarray(inp["x"], F64)
    T = x.shape[0]
    if C is None:
        C = capacity(T, spec.E, spec.k, spec.cf_num, spec.cf_den)
    logits = gate_logits(inp["x"], inp["Wg"], inp.get("bias"), round_f32=not exact_logits)
    idx = topk_route(logits, spec.k) if idx_override is None else np.ascontiguousarray(idx_override, np.int32)
    p, w = gate_weights(logits, idx, spec.renorm)
    carry0 = np.zeros(spec.E, np.int64) if carry is None else np.asarray(carry, np.int64)
    order = None
    if routing == "bpr":
        assert carry is None, "batch-prioritized routing orders the whole batch: no carry"
        slot, fill, order = assign_slots_bpr(idx, spec.E, C, bpr_importance(logits, idx))
    else:
        slot, fill = assign_slots(idx, spec.E, C, carry0)
    buf = dispatch(x, idx, slot, spec.E, C)
    H, A, O = expert_ffn(buf, carry0, fill, inp["W1"], inp["W2"], spec.act)
    y = combine(O, idx, slot, w)
    return dict(C=C, logits=logits, idx=idx, p=p, w=w, slot=slot, fill=fill, carry=carry0,
                buf=buf, H=H, A=A, O=O, y=y, order=order)


def layer_backward(spec, inp, fw):
    """Backward of ``layer_forward`` for L = sum <dy, y>: the dX chain, then the
    dW products (which need only tensors the forward and dX chain left)."""
    E, C = spec.E, fw["C"]
    T = fw["idx"].shape[0]
    dO, g = combine_bwd(inp["dy"], fw["O"], fw["idx"], fw["slot"], fw["w"], E, C)
    dH, dX = expert_bwd_dx(dO, fw["H"], fw["carry"], fw["fill"], inp["W1"], inp["W2"], spec.act)
    dl = gate_bwd(g, fw["p"], fw["w"], fw["idx"], spec.renorm)
    dx = dispatch_bwd(dX, fw["idx"], fw["slot"], T) + dl @ np.asarray(inp["Wg"], F64)
    dW1, dW2 = expert_bwd_dw(dO, fw["A"], dH, fw["buf"], fw["carry"], fw["fill"])
    dWg = dl.T @ np.asarray(inp["x"], F64)
    return dict(dO=dO, g=g, dH=dH, dX=dX, dlogits=dl, dx=dx, dW1=dW1, dW2=dW2, dWg=dWg)


# ----------------------------------------------------- per-row forms (sampled checks)
def expert_row_forward(x_row, W1e, W2e, kind: str):
    """One kept (token, expert) pair: h = W1_e x, a = act(h), o = W2_e a."""
    h = np.asarray(W1e, F64) @ np.asarray(x_row, F64)
    a = act(h, kind)
    o = np.asarray(W2e, F64) @ a
    return h, a, o


def expert_row_backward(x_row, dO_row, W1e, W2e, kind: str):
    """dX row of one kept pair: dA = W2_e^T dO, dH = dA * act'(h), dX = W1_e^T dH."""
    h = np.asarray(W1e, F64) @ np.asarray(x_row, F64)
    dA = np.asarray(W2e, F64).T @ np.asarray(dO_row, F64)
    dH = dA * act_grad(h, kind)
    dX = np.asarray(W1e, F64).T @ dH
    return dH, dX


def expert_rows(x, dy, idx, slot, w, e: int):
    """The rows expert e holds, in buffer order: (X_e, dO_e) with dO = w * dy."""
    T, k = idx.shape
    pairs = sorted((int(slot[t, r]), t, r) for t in range(T) for r in range(k)
                   if int(idx[t, r]) == e and slot[t, r] >= 0)
    ts = [t for _, t, _ in pairs]
    ws = np.array([w[t, r] for _, t, r in pairs], F64)
    X = np.asarray(x, F64)[ts]
    dO = ws[:, None] * np.asarray(dy, F64)[ts]
    return X, dO


def expert_dw1_row(X_rows, dO_rows, W1e, W2e, kind: str, i: int):
    """Row i of dW1_e = sum over the expert's rows m of dH[m][i] X[m], with
    dH[m][i] = <W2_e[:, i], dO[m]> * act'(<W1_e[i], X[m]>)."""
    h_i = X_rows @ np.asarray(W1e[i], F64)
    dH_i = (dO_rows @ np.asarray(W2e, F64)[:, i]) * act_grad(h_i, kind)
    return dH_i @ X_rows


def expert_dw2_col(X_rows, dO_rows, W1e, kind: str, c: int):
    """Column c of dW2_e = sum over the expert's rows m of dO[m] A[m][c], with
    A[m][c] = act(<W1_e[c], X[m]>)."""
    a_c = act(X_rows @ np.asarray(W1e[c], F64), kind)
    return dO_rows.T @ a_c
