"""CPU oracle for the pre-LN transformer block whose FFN is the MoE layer.

TEST INFRASTRUCTURE ONLY (see moe_oracle.py): used by tests/, smoke() and the
CPU-baseline leg of bench.py, never by the product path.

The block is the one the paper partitions along the batch (Sec. 2.3, Fig.
"part_all"; Sec. 5): h = x + Wo * Attn(LN1(x)), out = h + MoE(LN2(h)), with
causal multi-head self-attention.  Partitioning is defined to leave the
result unchanged, so the oracle is the unpartitioned block, in float64, and
its exact gradient for L = sum <dy, out>.

Readings: LayerNorm with eps 1e-5 and affine gain/bias; QKV projection
Wqkv [3d][d] laid out as q, k, v blocks, head h using columns h*hd .. h*hd+hd-1
of each; scores scaled by 1/sqrt(hd); no biases on the projections; the MoE
layer is moe_oracle's (capacity of the unpartitioned token count).

Storage precision: in a bf16 block every activation that lives in memory
between two operations is a bf16 tensor -- the LN1 output, q/k/v, the
attention output, the residual stream h and the MoE input m.  With
``round_acts`` (the default for a bf16 block) the oracle computes each
operation in float64 from the rounded inputs and rounds its result once to
bf16 (nearest, ties to even), so the top-k decision is taken on the same
bf16 MoE input a bf16 implementation sees.  The block output and every
gradient stay float64; the backward treats the rounding as the identity.
"""
from __future__ import annotations

import math

import numpy as np

from oracle import moe_oracle as M

F64 = np.float64
LN_EPS = 1e-5

__all__ = ["layernorm", "layernorm_bwd", "attention", "attention_bwd", "block_forward", "block_backward",
           "block_forward_tokens", "round_bf16_f64"]


def round_bf16_f64(a: np.ndarray) -> np.ndarray:
    """Round float64 values to bfloat16 (nearest, ties to even), returned as float64.

    The rounding is done once, on the float64 bits; going through float32
    first could round twice."""
    a = np.asarray(a, F64)
    u = a.view(np.uint64)
    # bf16 keeps the top 7 of float64's 52 mantissa bits: round at bit 45
    lsb = (u >> np.uint64(45)) & np.uint64(1)
    r = (u + np.uint64((1 << 44) - 1) + lsb) & ~np.uint64((1 << 45) - 1)
    return r.view(F64)


def layernorm(x, g, b, eps: float = LN_EPS):
    """y = (x - mean) / sqrt(var + eps) * g + b over the last axis (biased variance).
    Returns (y, xhat, rstd)."""
    x = np.asarray(x, F64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (x - mu) * rstd
    return xhat * np.asarray(g, F64) + np.asarray(b, F64), xhat, rstd


def layernorm_bwd(dy, xhat, rstd, g):
    """Gradients of layernorm: (dx, dg, db)."""
    dy = np.asarray(dy, F64)
    dxhat = dy * np.asarray(g, F64)
    dx = rstd * (dxhat - dxhat.mean(-1, keepdims=True) - xhat * (dxhat * xhat).mean(-1, keepdims=True))
    return dx, (dy * xhat).sum(0), dy.sum(0)


def _heads(t, B, S, H):
    return np.asarray(t, F64).reshape(B, S, H, -1).transpose(0, 2, 1, 3)   # [B][H][S][hd]


def _merge(t):
    B, H, S, hd = t.shape
    return t.transpose(0, 2, 1, 3).reshape(B * S, H * hd)


def attention(q, k, v, B, S, H):
    """Causal softmax(q k^T / sqrt(hd)) v per batch and head.  q, k, v: [B*S][H*hd].
    Returns (o [B*S][H*hd], p [B][H][S][S])."""
    qh, kh, vh = _heads(q, B, S, H), _heads(k, B, S, H), _heads(v, B, S, H)
    hd = qh.shape[-1]
    s = qh @ kh.transpose(0, 1, 3, 2) / math.sqrt(hd)
    mask = np.triu(np.ones((S, S), bool), 1)
    s = np.where(mask, -np.inf, s)
    s = s - s.max(-1, keepdims=True)
    p = np.exp(s)
    p /= p.sum(-1, keepdims=True)
    return _merge(p @ vh), p


def attention_bwd(do, q, k, v, p, B, S, H):
    """Gradients of attention for upstream do [B*S][H*hd]: (dq, dk, dv) in the same layout."""
    doh, qh, kh, vh = _heads(do, B, S, H), _heads(q, B, S, H), _heads(k, B, S, H), _heads(v, B, S, H)
    hd = qh.shape[-1]
    dv = p.transpose(0, 1, 3, 2) @ doh
    dp = doh @ vh.transpose(0, 1, 3, 2)
    ds = p * (dp - (dp * p).sum(-1, keepdims=True))
    dq = ds @ kh / math.sqrt(hd)
    dk = ds.transpose(0, 1, 3, 2) @ qh / math.sqrt(hd)
    return _merge(dq), _merge(dk), _merge(dv)


def block_forward(spec, inp, round_acts=None, exact_logits=False, C=None, idx_override=None):
    """spec: BlockSpec-like (B, S, d, heads, moe=LayerSpec-like).  inp: x, ln1_g, ln1_b, Wqkv,
    Wo, ln2_g, ln2_b, Wg, W1, W2 (and dy for the backward).  ``round_acts`` (default: the
    block is bf16) rounds the stored activations to bf16; ``exact_logits`` keeps the gate
    logits in float64 (for comparisons against float64 autograd); ``C`` is the expert
    capacity (default: that of the B*S tokens given); ``idx_override`` replaces the
    MoE layer's top-k choice (see moe_oracle.layer_forward)."""
    B, S, d, H = spec.B, spec.S, spec.d, spec.heads
    if round_acts is None:
        round_acts = spec.moe.dtype == "bf16"
    rnd = round_bf16_f64 if round_acts else (lambda t: t)
    x = np.asarray(inp["x"], F64)
    a, a_hat, a_rstd = layernorm(x, inp["ln1_g"], inp["ln1_b"])
    a = rnd(a)
    qkv = rnd(a @ np.asarray(inp["Wqkv"], F64).T)
    q, k, v = qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:]
    o, p = attention(q, k, v, B, S, H)
    o = rnd(o)
    h = rnd(x + o @ np.asarray(inp["Wo"], F64).T)
    m, m_hat, m_rstd = layernorm(h, inp["ln2_g"], inp["ln2_b"])
    m_in = rnd(m)
    moe_inp = {"x": m_in, "Wg": inp["Wg"], "W1": inp["W1"], "W2": inp["W2"], "bias": None}
    mw = M.layer_forward(spec.moe, moe_inp, exact_logits=exact_logits, C=C, idx_override=idx_override)
    out = h + mw["y"]
    return dict(a=a, a_hat=a_hat, a_rstd=a_rstd, q=q, k=k, v=v, o=o, p=p, h=h, m=m, m_in=m_in,
                m_hat=m_hat, m_rstd=m_rstd, moe=mw, moe_inp=moe_inp, out=out)


def block_backward(spec, inp, fw):
    B, S, d, H = spec.B, spec.S, spec.d, spec.heads
    dy = np.asarray(inp["dy"], F64)
    mb = M.layer_backward(spec.moe, {**fw["moe_inp"], "dy": dy}, fw["moe"])
    dm = mb["dx"]
    dh_ln, dln2_g, dln2_b = layernorm_bwd(dm, fw["m_hat"], fw["m_rstd"], inp["ln2_g"])
    dh = dy + dh_ln
    Wo = np.asarray(inp["Wo"], F64)
    do = dh @ Wo
    dWo = dh.T @ fw["o"]
    dq, dk, dv = attention_bwd(do, fw["q"], fw["k"], fw["v"], fw["p"], B, S, H)
    dqkv = np.concatenate([dq, dk, dv], axis=1)
    Wqkv = np.asarray(inp["Wqkv"], F64)
    da = dqkv @ Wqkv
    dWqkv = dqkv.T @ fw["a"]
    dx_ln, dln1_g, dln1_b = layernorm_bwd(da, fw["a_hat"], fw["a_rstd"], inp["ln1_g"])
    dx = dh + dx_ln
    return dict(dx=dx, dh=dh, dm=dm, do=do, dq=dq, dk=dk, dv=dv, dqkv=dqkv, da=da, dWo=dWo, dWqkv=dWqkv,
                dln1_g=dln1_g, dln1_b=dln1_b, dln2_g=dln2_g, dln2_b=dln2_b, moe=mb)


def block_forward_tokens(spec, inp, seq, positions, round_acts=None):
    """The block at selected positions of sequence ``seq`` only, from that
    sequence's causal prefix (for sampled checks of large batches).

    Causal attention makes a token's h depend only on its sequence's earlier
    tokens, and the MoE output of a token none of whose choices is dropped
    depends only on the token itself, so this equals block_forward on those
    rows whenever the batch drops nothing (the caller checks that).  Returns
    h, m_in, logits, idx, w and out for the positions, in the given order."""
    S, d, H = spec.S, spec.d, spec.heads
    lay = spec.moe
    if round_acts is None:
        round_acts = lay.dtype == "bf16"
    rnd = round_bf16_f64 if round_acts else (lambda t: t)
    pos = np.asarray(positions, np.int64)
    P = int(pos.max()) + 1
    x = np.asarray(inp["x"], F64)[seq * S: seq * S + P]
    a = rnd(layernorm(x, inp["ln1_g"], inp["ln1_b"])[0])
    qkv = rnd(a @ np.asarray(inp["Wqkv"], F64).T)
    o, _ = attention(qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:], 1, P, H)
    o = rnd(o[pos])
    h = rnd(x[pos] + o @ np.asarray(inp["Wo"], F64).T)
    m_in = rnd(layernorm(h, inp["ln2_g"], inp["ln2_b"])[0])
    logits = M.gate_logits(m_in, inp["Wg"], None)
    idx = M.topk_route(logits, lay.k)
    _, w = M.gate_weights(logits, idx, lay.renorm)
    y = np.zeros_like(h)
    for t in range(len(pos)):
        for r in range(lay.k):
            e = int(idx[t, r])
            y[t] += w[t, r] * M.expert_row_forward(m_in[t], inp["W1"][e], inp["W2"][e], lay.act)[2]
    return dict(h=h, m_in=m_in, logits=logits, idx=idx, w=w, out=h + y)
