"""Pins for the block oracle (CPU only): LayerNorm closed forms, attention
against torch's float64 scaled_dot_product_attention, the causal first-token
identity, exact bf16 rounding, and the whole block's gradient against torch
float64 autograd on an independently written block."""
import math
from types import SimpleNamespace

import numpy as np
import pytest
import torch

from oracle import block_oracle as BO
from oracle import moe_oracle as M
from synth import round_bf16


def test_layernorm_unit_affine_gives_zero_mean_unit_variance():
    x = np.random.default_rng(0).standard_normal((7, 33)) * 3 + 2
    y, xhat, rstd = BO.layernorm(x, np.ones(33), np.zeros(33))
    np.testing.assert_allclose(y.mean(1), 0, atol=1e-14)
    np.testing.assert_allclose(y.var(1), 1 - BO.LN_EPS * rstd[:, 0] ** 2, rtol=1e-12)   # var/(var+eps)


def test_layernorm_bwd_matches_torch():
    rng = np.random.default_rng(1)
    x, g, b, dy = rng.standard_normal((5, 16)), rng.standard_normal(16), rng.standard_normal(16), rng.standard_normal((5, 16))
    _, xhat, rstd = BO.layernorm(x, g, b)
    dx, dg, db = BO.layernorm_bwd(dy, xhat, rstd, g)
    t = [torch.tensor(a, requires_grad=True) for a in (x, g, b)]
    (torch.nn.functional.layer_norm(t[0], (16,), t[1], t[2], eps=BO.LN_EPS) * torch.tensor(dy)).sum().backward()
    for got, tt in zip((dx, dg, db), t):
        np.testing.assert_allclose(got, tt.grad.numpy(), rtol=1e-11, atol=1e-13)


@pytest.mark.parametrize("B,S,H,hd", [(2, 9, 3, 4), (1, 17, 2, 8)])
def test_attention_matches_sdpa_and_backward_matches_autograd(B, S, H, hd):
    rng = np.random.default_rng(B * 100 + S)
    q, k, v, do = (rng.standard_normal((B * S, H * hd)) for _ in range(4))
    o, p = BO.attention(q, k, v, B, S, H)
    th = lambda a: torch.tensor(a).reshape(B, S, H, hd).transpose(1, 2).clone().requires_grad_(True)
    tq, tk, tv = th(q), th(k), th(v)
    to = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True)
    np.testing.assert_allclose(o, to.transpose(1, 2).reshape(B * S, H * hd).detach().numpy(), rtol=1e-12, atol=1e-13)
    (to * th(do).detach()).sum().backward()
    dq, dk, dv = BO.attention_bwd(do, q, k, v, p, B, S, H)
    for got, tt in zip((dq, dk, dv), (tq, tk, tv)):
        np.testing.assert_allclose(got, tt.grad.transpose(1, 2).reshape(B * S, H * hd).numpy(), rtol=1e-11, atol=1e-12)


def test_causal_first_token_attends_only_to_itself():
    rng = np.random.default_rng(3)
    B, S, H, hd = 2, 6, 2, 4
    q, k, v = (rng.standard_normal((B * S, H * hd)) for _ in range(3))
    o, _ = BO.attention(q, k, v, B, S, H)
    for b in range(B):
        np.testing.assert_allclose(o[b * S], v[b * S], rtol=0, atol=1e-15)


def test_round_bf16_f64_matches_float32_rounding_on_float32_values():
    x = (np.random.default_rng(4).standard_normal(10000) * 10).astype(np.float32)
    np.testing.assert_array_equal(BO.round_bf16_f64(x.astype(np.float64)), round_bf16(x).astype(np.float64))
    # ties to even and a value just above a tie
    one = 1.0
    tie = one + 2.0 ** -8                      # halfway between 1 and 1 + 2^-7
    assert BO.round_bf16_f64(np.array([tie]))[0] == one
    assert BO.round_bf16_f64(np.array([tie + 2.0 ** -40]))[0] == one + 2.0 ** -7
    assert BO.round_bf16_f64(np.array([one + 3 * 2.0 ** -8]))[0] == one + 2 * 2.0 ** -7


def _spec(B=2, S=8, d=16, H=2, E=4, k=2, f=24, act="gelu_tanh"):
    moe = SimpleNamespace(T=B * S, d=d, f=f, E=E, k=k, cf_num=5, cf_den=4, act=act, renorm=1, dtype="f32")
    return SimpleNamespace(B=B, S=S, d=d, heads=H, moe=moe)


def _inputs(spec, seed):
    rng = np.random.default_rng(seed)
    d, E, f = spec.d, spec.moe.E, spec.moe.f
    T = spec.B * spec.S
    return dict(x=rng.standard_normal((T, d)), dy=rng.standard_normal((T, d)),
                ln1_g=1 + 0.1 * rng.standard_normal(d), ln1_b=0.1 * rng.standard_normal(d),
                ln2_g=1 + 0.1 * rng.standard_normal(d), ln2_b=0.1 * rng.standard_normal(d),
                Wqkv=0.3 * rng.standard_normal((3 * d, d)), Wo=0.3 * rng.standard_normal((d, d)),
                Wg=0.5 * rng.standard_normal((E, d)), W1=0.3 * rng.standard_normal((E, f, d)),
                W2=0.3 * rng.standard_normal((E, d, f)))


def _torch_block(spec, inp, fw, prm):
    """Independent block in torch float64: routing and kept set fixed from the forward."""
    x, g1, b1, Wqkv, Wo, g2, b2, Wg, W1, W2 = prm
    B, S, d, H = spec.B, spec.S, spec.d, spec.heads
    hd = d // H
    a = torch.nn.functional.layer_norm(x, (d,), g1, b1, eps=BO.LN_EPS)
    q, k, v = (a @ Wqkv.T).split(d, dim=1)
    sh = lambda t: t.reshape(B, S, H, hd).transpose(1, 2)
    o = torch.nn.functional.scaled_dot_product_attention(sh(q), sh(k), sh(v), is_causal=True)
    h = x + o.transpose(1, 2).reshape(B * S, d) @ Wo.T
    m = torch.nn.functional.layer_norm(h, (d,), g2, b2, eps=BO.LN_EPS)
    p = torch.softmax(m @ Wg.T, dim=1)
    mw = fw["moe"]
    idx = torch.as_tensor(mw["idx"].astype(np.int64))
    sel = torch.gather(p, 1, idx)
    w = sel / sel.sum(1, keepdim=True)
    kept = torch.as_tensor(mw["slot"] >= 0, dtype=torch.float64)
    y = torch.zeros_like(m)
    for r in range(spec.moe.k):
        for e in range(spec.moe.E):
            msk = (idx[:, r] == e).to(torch.float64) * kept[:, r] * w[:, r]
            y = y + msk[:, None] * (torch.nn.functional.gelu(m @ W1[e].T, approximate="tanh") @ W2[e].T)
    return h + y


def test_block_gradients_match_torch_autograd():
    spec = _spec()
    inp = _inputs(spec, 11)
    fw = BO.block_forward(spec, inp, exact_logits=True)
    names = ("x", "ln1_g", "ln1_b", "Wqkv", "Wo", "ln2_g", "ln2_b", "Wg", "W1", "W2")
    prm = [torch.tensor(inp[n], requires_grad=True) for n in names]
    out = _torch_block(spec, inp, fw, prm)
    np.testing.assert_allclose(fw["out"], out.detach().numpy(), rtol=1e-11, atol=1e-12)
    (out * torch.tensor(inp["dy"])).sum().backward()
    bw = BO.block_backward(spec, inp, fw)
    got = dict(x=bw["dx"], ln1_g=bw["dln1_g"], ln1_b=bw["dln1_b"], Wqkv=bw["dWqkv"], Wo=bw["dWo"],
               ln2_g=bw["dln2_g"], ln2_b=bw["dln2_b"], Wg=bw["moe"]["dWg"], W1=bw["moe"]["dW1"], W2=bw["moe"]["dW2"])
    for n, t in zip(names, prm):
        np.testing.assert_allclose(got[n], t.grad.numpy(), rtol=1e-9, atol=1e-11, err_msg=n)


def test_block_chunked_routing_equals_unchunked():
    """Batch partitions with capacity carry route exactly like the whole batch (Sec. 2.3)."""
    spec = _spec(B=4, S=8)
    inp = _inputs(spec, 12)
    fw = BO.block_forward(spec, inp)
    mw = fw["moe"]
    carry = np.zeros(spec.moe.E, np.int64)
    T = spec.B * spec.S
    for c in range(4):
        sl = slice(c * T // 4, (c + 1) * T // 4)
        part = M.layer_forward(spec.moe, {**fw["moe_inp"], "x": fw["m_in"][sl]}, carry=carry, C=mw["C"])
        np.testing.assert_array_equal(part["slot"], mw["slot"][sl])
        np.testing.assert_allclose(part["y"], mw["y"][sl], rtol=1e-13, atol=1e-14)
        carry = part["fill"]


def _bf16_spec():
    sp = _spec(B=2, S=16, d=32, H=2, E=4, k=2, f=48)
    sp.moe.dtype = "bf16"
    return sp


def _is_bf16(a):
    a = np.asarray(a, np.float64)
    return np.array_equal(BO.round_bf16_f64(a), a)


def test_bf16_block_stores_bf16_activations():
    """A bf16 block's stored activations are bf16 values; the float32 block's are not."""
    spec = _bf16_spec()
    inp = {k: (BO.round_bf16_f64(v) if isinstance(v, np.ndarray) else v) for k, v in _inputs(spec, 13).items()}
    fw = BO.block_forward(spec, inp)
    for n in ("a", "q", "k", "v", "o", "h", "m_in"):
        assert _is_bf16(fw[n]), n
    raw = BO.block_forward(spec, inp, round_acts=False)
    for n in ("a", "q", "o", "h"):
        assert not _is_bf16(raw[n]), n


def test_bf16_block_rounding_stays_within_bf16_error():
    """Rounding the stored activations moves the block output by bf16-sized amounts only."""
    spec = _bf16_spec()
    inp = {k: (BO.round_bf16_f64(v) if isinstance(v, np.ndarray) else v) for k, v in _inputs(spec, 14).items()}
    fw = BO.block_forward(spec, inp, exact_logits=True)
    raw = BO.block_forward(spec, inp, round_acts=False, exact_logits=True)
    np.testing.assert_array_equal(fw["moe"]["idx"], raw["moe"]["idx"])
    for n in ("h", "m", "out"):
        err = np.abs(fw[n] - raw[n]).max() / np.abs(raw[n]).max()
        assert 0 < err < 2.0 ** -6, (n, err)


def test_block_forward_tokens_matches_block_forward():
    """The sampled-token form equals the whole-batch block on rows whose choices are all kept."""
    spec = _bf16_spec()
    spec.moe.cf_num, spec.moe.cf_den = 4, 1          # capacity large enough that nothing drops
    inp = {k: (BO.round_bf16_f64(v) if isinstance(v, np.ndarray) else v) for k, v in _inputs(spec, 15).items()}
    fw = BO.block_forward(spec, inp)
    assert (fw["moe"]["slot"] >= 0).all()
    pos = [0, 5, 15, 9]
    got = BO.block_forward_tokens(spec, inp, 1, pos)
    rows = [spec.S + p for p in pos]
    for n in ("h", "m_in", "out"):
        np.testing.assert_allclose(got[n], fw[n][rows], rtol=1e-12, atol=1e-12, err_msg=n)
    np.testing.assert_array_equal(got["idx"], fw["moe"]["idx"][rows])
    np.testing.assert_array_equal(got["logits"], fw["moe"]["logits"][rows])
