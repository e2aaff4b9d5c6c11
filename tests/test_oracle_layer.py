"""Pins for the oracle's expert FFN, combine and backward (CPU only).

References used here are independent of the oracle's buffer-based code path:
a dense-masked formula (every token through every expert, masked by the
routing), identity-expert special cases, central finite differences in float64
and torch CPU float64 autograd on the dense-masked formula.
"""
import math
from types import SimpleNamespace

import numpy as np
import pytest
import torch

from oracle import moe_oracle as O


def _spec(T=48, d=8, f=16, E=4, k=2, num=5, den=4, act="gelu_tanh", renorm=1):
    return SimpleNamespace(T=T, d=d, f=f, E=E, k=k, cf_num=num, cf_den=den, act=act, renorm=renorm)


def _inputs(spec, seed, skew=0.0, w_std=0.3):
    rng = np.random.default_rng(seed)
    inp = dict(
        x=rng.standard_normal((spec.T, spec.d)),
        Wg=rng.standard_normal((spec.E, spec.d)) * 0.5,
        W1=rng.standard_normal((spec.E, spec.f, spec.d)) * w_std,
        W2=rng.standard_normal((spec.E, spec.d, spec.f)) * w_std,
        dy=rng.standard_normal((spec.T, spec.d)),
        bias=None,
    )
    if skew:
        inp["bias"] = np.linspace(skew, 0.0, spec.E)       # expert 0 overloaded
    return inp


def _dense_masked_forward(spec, inp, fw):
    """y_t = sum_e M[t,e] W[t,e] FFN_e(x_t): every token through every expert
    with numpy matmul, then masked by which (t, e) pairs were kept."""
    x = inp["x"]
    T, E = x.shape[0], spec.E
    M = np.zeros((T, E))
    Wt = np.zeros((T, E))
    for t in range(T):
        for r in range(spec.k):
            if fw["slot"][t, r] >= 0:
                M[t, fw["idx"][t, r]] = 1.0
                Wt[t, fw["idx"][t, r]] = fw["w"][t, r]
    y = np.zeros_like(x)
    for e in range(E):
        h = x @ inp["W1"][e].T
        y += (M[:, e] * Wt[:, e])[:, None] * (O.act(h, spec.act) @ inp["W2"][e].T)
    return y


@pytest.mark.parametrize("act,renorm,k,skew", [("relu", 0, 1, 0.0), ("gelu_tanh", 1, 2, 0.0),
                                               ("gelu_tanh", 1, 2, 3.0), ("gelu_erf", 0, 2, 2.0),
                                               ("relu", 1, 3, 1.0)])
def test_forward_matches_dense_masked(act, renorm, k, skew):
    spec = _spec(T=64, E=5, k=k, act=act, renorm=renorm, num=1, den=1)
    inp = _inputs(spec, seed=k * 10 + renorm, skew=skew)
    fw = O.layer_forward(spec, inp)
    if skew:
        assert (fw["slot"] < 0).any(), "expected drops with a skewed gate"
    np.testing.assert_allclose(fw["y"], _dense_masked_forward(spec, inp, fw), rtol=1e-12, atol=1e-13)


def test_identity_experts_top1_scale_inputs_by_gate_weight():
    spec = _spec(T=40, d=6, f=6, E=3, k=1, act="identity", renorm=0, num=1, den=1)
    inp = _inputs(spec, seed=3, skew=2.0)
    inp["W1"] = np.tile(np.eye(6), (3, 1, 1))
    inp["W2"] = np.tile(np.eye(6), (3, 1, 1))
    fw = O.layer_forward(spec, inp)
    p = O.softmax(fw["logits"].astype(np.float64))
    kept = fw["slot"][:, 0] >= 0
    assert (~kept).any()
    expect = np.where(kept[:, None], p.max(1)[:, None] * inp["x"], 0.0)
    np.testing.assert_allclose(fw["y"], expect, rtol=1e-14, atol=0)


def test_identity_experts_renorm_no_drops_returns_inputs():
    spec = _spec(T=40, d=6, f=6, E=4, k=2, act="identity", renorm=1, num=4, den=1)
    inp = _inputs(spec, seed=4)
    inp["W1"] = np.tile(np.eye(6), (4, 1, 1))
    inp["W2"] = np.tile(np.eye(6), (4, 1, 1))
    fw = O.layer_forward(spec, inp)
    assert (fw["slot"] >= 0).all()
    np.testing.assert_allclose(fw["y"], inp["x"], rtol=1e-14, atol=1e-15)


def test_all_choices_dropped_gives_zero_row():
    spec = _spec(T=20, E=2, k=1, act="relu", renorm=0, num=1, den=4)    # C = ceil(20/8) = 3
    inp = _inputs(spec, seed=9, skew=5.0)
    fw = O.layer_forward(spec, inp)
    dropped = (fw["slot"] < 0).all(1)
    assert dropped.any()
    assert np.all(fw["y"][dropped] == 0.0)


def test_batch_partition_identity_for_matmul():
    # [X1; X2] W = [X1 W; X2 W] (Operator Partition Pass, partition axis inference)
    rng = np.random.default_rng(0)
    X, W = rng.standard_normal((10, 7)), rng.standard_normal((7, 5))
    np.testing.assert_array_equal(np.vstack([X[:4] @ W, X[4:] @ W]), X @ W)


def test_chunked_forward_equals_unchunked():
    spec = _spec(T=96, E=4, k=2, num=1, den=1)
    inp = _inputs(spec, seed=21, skew=1.5)
    full = O.layer_forward(spec, inp)
    C = full["C"]
    carry = np.zeros(spec.E, np.int64)
    ys = []
    for a in range(0, 96, 24):
        part = {k: (v[a:a + 24] if k in ("x", "dy") else v) for k, v in inp.items()}
        fw = O.layer_forward(spec, part, carry=carry, C=C)
        ys.append(fw["y"])
        np.testing.assert_array_equal(fw["slot"], full["slot"][a:a + 24])
        carry = fw["fill"]
    np.testing.assert_array_equal(carry, full["fill"])
    np.testing.assert_allclose(np.vstack(ys), full["y"], rtol=1e-13, atol=1e-14)


# ------------------------------------------------------------------------ gradients
def _loss(spec, inp, C):
    fw = O.layer_forward(spec, inp, C=C, exact_logits=True)
    return float(np.sum(inp["dy"] * fw["y"])), fw


@pytest.mark.parametrize("act,renorm,k,skew", [("gelu_tanh", 1, 2, 0.0), ("relu", 0, 1, 0.0),
                                               ("gelu_tanh", 1, 2, 3.0), ("gelu_erf", 0, 2, 0.0)])
def test_gradients_match_central_finite_differences(act, renorm, k, skew):
    spec = _spec(T=24, d=6, f=10, E=4, k=k, act=act, renorm=renorm, num=1, den=1)
    inp = _inputs(spec, seed=31 + k + renorm, skew=skew)
    C = O.capacity(spec.T, spec.E, spec.k, spec.cf_num, spec.cf_den)
    _, fw = _loss(spec, inp, C)
    gr = O.layer_backward(spec, inp, fw)
    rng = np.random.default_rng(77)
    h = 1e-6
    checked = 0
    for name, gname in (("x", "dx"), ("Wg", "dWg"), ("W1", "dW1"), ("W2", "dW2")):
        for _ in range(25):
            pos = tuple(rng.integers(0, s) for s in inp[name].shape)
            plus = {**inp, name: inp[name].copy()}
            minus = {**inp, name: inp[name].copy()}
            plus[name][pos] += h
            minus[name][pos] -= h
            lp, fp = _loss(spec, plus, C)
            lm, fm = _loss(spec, minus, C)
            if not (np.array_equal(fp["slot"], fw["slot"]) and np.array_equal(fm["slot"], fw["slot"])
                    and np.array_equal(fp["idx"], fw["idx"]) and np.array_equal(fm["idx"], fw["idx"])):
                continue                                   # routing changed: not differentiable here
            if act == "relu":
                Hs = np.concatenate([fw["H"][e, :fw["fill"][e]].ravel() for e in range(spec.E)])
                if np.min(np.abs(Hs)) < 1e-4:
                    continue
            fd = (lp - lm) / (2 * h)
            an = gr[gname][pos]
            assert abs(fd - an) <= 1e-6 * max(1.0, abs(an)), (name, pos, fd, an)
            checked += 1
    assert checked >= 60


def _torch_dense_loss(spec, inp, fw, params):
    """Independent second reference: dense-masked layer in torch float64 with
    autograd; routing and the kept mask are fixed from the forward."""
    x, Wg, W1, W2 = params
    l = x @ Wg.T
    if inp["bias"] is not None:
        l = l + torch.as_tensor(inp["bias"])
    p = torch.softmax(l, dim=1)
    idx = torch.as_tensor(fw["idx"].astype(np.int64))
    sel = torch.gather(p, 1, idx)
    w = sel / sel.sum(1, keepdim=True) if spec.renorm else sel
    kept = torch.as_tensor(fw["slot"] >= 0, dtype=torch.float64)
    y = torch.zeros_like(x)
    for r in range(spec.k):
        for e in range(spec.E):
            m = (idx[:, r] == e).to(torch.float64) * kept[:, r] * w[:, r]
            h = x @ W1[e].T
            if spec.act == "relu":
                a = torch.relu(h)
            elif spec.act == "gelu_tanh":
                a = torch.nn.functional.gelu(h, approximate="tanh")
            else:
                a = torch.nn.functional.gelu(h)
            y = y + m[:, None] * (a @ W2[e].T)
    return (torch.as_tensor(inp["dy"]) * y).sum()


@pytest.mark.parametrize("act,renorm,k,skew", [("gelu_tanh", 1, 2, 2.0), ("relu", 0, 1, 1.0),
                                               ("gelu_erf", 0, 2, 0.0), ("gelu_tanh", 1, 3, 0.5)])
def test_gradients_match_torch_autograd_dense(act, renorm, k, skew):
    spec = _spec(T=40, d=8, f=12, E=5, k=k, act=act, renorm=renorm, num=1, den=1)
    inp = _inputs(spec, seed=50 + k, skew=skew)
    fw = O.layer_forward(spec, inp, exact_logits=True)
    gr = O.layer_backward(spec, inp, fw)
    params = [torch.tensor(inp[n], dtype=torch.float64, requires_grad=True)
              for n in ("x", "Wg", "W1", "W2")]
    _torch_dense_loss(spec, inp, fw, params).backward()
    for p, n in zip(params, ("dx", "dWg", "dW1", "dW2")):
        np.testing.assert_allclose(gr[n], p.grad.numpy(), rtol=1e-10, atol=1e-12, err_msg=n)


def test_empty_expert_gets_zero_weight_gradient():
    spec = _spec(T=30, E=4, k=1, renorm=0, act="relu", num=1, den=1)
    inp = _inputs(spec, seed=8)
    inp["bias"] = np.array([5.0, 5.0, -50.0, 5.0])        # expert 2 never chosen
    fw = O.layer_forward(spec, inp)
    assert fw["fill"][2] == 0
    gr = O.layer_backward(spec, inp, fw)
    assert np.all(gr["dW1"][2] == 0) and np.all(gr["dW2"][2] == 0)


def test_row_forms_match_layer():
    spec = _spec(T=30, E=3, k=2)
    inp = _inputs(spec, seed=12)
    fw = O.layer_forward(spec, inp)
    bw = O.layer_backward(spec, inp, fw)
    for t in range(spec.T):
        for r in range(spec.k):
            s = fw["slot"][t, r]
            if s < 0:
                continue
            e = fw["idx"][t, r]
            h, a, o = O.expert_row_forward(inp["x"][t], inp["W1"][e], inp["W2"][e], spec.act)
            np.testing.assert_allclose(o, fw["O"][e, s], rtol=1e-12, atol=1e-14)
            dH, dX = O.expert_row_backward(inp["x"][t], bw["dO"][e, s], inp["W1"][e],
                                           inp["W2"][e], spec.act)
            np.testing.assert_allclose(dX, bw["dX"][e, s], rtol=1e-12, atol=1e-14)


def test_gelu_tanh_closed_values():
    assert O.act(np.array([0.0]), "gelu_tanh")[0] == 0.0
    np.testing.assert_allclose(O.act_grad(np.array([0.0]), "gelu_tanh"), 0.5, rtol=1e-15)
    # large |h|: gelu -> relu
    np.testing.assert_allclose(O.act(np.array([12.0, -12.0]), "gelu_tanh"), [12.0, 0.0], atol=1e-12)
    hs = np.linspace(-4, 4, 41)
    num = (O.act(hs + 1e-6, "gelu_tanh") - O.act(hs - 1e-6, "gelu_tanh")) / 2e-6
    np.testing.assert_allclose(O.act_grad(hs, "gelu_tanh"), num, rtol=1e-7, atol=1e-9)
    ref = 0.5 * hs * (1 + np.array([math.erf(v / math.sqrt(2)) for v in hs]))
    np.testing.assert_allclose(O.act(hs, "gelu_erf"), ref, rtol=1e-13, atol=1e-15)


def test_sampled_dw_forms_match_layer():
    spec = _spec(T=60, E=3, k=2, act="gelu_tanh")
    inp = _inputs(spec, seed=13, skew=1.0)
    fw = O.layer_forward(spec, inp)
    bw = O.layer_backward(spec, inp, fw)
    for e in range(spec.E):
        X, dO = O.expert_rows(inp["x"], inp["dy"], fw["idx"], fw["slot"], fw["w"], e)
        n = int(fw["fill"][e])
        np.testing.assert_allclose(X, fw["buf"][e, :n], rtol=0, atol=0)
        np.testing.assert_allclose(dO, bw["dO"][e, :n], rtol=1e-15, atol=0)
        for i in (0, spec.f - 1, 5):
            np.testing.assert_allclose(O.expert_dw1_row(X, dO, inp["W1"][e], inp["W2"][e], spec.act, i),
                                       bw["dW1"][e, i], rtol=1e-11, atol=1e-13)
        for c in (0, spec.f - 1, 7):
            np.testing.assert_allclose(O.expert_dw2_col(X, dO, inp["W1"][e], spec.act, c),
                                       bw["dW2"][e, :, c], rtol=1e-11, atol=1e-13)


def test_idx_override_follows_the_given_choice():
    """idx_override replaces only the top-k choice: its own choice given back
    changes nothing; another choice is followed, with its weights taken from
    the same softmax and the result still equal to the dense-masked formula."""
    spec = _spec(T=40, E=5, k=2, num=1, den=1)
    inp = _inputs(spec, seed=77)
    fw = O.layer_forward(spec, inp)
    same = O.layer_forward(spec, inp, idx_override=fw["idx"])
    for n in ("idx", "w", "slot", "fill", "y"):
        np.testing.assert_array_equal(same[n], fw[n])
    idx2 = fw["idx"].copy()
    idx2[3] = idx2[3][::-1]                       # same experts, other rank order
    third = [e for e in range(spec.E) if e not in idx2[7]][0]
    idx2[7, 1] = third                            # another second choice
    alt = O.layer_forward(spec, inp, idx_override=idx2)
    np.testing.assert_array_equal(alt["idx"], idx2)
    p = O.softmax(fw["logits"].astype(np.float64))
    sel = p[7, idx2[7]]
    np.testing.assert_allclose(alt["w"][7], sel / sel.sum(), rtol=1e-15)
    np.testing.assert_allclose(alt["y"], _dense_masked_forward(spec, inp, alt), rtol=1e-12, atol=1e-13)
    changed = {3, 7}
    keep = [t for t in range(spec.T) if t not in changed and (fw["slot"][t] == alt["slot"][t]).all()]
    np.testing.assert_allclose(alt["y"][keep], fw["y"][keep], rtol=1e-13, atol=1e-14)
