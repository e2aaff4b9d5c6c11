"""GPU parity of batch-prioritized routing (moe_dispatch_bpr) against the
oracle, through the C ABI.  The visiting order, slots, fills and dispatched
rows must match bit for bit; the layer built on them (experts, combine,
backward) within the workload's normwise tolerance (1e-5 float32, 2e-2 bf16).
"""
import numpy as np
import pytest

from oracle import moe_oracle as O
from synth import LayerSpec, layer_inputs, layer_spec
from tests.gpu_harness import TOL, assert_close, ebuf, expert_host, host, kept_rows, log, run_layer, spec_C, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def L():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    from paper_2404_19429_amd import lancet_moe
    return lancet_moe


def _s(name, **kw):
    base = dict(name=name, T=1000, d=256, f=512, E=8, k=2, cf_num=1, cf_den=1, dtype="bf16", act="gelu_tanh",
                renorm=1, seed=21)
    base.update(kw)
    return LayerSpec(**base)


SMALL = {
    "bf16_T1000_E8_k2_cf1": _s("a"),
    "bf16_zipf_T777_E16_drops": _s("b", T=777, d=128, f=192, E=16, zipf_s=1.2, seed=22),
    "bf16_top1_T513_E4_cf3/4": _s("c", T=513, d=128, f=256, E=4, k=1, renorm=0, act="relu", cf_num=3, cf_den=4,
                                  seed=23),
    "f32_k3_T300_E5_cf1/2": _s("d", T=300, d=40, f=24, E=5, k=3, cf_den=2, dtype="f32", act="gelu_erf", seed=24),
    "f32_T37_E2_top1": _s("e", T=37, d=16, f=8, E=2, k=1, renorm=0, act="relu", dtype="f32", seed=25),
    "f32_T1_E4": _s("f", T=1, d=64, f=64, E=4, dtype="f32", seed=26),
    "bf16_G4_T640_E8_cf3/4": _s("h", T=640, d=128, f=128, E=8, G=4, cf_num=3, cf_den=4, seed=28),
}


@pytest.mark.parametrize("case", list(SMALL))
def test_bpr_layer_matches_oracle(L, case):
    spec = SMALL[case]
    inp = layer_inputs(spec)
    C = spec_C(spec)
    tol = TOL[spec.dtype]
    log(f"[bpr layer] {case}: T={spec.T} d={spec.d} f={spec.f} E={spec.E} k={spec.k} C={C} {spec.dtype}")
    fw = O.layer_forward(spec, inp, routing="bpr")
    bw = O.layer_backward(spec, inp, fw)
    b, _ = run_layer(L, spec, inp, C, routing="bpr")
    fill = fw["fill"]
    np.testing.assert_array_equal(host(b.idx), fw["idx"])
    np.testing.assert_array_equal(host(b.order)[:spec.T], fw["order"])
    np.testing.assert_array_equal(host(b.slot), fw["slot"])
    np.testing.assert_array_equal(host(b.fill), fill)
    np.testing.assert_array_equal(kept_rows(ebuf(b, "send_buf"), fill), kept_rows(fw["buf"], fill))
    for name in ("H", "A", "O"):
        assert_close(name, kept_rows(ebuf(b, name), fill), kept_rows(fw[name], fill), tol)
    assert_close("y", host(b.y), fw["y"], tol)
    assert_close("dlogits", host(b.dlogits), bw["dlogits"], tol)
    assert_close("dx", host(b.dx), bw["dx"], tol)
    assert_close("dW1", host(b.dW1), bw["dW1"], tol)
    assert_close("dW2", host(b.dW2), bw["dW2"], tol)
    assert_close("dWg", host(b.dWg), bw["dWg"], tol)


def _gate_and_bpr(L, spec, T=None, with_order=True):
    inp = layer_inputs(spec, with_weights=False)
    T = spec.T if T is None else T
    C = max(1, spec_C(spec, T))          # (C >= 1 is required even for an empty batch)
    dt = torch.bfloat16 if spec.dtype == "bf16" else torch.float32
    cfg = L.make_cfg(T, spec.d, spec.f, spec.E, spec.k, C, spec.G, spec.dtype, spec.act, spec.renorm)
    x, Wg = to_dev(inp["x"][:T], dt), to_dev(inp["Wg"], dt)
    bias = None if inp["bias"] is None else torch.as_tensor(inp["bias"]).cuda()
    i32 = dict(dtype=torch.int32, device="cuda")
    logits = torch.empty(T, spec.E, dtype=torch.float32, device="cuda")
    idx, slot = torch.empty(T, spec.k, **i32), torch.empty(T, spec.k, **i32)
    w = torch.empty(T, spec.k, dtype=torch.float32, device="cuda")
    fill = torch.full((spec.E,), -7, **i32)
    order = torch.full((max(T, 1),), -7, **i32) if with_order else None
    send = torch.full((L.expert_numel(cfg, spec.d),), float("nan"), dtype=dt, device="cuda")
    ws = torch.empty(L.moe_workspace_bytes(cfg, L.MOE_CALL_DISPATCH_BPR), dtype=torch.uint8, device="cuda")
    L.moe_gate_topk(cfg, x, Wg, bias, logits, idx, w)
    L.moe_dispatch_bpr(cfg, x, logits, idx, fill, slot, send, order, ws)
    torch.cuda.synchronize()
    return inp, cfg, C, dict(idx=host(idx), slot=host(slot), fill=host(fill),
                             order=None if order is None else host(order)[:T], send=send, x=x)


@pytest.mark.parametrize("n", [2, 4])
def test_bpr_full_size(L, n):
    """The 8192-token layer and the Zipf-skewed 32768-token, 64-expert one
    (where capacity drops most): order, slots, fills bit for bit, and every
    kept row of the send buffer is its token's row."""
    spec = layer_spec(n)
    log(f"[bpr full] {spec.name}")
    inp, cfg, C, g = _gate_and_bpr(L, spec)
    logits = O.gate_logits(inp["x"], inp["Wg"], inp["bias"])
    idx = O.topk_route(logits, spec.k)
    np.testing.assert_array_equal(g["idx"], idx)
    slot, fill, order = O.assign_slots_bpr(idx, spec.E, C, O.bpr_importance(logits, idx))
    np.testing.assert_array_equal(g["order"], order)
    np.testing.assert_array_equal(g["slot"], slot)
    np.testing.assert_array_equal(g["fill"], fill)
    if n == 4:
        assert int(fill.sum()) < spec.k * spec.T, "the skewed workload must drop tokens"
    buf = expert_host(g["send"], cfg, spec.d)
    t, r = np.nonzero(slot >= 0)
    np.testing.assert_array_equal(buf[idx[t, r], slot[t, r]], host(g["x"])[t])


def test_bpr_without_order_output_and_repeat(L):
    spec = SMALL["bf16_zipf_T777_E16_drops"]
    _, _, _, g1 = _gate_and_bpr(L, spec, with_order=True)
    _, _, _, g2 = _gate_and_bpr(L, spec, with_order=False)
    np.testing.assert_array_equal(g1["slot"], g2["slot"])
    np.testing.assert_array_equal(g1["fill"], g2["fill"])


def test_bpr_zero_tokens(L):
    spec = SMALL["f32_T1_E4"]
    _, _, _, g = _gate_and_bpr(L, spec, T=0)
    np.testing.assert_array_equal(g["fill"], np.zeros(spec.E, np.int32))


def test_bpr_many_tiles(L):
    """70 000 tokens: 18 sorted tiles of 4096, merged in two groups."""
    spec = _s("g", T=70000, d=64, f=64, E=8, k=2, cf_num=3, cf_den=4, seed=27)
    log(f"[bpr tiles] T={spec.T}")
    inp, cfg, C, g = _gate_and_bpr(L, spec)
    logits = O.gate_logits(inp["x"], inp["Wg"], inp["bias"])
    idx = O.topk_route(logits, spec.k)
    slot, fill, order = O.assign_slots_bpr(idx, spec.E, C, O.bpr_importance(logits, idx))
    np.testing.assert_array_equal(g["order"], order)
    np.testing.assert_array_equal(g["slot"], slot)
    np.testing.assert_array_equal(g["fill"], fill)


def test_bpr_all_equal_importance_keeps_token_order(L):
    """Every token's logits a permutation of one vector: one importance for all
    9000 tokens, so the order is token order and the slots equal moe_dispatch's."""
    T, E, k, d = 9000, 8, 2, 64
    rng = np.random.default_rng(29)
    base = rng.standard_normal(E).astype(np.float32)
    logits = np.stack([rng.permutation(base) for _ in range(T)])
    idx = O.topk_route(logits, k)
    C = O.capacity(T, E, k, 1, 1)
    cfg = L.make_cfg(T, d, d, E, k, C, 1, "bf16", "gelu_tanh", 1)
    i32 = dict(dtype=torch.int32, device="cuda")
    x = torch.zeros(T, d, dtype=torch.bfloat16, device="cuda")
    lg = torch.from_numpy(logits).cuda()
    ix = torch.from_numpy(idx).cuda()
    fill, slot, order = torch.empty(E, **i32), torch.empty(T, k, **i32), torch.empty(T, **i32)
    send = torch.empty(L.expert_numel(cfg, d), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(L.moe_workspace_bytes(cfg, L.MOE_CALL_DISPATCH_BPR), dtype=torch.uint8, device="cuda")
    L.moe_dispatch_bpr(cfg, x, lg, ix, fill, slot, send, order, ws)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(order), np.arange(T))
    s_tok, f_tok = O.assign_slots(idx, E, C)
    np.testing.assert_array_equal(host(slot), s_tok)
    np.testing.assert_array_equal(host(fill), f_tok)
