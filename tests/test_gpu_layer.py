"""GPU parity of the MoE layer (forward + backward) against the CPU oracle,
through the C ABI.  Routing (logits to 1 ulp, idx, slot, fill, dropped sets)
must match bit for bit; floats within the normwise tolerance of the workload's
dtype (1e-5 float32, 2e-2 bf16).
"""
from dataclasses import replace

import numpy as np
import pytest

from oracle import moe_oracle as O
from synth import LayerSpec, layer_inputs, layer_spec
from tests.gpu_harness import (TOL, assert_close, bf16_ulp, ebuf, host, kept_rows, ksplit_xcds, log, nan_fill,
                               run_layer, spec_C, to_dev)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def L():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    from paper_2404_19429_amd import lancet_moe
    return lancet_moe


def _s(name, **kw):
    base = dict(name=name, T=1000, d=256, f=512, E=8, k=2, cf_num=5, cf_den=4, dtype="bf16", act="gelu_tanh",
                renorm=1, seed=11)
    base.update(kw)
    return LayerSpec(**base)


SMALL = {
    "c1_tiny_fp32": layer_spec(1),
    "bf16_T1000_d256_f512_E8": _s("a"),
    "bf16_zipf_T777_d128_f192_E16_drops": _s("b", T=777, d=128, f=192, E=16, cf_num=1, cf_den=1, zipf_s=1.2, seed=12),
    "bf16_E64_T600_d64_f128_zipf": _s("c", T=600, d=64, f=128, E=64, cf_num=1, cf_den=1, zipf_s=1.2, seed=13),
    "bf16_top1_relu_T512": _s("d", T=512, d=128, f=256, E=4, k=1, renorm=0, act="relu", seed=14),
    "f32_k3_erf_T300_d40_f24_drops": _s("e", T=300, d=40, f=24, E=5, k=3, cf_num=1, cf_den=2, dtype="f32",
                                        act="gelu_erf", seed=15),
    "bf16_G4_T640_d128_f128_E8": _s("f", T=640, d=128, f=128, E=8, G=4, seed=16),
    "f32_top1_E2_T129": _s("g", T=129, d=16, f=8, E=2, k=1, renorm=0, act="relu", dtype="f32", cf_num=1,
                           cf_den=1, seed=17),
    # the largest top-k and expert count the library takes (k = 8 of 64 experts), with drops
    "bf16_k8_E64_T300_d128_f64_drops": _s("h", T=300, d=128, f=64, E=64, k=8, cf_num=1, cf_den=2, seed=18),
}


def _check_layer(L, spec):
    inp = layer_inputs(spec)
    C = spec_C(spec)
    tol = TOL[spec.dtype]
    log(f"[layer] {spec.name}: T={spec.T} d={spec.d} f={spec.f} E={spec.E} k={spec.k} C={C} {spec.dtype}")
    fw = O.layer_forward(spec, inp)
    bw = O.layer_backward(spec, inp, fw)
    log(f"[layer] {spec.name}: oracle done")
    b, _ = run_layer(L, spec, inp, C)
    log(f"[layer] {spec.name}: GPU step done")
    fill = fw["fill"]

    np.testing.assert_array_max_ulp(host(b.logits), fw["logits"], maxulp=1)
    np.testing.assert_array_equal(host(b.idx), fw["idx"])
    np.testing.assert_array_equal(host(b.slot), fw["slot"])
    np.testing.assert_array_equal(host(b.fill), fill)
    assert_close("w", host(b.w), fw["w"], 1e-5)
    np.testing.assert_array_equal(kept_rows(ebuf(b, "send_buf"), fill), kept_rows(fw["buf"], fill))
    for name in ("H", "A", "O"):
        assert_close(name, kept_rows(ebuf(b, name), fill), kept_rows(fw[name], fill), tol)
    assert_close("y", host(b.y), fw["y"], tol)
    for name in ("dO", "dH"):
        assert_close(name, kept_rows(ebuf(b, name), fill), kept_rows(bw[name], fill), tol)
    assert_close("dXe", kept_rows(ebuf(b, "dXe"), fill), kept_rows(bw["dX"], fill), tol)
    assert_close("dlogits", host(b.dlogits), bw["dlogits"], tol)
    assert_close("dx", host(b.dx), bw["dx"], tol)
    assert_close("dW1", host(b.dW1), bw["dW1"], tol)
    assert_close("dW2", host(b.dW2), bw["dW2"], tol)
    assert_close("dWg", host(b.dWg), bw["dWg"], tol)
    return b


@pytest.mark.parametrize("case", list(SMALL))
def test_layer_matches_oracle(L, case):
    _check_layer(L, SMALL[case])


def test_layer_is_deterministic_and_dw_stream_independent(L):
    spec = SMALL["bf16_zipf_T777_d128_f192_E16_drops"]
    inp = layer_inputs(spec)
    C = spec_C(spec)
    b1, _ = run_layer(L, spec, inp, C)
    side = torch.cuda.Stream()
    b2, _ = run_layer(L, spec, inp, C, dw_stream=side)
    fill = host(b1.fill)
    for name in ("logits", "idx", "w", "slot", "fill", "y", "dlogits", "dx", "dW1", "dW2", "dWg"):
        np.testing.assert_array_equal(host(getattr(b1, name)), host(getattr(b2, name)), err_msg=name)
    for name in ("send_buf", "H", "A", "O", "dO", "dH", "dXe"):
        np.testing.assert_array_equal(kept_rows(ebuf(b1, name), fill),
                                      kept_rows(ebuf(b2, name), fill), err_msg=name)


def test_product_timing_counts_every_product_and_leaves_results_unchanged(L):
    """moe_product_timing: one event pair per expert product of the step
    (six products, positive durations), nothing recorded once it is off, and
    every output bit for bit the same as without timing."""
    spec = SMALL["bf16_zipf_T777_d128_f192_E16_drops"]
    inp = layer_inputs(spec)
    C = spec_C(spec)
    b0, _ = run_layer(L, spec, inp, C)
    L.moe_product_timing(True)
    try:
        b1, _ = run_layer(L, spec, inp, C)
        ms, counts = L.moe_product_times()
    finally:
        L.moe_product_timing(False)
    log(f"[timing] {dict(zip(L.PRODUCTS, np.round(ms, 4)))}")
    assert counts.tolist() == [1] * len(L.PRODUCTS)
    assert np.all(ms > 0)
    run_layer(L, spec, inp, C)
    ms2, counts2 = L.moe_product_times()
    assert counts2.tolist() == [0] * len(L.PRODUCTS) and np.all(ms2 == 0)
    fill = host(b0.fill)
    for name in ("y", "dlogits", "dx", "dW1", "dW2", "dWg"):
        np.testing.assert_array_equal(host(getattr(b0, name)), host(getattr(b1, name)), err_msg=name)
    for name in ("H", "A", "O", "dO", "dH", "dXe"):
        np.testing.assert_array_equal(kept_rows(ebuf(b0, name), fill), kept_rows(ebuf(b1, name), fill),
                                      err_msg=name)


def _unpack_weights(t, E, R, X):
    """[E][R][X] packed (16 x 32 blocks) bf16 matrices as row-major numpy."""
    return host(t).reshape(E, R // 16, X // 32, 16, 32).transpose(0, 1, 3, 2, 4).reshape(E, R, X)


def test_packed_weight_gradients_equal_row_major(L):
    """wpacked = 1: dW1/dW2 are the same values as the row-major gradients,
    bit for bit, stored in the blocked layout of the packed weights."""
    spec = SMALL["bf16_zipf_T777_d128_f192_E16_drops"]
    inp = layer_inputs(spec)
    C = spec_C(spec)
    b, dev = run_layer(L, spec, inp, C)
    cfg = L.make_cfg(spec.T, spec.d, spec.f, spec.E, spec.k, C, spec.G, spec.dtype, spec.act, spec.renorm,
                     wpacked=1)
    dW1p, dW2p, dWg = torch.full_like(b.dW1, float("nan")), torch.full_like(b.dW2, float("nan")), b.dWg.clone()
    L.moe_bwd_dw(cfg, dev["x"], b.dlogits, b.carry, b.fill, b.send_buf, b.A, b.dO, b.dH, dW1p, dW2p, dWg, b.ws_dw)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(_unpack_weights(dW1p, spec.E, spec.f, spec.d), host(b.dW1).reshape(spec.E, spec.f, spec.d))
    np.testing.assert_array_equal(_unpack_weights(dW2p, spec.E, spec.d, spec.f), host(b.dW2).reshape(spec.E, spec.d, spec.f))
    np.testing.assert_array_equal(host(dWg), host(b.dWg))


def _partitioned_forward(L, spec, inp, dev, C, n, ksplit):
    """The layer forward in n batch partitions through the C ABI, each
    dispatch continuing from the capacity the previous partitions used."""
    Tc = spec.T // n
    cfg = L.make_cfg(Tc, spec.d, spec.f, spec.E, spec.k, C, 1, spec.dtype, spec.act, spec.renorm, ksplit=ksplit)
    b = L.alloc_layer(L.make_cfg(spec.T, spec.d, spec.f, spec.E, spec.k, C, 1, spec.dtype, spec.act, spec.renorm))
    nan_fill(b)
    bias = None if inp.get("bias") is None else torch.as_tensor(inp["bias"], dtype=torch.float32).cuda()
    fills = [torch.zeros(spec.E, dtype=torch.int32, device="cuda")]
    ws = torch.empty(max(16, L.moe_workspace_bytes(cfg, L.MOE_CALL_DISPATCH)), dtype=torch.uint8, device="cuda")
    L.moe_pack_weights(cfg, dev["W1"], dev["W2"], b.W1p, b.W2p)
    for i in range(n):
        sl = slice(i * Tc, (i + 1) * Tc)
        xi = dev["x"][sl]
        L.moe_gate_topk(cfg, xi, dev["Wg"], bias, b.logits[sl], b.idx[sl], b.w[sl])
        fills.append(torch.empty(spec.E, dtype=torch.int32, device="cuda"))
        L.moe_dispatch(cfg, xi, b.idx[sl], fills[i], fills[i + 1], b.slot[sl], b.send_buf, ws)
        L.moe_expert_ffn_fwd(cfg, b.send_buf, fills[i], fills[i + 1], b.W1p, b.W2p, b.H, b.A, b.O, b.ws_ffn)
        L.moe_combine(cfg, b.O, b.idx[sl], b.slot[sl], b.w[sl], b.y[sl])
    torch.cuda.synchronize()
    return b, fills


def test_batch_partitions_with_capacity_carry_equal_unpartitioned(L):
    """Four batch partitions, each continuing from the capacity the previous ones
    used: routing and drops equal the unpartitioned layer (Sec. 2.3), and with
    ksplit = 0 (every output element one K sum in order) every kept row of
    every buffer and the output are bitwise the unpartitioned ones."""
    spec = _s("chunks", T=1024, d=128, f=256, E=8, cf_num=1, cf_den=1, zipf_s=0.8, seed=21)
    inp = layer_inputs(spec)
    C = spec_C(spec)
    fw = O.layer_forward(spec, inp)
    full, dev = run_layer(L, spec, inp, C, backward=False, ksplit=0)
    b, fills = _partitioned_forward(L, spec, inp, dev, C, 4, ksplit=0)
    np.testing.assert_array_equal(host(b.slot), fw["slot"])
    np.testing.assert_array_equal(host(fills[-1]), fw["fill"])
    fill = fw["fill"]
    for name in ("send_buf", "H", "A", "O"):
        np.testing.assert_array_equal(kept_rows(ebuf(b, name), fill), kept_rows(ebuf(full, name), fill), err_msg=name)
    np.testing.assert_array_equal(host(b.y), host(full.y))
    # carries are the per-partition fills; every partition filled a contiguous, disjoint row range
    f = np.stack([host(t) for t in fills])
    assert np.all(np.diff(f, axis=0) >= 0)


# A shape whose plain-store products (expert_out, dXe: 16 experts x 8 column
# tiles) leave a short last round on every XCD of the 256-CU device, so with
# ksplit = 1 their last tiles' K sums are split over several blocks and added
# by the fix-up kernel.
KSPLIT_CASE = _s("ksplit", T=4096, d=2048, f=512, E=16, seed=32)


def _ksplit_bound(a_rows, b_mat, o1, o2):
    """Largest allowed |o1 - o2| per element for two float32 evaluations of the
    same K-term dot products o = a b^T, each rounded once to bf16: each float
    sum is within gamma_K sum|a||b| of the exact one (gamma_K = K u / (1 - K u),
    u = 2^-24), so the two sums differ by at most twice that, and each rounding
    adds at most half a bf16 ulp of its value."""
    K = a_rows.shape[1]
    u = 2.0 ** -24
    gamma = K * u / (1 - K * u)
    S = np.abs(np.asarray(a_rows, np.float64)) @ np.abs(np.asarray(b_mat, np.float64)).T
    return 2 * gamma * S + bf16_ulp(np.maximum(np.abs(o1), np.abs(o2)))


def test_ksplit_products_match_oracle_and_whole_k_sums(L):
    """ksplit = 1 on a case that splits the last round's K sums on every XCD:
    every output against the oracle; expert_out, dXe and y against the run with
    ksplit = 0 within the derived bound of float summation order; everything
    before the split products bitwise."""
    spec = KSPLIT_CASE
    inp = layer_inputs(spec)
    C = spec_C(spec)
    fw = O.layer_forward(spec, inp)
    fill = fw["fill"]
    n_split = ksplit_xcds(np.zeros(spec.E), fill, C, spec.d)
    log(f"[ksplit] XCDs whose last round is K-split: {n_split} of 8")
    assert n_split >= 4, "the case no longer exercises the K-split schedule"
    b1 = _check_layer(L, spec)                         # ksplit = 1 (the default)
    b0, _ = run_layer(L, spec, inp, C, ksplit=0)
    for name in ("logits", "idx", "w", "slot", "fill"):
        np.testing.assert_array_equal(host(getattr(b1, name)), host(getattr(b0, name)), err_msg=name)
    for name in ("send_buf", "H", "A", "dO", "dH"):
        np.testing.assert_array_equal(kept_rows(ebuf(b1, name), fill), kept_rows(ebuf(b0, name), fill), err_msg=name)
    W1 = inp["W1"].astype(np.float64)
    W2 = inp["W2"].astype(np.float64)
    A1, dH1 = ebuf(b1, "A"), ebuf(b1, "dH")
    O1, O0 = ebuf(b1, "O"), ebuf(b0, "O")
    X1, X0 = ebuf(b1, "dXe"), ebuf(b0, "dXe")
    boundO = np.zeros(O1.shape, np.float64)
    worst = 0.0
    for e in range(spec.E):
        n = int(fill[e])
        bo = _ksplit_bound(A1[e, :n], W2[e], O1[e, :n], O0[e, :n])
        assert np.all(np.abs(O1[e, :n] - O0[e, :n]) <= bo), f"expert_out of expert {e}"
        bx = _ksplit_bound(dH1[e, :n], W1[e].T, X1[e, :n], X0[e, :n])
        assert np.all(np.abs(X1[e, :n] - X0[e, :n]) <= bx), f"dXe of expert {e}"
        boundO[e, :n] = bo
        worst = max(worst, float(np.max(np.abs(O1[e, :n] - O0[e, :n]) / bo)))
    log(f"[ksplit] largest expert_out difference / bound: {worst:.3f}")
    # y_t = sum_r w_r O_r in float, rounded once to bf16: the expert_out bounds
    # carried through the weights, the float sums' own rounding, one bf16 rounding
    idx, slot, w = fw["idx"], fw["slot"], host(b1.w).astype(np.float64)
    y1, y0 = host(b1.y), host(b0.y)
    by = np.zeros(y1.shape, np.float64)
    mag = np.zeros(y1.shape, np.float64)
    for r in range(spec.k):
        kept = slot[:, r] >= 0
        e, s_ = idx[kept, r], slot[kept, r]
        by[kept] += w[kept, r][:, None] * boundO[e, s_]
        mag[kept] += w[kept, r][:, None] * np.maximum(np.abs(O1[e, s_]), np.abs(O0[e, s_]))
    by += bf16_ulp(np.maximum(np.abs(y1), np.abs(y0))) + 2.0 ** -22 * mag
    assert np.all(np.abs(y1 - y0) <= by), "y"


def test_zero_tokens(L):
    spec = _s("empty", T=0, d=64, f=64, E=4)
    C = 8
    cfg = L.make_cfg(0, spec.d, spec.f, spec.E, spec.k, C, 1, "bf16", "gelu_tanh", 1)
    b = L.alloc_layer(cfg)
    nan_fill(b)
    carry = torch.tensor([0, 3, 8, 1], dtype=torch.int32, device="cuda")
    b.carry.copy_(carry)
    W = torch.zeros(spec.E, spec.f, spec.d, dtype=torch.bfloat16, device="cuda")
    x = torch.zeros(0, spec.d, dtype=torch.bfloat16, device="cuda")
    L.moe_gate_topk(cfg, x, torch.zeros(4, 64, dtype=torch.bfloat16, device="cuda"), None, b.logits, b.idx, b.w)
    L.moe_dispatch(cfg, x, b.idx, b.carry, b.fill, b.slot, b.send_buf, b.ws_dispatch)
    # rows [carry, fill) are empty, so the experts and the dW products see no rows
    L.moe_pack_weights(cfg, W, W.clone(), b.W1p, b.W2p)
    L.moe_expert_ffn_fwd(cfg, b.send_buf, b.carry, b.fill, b.W1p, b.W2p, b.H, b.A, b.O, b.ws_ffn)
    L.moe_combine(cfg, b.O, b.idx, b.slot, b.w, b.y)
    L.moe_bwd_dw(cfg, x, b.dlogits, b.carry, b.fill, b.send_buf, b.A, b.dO, b.dH, b.dW1, b.dW2, b.dWg, b.ws_dw)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(b.fill), [0, 3, 8, 1])
    assert np.all(host(b.dW1) == 0) and np.all(host(b.dW2) == 0) and np.all(host(b.dWg) == 0)


# ------------------------------------------------------------- full-size workloads
@pytest.mark.timeout(600)
@pytest.mark.parametrize("n", [2, 3, 4])
def test_full_size_config_matches_oracle(L, n):
    """The workloads at full size, every element of every output against the
    oracle: routing bit-exact, every kept row of H, A, expert_out, dO, dH, dXe,
    the output, dlogits, dx, dW1, dW2 and dWg within the bf16 tolerance."""
    spec = layer_spec(n)
    log(f"[full] config {n}: {spec.name}")
    b = _check_layer(L, spec)
    fill = host(b.fill)
    C = spec_C(spec)
    log(f"[full] config {n}: kept {int(fill.sum())} of {spec.k * spec.T}; K-split XCDs in the plain-store "
        f"products: {ksplit_xcds(np.zeros(spec.E), fill, C, spec.d)} of 8")
    if n == 4:
        assert int(fill.sum()) < spec.k * spec.T, "the Zipf-skewed workload must drop tokens"
    for e in [e for e in range(spec.E) if fill[e] == 0][:8]:
        assert torch.count_nonzero(b.dW1[e]).item() == 0 and torch.count_nonzero(b.dW2[e]).item() == 0, e
