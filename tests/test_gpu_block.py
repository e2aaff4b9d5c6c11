"""GPU parity of the partitioned pre-LN MoE block (forward + backward) through
the C ABI moe_block_chunked.

* Small blocks against the float64 oracle: every stored activation, the
  routing (exact; the logits within tolerance), the block output, every
  intermediate gradient and every weight gradient (normwise bf16 tolerance).
* Partitioning changes nothing: n_chunks partitions and one partition give
  bitwise identical outputs, routing and gradients (capacity carried across
  partitions, Sec. 2.3 "Challenge 1"), with and without token drops; the
  deferred weight-gradient stream gives the same bits as a single stream.
* The full-size block (8 x 2048 tokens, d 2048, 16 heads, 16 experts, d_ff
  8192): partitioned vs unpartitioned bitwise; the MoE layer of all 16384
  tokens against the layer oracle run on the GPU's own MoE input (routing,
  slots and fills bit-exact; the layer output, dm, dlogits, dW1, dW2, dWg as
  whole tensors); two whole sequences through the block oracle (every
  activation and activation gradient of their tokens); identities of the
  backward that hold at any size.

Routing near-ties: the GPU and the oracle see the same bf16 MoE input up to
rare 1-ulp differences upstream, so a token's top-k may legitimately differ
only where two of its top k+1 oracle logits are within twice the observed
logit error; any other difference fails.
"""
import numpy as np
import pytest

from oracle import block_oracle as BO
from oracle import moe_oracle as O
from synth import BLOCK5, block_inputs, block_spec
from tests.gpu_harness import TOL, assert_close, host, log, normwise, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
TOLB = TOL["bf16"]


@pytest.fixture(scope="module")
def L():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    from paper_2404_19429_amd import lancet_moe
    return lancet_moe


def _cfg(L, spec):
    m = spec.moe
    C = O.capacity(spec.B * spec.S, m.E, m.k, m.cf_num, m.cf_den)
    return L.make_block_cfg(spec.B, spec.S, spec.heads, m.f, m.E, m.k, C, m.G, m.act, m.renorm), C


def _upload(L, inp):
    bf = torch.bfloat16
    w = {n: to_dev(inp[n], bf).reshape(-1) for n in L.BLOCK_WEIGHTS}
    return w, to_dev(inp["x"], bf).reshape(-1), to_dev(inp["dy"], bf).reshape(-1)


def run_block(L, spec, dev, n_chunks, passes=3, same_stream=False):
    cfg, C = _cfg(L, spec)
    w, x, dy = dev
    b = L.alloc_block(cfg, n_chunks)
    for n in ("send_buf", "H", "A", "expert_out", "dO", "dH", "dXe"):
        b[n].fill_(float("nan"))  # rows past an expert's fill must never be read
    out, dx = torch.empty_like(x), torch.empty_like(x)
    if same_stream:
        streams = [torch.cuda.current_stream()] * 3
    else:
        streams = [torch.cuda.Stream() for _ in range(3)]
        streams[0].wait_stream(torch.cuda.current_stream())
    log(f"[block] B={spec.B} S={spec.S} d={spec.d} heads={spec.heads} E={spec.moe.E} f={spec.moe.f} C={C} "
        f"n_chunks={n_chunks} passes={passes} same_stream={same_stream}")
    L.moe_block_chunked(cfg, w, b, x, out, dy, dx, b, passes, n_chunks, streams, b["ws"])
    torch.cuda.synchronize()
    b["out"], b["dx"] = out, dx
    return cfg, C, b


def _near_tie(lo, k, eps):
    s = -np.sort(-np.asarray(lo, np.float64), axis=1)[:, :k + 1]
    return (-np.diff(s, axis=1) <= 2 * eps).any(axis=1)


def _check_routing(lg, lo, idx_g, idx_o, k):
    """Logits within tolerance; top-k exact except at near-ties, where the GPU's
    choice must still be a valid top-k of the oracle logits.  Returns the flipped tokens."""
    assert_close("logits", lg, lo, TOLB)
    eps = float(np.abs(lg - lo).max())
    flips = np.nonzero((idx_g != idx_o).any(axis=1))[0]
    tie = _near_tie(lo, k, eps)
    log(f"  logit error {eps:.2e}, near-tie tokens {int(tie.sum())}, flips {len(flips)}")
    bad = [t for t in flips if not tie[t]]
    assert not bad, f"routing differs away from a near-tie at tokens {bad[:5]} (logit error {eps:.2e})"
    for t in flips:
        kth = np.sort(lo[t])[-k]
        assert all(lo[t][e] >= kth - 2 * eps for e in idx_g[t]), f"token {t}: invalid top-k {idx_g[t]}"
    return flips


SMALL = {
    "B2_S200_d256_f256_E8_2chunks": block_spec(B=2, S=200, d=256, heads=2, moe_f=256, moe_E=8, n_chunks=2,
                                               seed=21),
    "B4_S37_d128_f128_E4_4chunks": block_spec(B=4, S=37, d=128, heads=1, moe_f=128, moe_E=4, n_chunks=4, seed=22),
    "B4_S64_d256_f192_E8_drops_4chunks": block_spec(B=4, S=64, d=256, heads=2, moe_f=192, moe_E=8, moe_cf_num=1,
                                                    moe_cf_den=2, n_chunks=4, seed=23),
}


@pytest.mark.parametrize("case", list(SMALL))
def test_block_matches_oracle(L, case):
    spec = SMALL[case]
    inp = block_inputs(spec)
    T, d, E, k = spec.B * spec.S, spec.d, spec.moe.E, spec.moe.k
    fw = BO.block_forward(spec, inp)
    bw = BO.block_backward(spec, inp, fw)
    cfg, C, b = run_block(L, spec, _upload(L, inp), spec.n_chunks)
    mw = fw["moe"]

    qkv = np.concatenate([fw["q"], fw["k"], fw["v"]], axis=1)
    for name, ref in (("a", fw["a"]), ("qkv", qkv), ("attn", fw["o"]), ("h", fw["h"]), ("m", fw["m_in"])):
        assert_close(name, host(b[name]).reshape(ref.shape), ref, TOLB)
    idx = host(b["idx"]).reshape(T, k)
    flips = _check_routing(host(b["logits"]).reshape(T, E), mw["logits"], idx, mw["idx"], k)
    assert len(flips) == 0, f"near-tie routing flips at tokens {flips}: the float comparison below needs none"
    np.testing.assert_array_equal(host(b["slot"]).reshape(T, k), mw["slot"])
    np.testing.assert_array_equal(host(b["fill"]).reshape(-1, E)[-1], mw["fill"])
    assert_close("w", host(b["w"]).reshape(T, k), mw["w"], TOLB)
    assert_close("out", host(b["out"]).reshape(T, d), fw["out"], TOLB)

    mb = bw["moe"]
    for name, ref in (("dm", bw["dm"]), ("dh", bw["dh"]), ("dattn", bw["do"]), ("dqkv", bw["dqkv"]),
                      ("da", bw["da"]), ("dx", bw["dx"]), ("dlogits", mb["dlogits"])):
        assert_close(name, host(b[name]).reshape(ref.shape), ref, TOLB)
    for name, ref in (("dWqkv", bw["dWqkv"]), ("dWo", bw["dWo"]), ("dln1_g", bw["dln1_g"]),
                      ("dln1_b", bw["dln1_b"]), ("dln2_g", bw["dln2_g"]), ("dln2_b", bw["dln2_b"]),
                      ("dWg", mb["dWg"]), ("dW1", mb["dW1"]), ("dW2", mb["dW2"])):
        assert_close(name, host(b[name]).reshape(ref.shape), ref, TOLB)


_COMPARED = ("out", "dx", "logits", "idx", "w", "slot", "a", "qkv", "attn", "h", "m", "dm", "dh", "dattn", "dqkv",
             "da", "dlogits", "dWqkv", "dWo", "dln1_g", "dln1_b", "dln2_g", "dln2_b", "dWg", "dW1", "dW2")


def _assert_bitwise(b1, b2, E, label, names=_COMPARED):
    for n in names:
        assert torch.equal(b1[n].view(torch.int16) if b1[n].dtype == torch.bfloat16 else b1[n],
                           b2[n].view(torch.int16) if b2[n].dtype == torch.bfloat16 else b2[n]), f"{label}: {n}"
    assert torch.equal(b1["fill"].view(-1, E)[-1], b2["fill"].view(-1, E)[-1]), f"{label}: final fill"


# The block's expert products take every K sum whole and in order, so every
# output, routing and gradient is bitwise the same for any number of partitions.
def _assert_partition_equivalent(b1, b2, E, label):
    _assert_bitwise(b1, b2, E, label)


@pytest.mark.parametrize("case", ["B4_S37_d128_f128_E4_4chunks", "B4_S64_d256_f192_E8_drops_4chunks"])
def test_partitions_equal_unpartitioned(L, case):
    spec = SMALL[case]
    inp = block_inputs(spec)
    dev = _upload(L, inp)
    E = spec.moe.E
    _, C, b1 = run_block(L, spec, dev, 1)
    for n in (2, spec.B):
        _, _, bn = run_block(L, spec, dev, n)
        _assert_partition_equivalent(b1, bn, E, f"{n} partitions vs 1")
        fills = host(bn["fill"]).reshape(n, E)
        assert (np.diff(np.concatenate([np.zeros((1, E), np.int64), fills]), axis=0) >= 0).all()
        assert (fills[-1] <= C).all()
    if "drops" in case:
        assert (host(b1["slot"]) < 0).any(), "the drop case should drop tokens"


def test_deferred_weight_stream_and_repeat_are_bitwise_stable(L):
    spec = SMALL["B2_S200_d256_f256_E8_2chunks"]
    dev = _upload(L, block_inputs(spec))
    _, _, b1 = run_block(L, spec, dev, 2)
    _, _, b2 = run_block(L, spec, dev, 2, same_stream=True)
    _assert_bitwise(b1, b2, spec.moe.E, "three streams vs one")
    _, _, b3 = run_block(L, spec, dev, 2)
    _assert_bitwise(b1, b3, spec.moe.E, "repeat")


def test_forward_then_backward_passes_equal_combined(L):
    spec = SMALL["B4_S37_d128_f128_E4_4chunks"]
    dev = _upload(L, block_inputs(spec))
    _, _, b1 = run_block(L, spec, dev, 4, passes=3)
    cfg, C = _cfg(L, spec)
    w, x, dy = dev
    b2 = L.alloc_block(cfg, 4)
    out, dx = torch.empty_like(x), torch.empty_like(x)
    s = torch.cuda.current_stream()
    L.moe_block_chunked(cfg, w, b2, x, out, dy, dx, b2, L.MOE_BLOCK_FWD, 4, [s] * 3, b2["ws"])
    L.moe_block_chunked(cfg, w, b2, x, out, dy, dx, b2, L.MOE_BLOCK_BWD, 4, [s] * 3, b2["ws"])
    torch.cuda.synchronize()
    b2["out"], b2["dx"] = out, dx
    _assert_bitwise(b1, b2, spec.moe.E, "separate passes")


# ------------------------------------------------------------------ full size
@pytest.fixture(scope="module")
def full(L):
    spec = BLOCK5
    log(f"[block full] generating inputs for {spec.name}")
    inp = block_inputs(spec)
    dev = _upload(L, inp)
    _, C, b4 = run_block(L, spec, dev, spec.n_chunks)
    return spec, inp, dev, C, b4


def test_full_size_partitioned_equals_unpartitioned(L, full):
    spec, inp, dev, C, b4 = full
    _, _, b1 = run_block(L, spec, dev, 1)
    _assert_partition_equivalent(b4, b1, spec.moe.E, "4 partitions vs 1 at full size")


def test_full_size_sampled_forward_matches_oracle(L, full):
    spec, inp, dev, C, b = full
    T, d, E, k, S = spec.B * spec.S, spec.d, spec.moe.E, spec.moe.k, spec.S
    fill = host(b["fill"]).reshape(-1, E)[-1]
    assert fill.sum() == T * k and (fill <= C).all(), "the full-size block is expected to drop no token"
    out = host(b["out"]).reshape(T, d)
    h = host(b["h"]).reshape(T, d)
    m = host(b["m"]).reshape(T, d)
    lg = host(b["logits"]).reshape(T, E)
    idx = host(b["idx"]).reshape(T, k)
    rng = np.random.default_rng(5)
    for seq in (1, 6):  # partitions 0 and 3
        pos = np.unique(np.concatenate([[0, 1, 63, 64, 127, 128, S - 1], rng.integers(0, S, 5)]))
        log(f"[block full] oracle prefix of sequence {seq}, positions {pos.tolist()}")
        ref = BO.block_forward_tokens(spec, inp, seq, pos)
        rows = seq * S + pos
        assert_close("h", h[rows], ref["h"], TOLB)
        assert_close("m", m[rows], ref["m_in"], TOLB)
        flips = _check_routing(lg[rows], ref["logits"], idx[rows], ref["idx"], k)
        keep = np.setdiff1d(np.arange(len(pos)), flips)
        log(f"[block full] near-tie flips among sampled tokens: {len(flips)}")
        assert_close("out", out[rows][keep], ref["out"][keep], TOLB)


def test_full_size_backward_identities(L, full):
    """Identities of the backward that hold at any size, on the GPU's own tensors."""
    spec, inp, dev, C, b = full
    T, d, E, S, H = spec.B * spec.S, spec.d, spec.moe.E, spec.S, spec.heads
    f64 = lambda n, *shape: host(b[n]).astype(np.float64).reshape(*shape)
    dm, da, dh, dx = f64("dm", T, d), f64("da", T, d), f64("dh", T, d), f64("dx", T, d)
    # LayerNorm bias gradients are column sums of the incoming gradient
    assert normwise(host(b["dln2_b"]), dm.sum(0)) < 1e-3
    assert normwise(host(b["dln1_b"]), da.sum(0)) < 1e-3
    # the gain gradient pairs it with the normalised input
    hh = f64("h", T, d)
    xhat2 = (hh - host(b["ln2_mean"])[:, None]) * host(b["ln2_rstd"])[:, None]
    assert normwise(host(b["dln2_g"]), (dm * xhat2).sum(0)) < 1e-3
    # LN backward output has zero row mean: rows of dx - dh sum to 0
    r = (dx - dh).sum(1)
    assert np.abs(r).max() <= 2e-2 * np.abs(dx - dh).sum(1).max()
    # weight gradients are products of saved tensors (sampled rows)
    rng = np.random.default_rng(6)
    j = rng.choice(d, 8, replace=False)
    assert_close("dWo rows", host(b["dWo"]).reshape(d, d)[j], dh[:, j].T @ f64("attn", T, d), TOLB)
    j3 = rng.choice(3 * d, 8, replace=False)
    assert_close("dWqkv rows", host(b["dWqkv"]).reshape(3 * d, d)[j3],
                 f64("dqkv", T, 3 * d)[:, j3].T @ f64("a", T, d), TOLB)
    assert_close("dWg", host(b["dWg"]).reshape(E, d), f64("dlogits", T, E).T @ f64("m", T, d), TOLB)
    # attention: per sequence and head, dS rows sum to 0, so dK sums to 0 over keys;
    # P rows sum to 1, so dV summed over keys equals dO summed over queries
    dqkv = f64("dqkv", spec.B, S, 3, H, 128)
    dattn = f64("dattn", spec.B, S, H, 128)
    dk_sum = dqkv[:, :, 1].sum(1)
    assert np.abs(dk_sum).max() <= 2e-2 * np.abs(dqkv[:, :, 1]).sum(1).max()
    assert normwise(dqkv[:, :, 2].sum(1), dattn.sum(1)) < 2e-2


@pytest.mark.timeout(600)
def test_full_size_moe_layer_matches_layer_oracle(L, full):
    """The block's MoE layer at full size against the layer oracle fed the
    GPU's own MoE input m and the block's upstream gradient: routing, slots
    and fills bit-exact over all 16384 tokens; y = out - h, dm, dlogits, dW1,
    dW2 and dWg as whole tensors.  This separates the MoE path from the
    LayerNorm and attention rounding upstream of it."""
    spec, inp, dev, C, b = full
    T, d, E, k = spec.B * spec.S, spec.d, spec.moe.E, spec.moe.k
    m = host(b["m"]).reshape(T, d)
    moe_inp = {"x": m, "Wg": inp["Wg"], "W1": inp["W1"], "W2": inp["W2"], "bias": None, "dy": inp["dy"]}
    log("[block full] layer oracle on the GPU's MoE input")
    fw = O.layer_forward(spec.moe, moe_inp, C=C)
    bw = O.layer_backward(spec.moe, moe_inp, fw)
    log("[block full] layer oracle done")
    np.testing.assert_array_max_ulp(host(b["logits"]).reshape(T, E), fw["logits"], maxulp=1)
    np.testing.assert_array_equal(host(b["idx"]).reshape(T, k), fw["idx"])
    np.testing.assert_array_equal(host(b["slot"]).reshape(T, k), fw["slot"])
    np.testing.assert_array_equal(host(b["fill"]).reshape(-1, E)[-1], fw["fill"])
    h = host(b["h"]).reshape(T, d).astype(np.float64)
    assert_close("out (= h + MoE(m))", host(b["out"]).reshape(T, d), h + fw["y"], TOLB)
    assert_close("dm", host(b["dm"]).reshape(T, d), bw["dx"], TOLB)
    assert_close("dlogits", host(b["dlogits"]).reshape(T, E), bw["dlogits"], TOLB)
    assert_close("dWg", host(b["dWg"]).reshape(E, d), bw["dWg"], TOLB)
    assert_close("dW1", host(b["dW1"]).reshape(bw["dW1"].shape), bw["dW1"], TOLB)
    assert_close("dW2", host(b["dW2"]).reshape(bw["dW2"].shape), bw["dW2"], TOLB)


@pytest.mark.timeout(600)
def test_full_size_whole_sequences_match_block_oracle(L, full):
    """Two whole sequences of the full-size block through the block oracle
    (the full batch drops no token, and a sequence alone with the batch's
    capacity drops none either, so each token's forward and backward depend
    only on its own sequence): every activation and activation gradient of
    their tokens.  Where a token's routing differs (the GPU's and the oracle's
    bf16 MoE inputs can differ by an ulp in rare elements), the GPU's choice
    must be a valid top-k of the oracle's logits within twice the logit error;
    the oracle then follows the GPU's choice for the comparison."""
    spec, inp, dev, C, b = full
    T, d, E, k, S = spec.B * spec.S, spec.d, spec.moe.E, spec.moe.k, spec.S
    fill = host(b["fill"]).reshape(-1, E)[-1]
    assert fill.sum() == T * k, "the full-size block is expected to drop no token"
    from dataclasses import replace
    sub = replace(spec, B=1, moe=replace(spec.moe, T=S))
    gpu = {n: host(b[n]).reshape(T, -1) for n in ("a", "qkv", "attn", "h", "m", "out", "logits", "idx", "dm", "dh",
                                                  "dattn", "dqkv", "da", "dx")}
    for seq in (1, 6):   # partitions 0 and 3
        rows = slice(seq * S, (seq + 1) * S)
        si = dict(inp)
        si["x"], si["dy"] = inp["x"][rows], inp["dy"][rows]
        log(f"[block full] block oracle on sequence {seq}")
        fw = BO.block_forward(sub, si, C=C)
        flips = _check_routing(gpu["logits"][rows], fw["moe"]["logits"], gpu["idx"][rows], fw["moe"]["idx"], k)
        if len(flips):
            log(f"[block full] sequence {seq}: {len(flips)} near-tie routing flips; the oracle follows the GPU there")
            fw = BO.block_forward(sub, si, C=C, idx_override=gpu["idx"][rows])
        assert (fw["moe"]["slot"] >= 0).all()
        bw = BO.block_backward(sub, si, fw)
        qkv = np.concatenate([fw["q"], fw["k"], fw["v"]], axis=1)
        for name, ref in (("a", fw["a"]), ("qkv", qkv), ("attn", fw["o"]), ("h", fw["h"]), ("m", fw["m_in"]),
                          ("out", fw["out"]), ("dm", bw["dm"]), ("dh", bw["dh"]), ("dattn", bw["do"]),
                          ("dqkv", bw["dqkv"]), ("da", bw["da"]), ("dx", bw["dx"])):
            assert_close(f"sequence {seq}: {name}", gpu[name][rows], ref, TOLB)


def test_dw_schedule_from_measured_times_orders_the_weight_stream(L):
    """The weight-gradient schedule pass applied to the block backward (Sec. 4,
    Alg. 1): the operations' times measured in this run (one stream,
    MOE_BLOCK_TIMED), the all-to-alls costed by an xGMI model, the planner's
    order given to the weight stream.  Every gradient is bitwise the same as
    with the default order and with the reverse order."""
    spec = SMALL["B4_S64_d256_f192_E8_drops_4chunks"]
    inp = block_inputs(spec)
    w, x, dy = _upload(L, inp)
    m = spec.moe
    C = O.capacity(spec.B * spec.S, m.E, m.k, m.cf_num, m.cf_den)

    def backward(order, passes=L.MOE_BLOCK_BWD, one_stream=False):
        cfg = L.make_block_cfg(spec.B, spec.S, spec.heads, m.f, m.E, m.k, C, m.G, m.act, m.renorm, dw_order=order)
        b = L.alloc_block(cfg, 4)
        out, dx = torch.empty_like(x), torch.empty_like(x)
        streams = [torch.cuda.current_stream()] * 3 if one_stream else [torch.cuda.Stream() for _ in range(3)]
        streams[0].wait_stream(torch.cuda.current_stream())
        L.moe_block_chunked(cfg, w, b, x, out, dy, dx, b, L.MOE_BLOCK_FWD, 4, streams, b["ws"])
        L.moe_block_chunked(cfg, w, b, x, out, dy, dx, b, passes, 4, streams, b["ws"])
        torch.cuda.synchronize()
        b["out"], b["dx"] = out, dx
        return b

    timed = backward(None, L.MOE_BLOCK_BWD | L.MOE_BLOCK_TIMED, one_stream=True)
    op_ms = L.moe_block_op_times()
    log("  op times (ms): " + ", ".join(f"{n} {t:.3f}" for n, t in zip(L.BLOCK_OPS, op_ms)))
    assert np.all(op_ms > 0) and np.all(np.isfinite(op_ms))
    kept = int(host(timed["fill"]).reshape(4, m.E)[-1].sum())
    a2a_ms = kept * spec.d * 2 / 8 / 153e9 * 1e3     # the slice to one of 7 peers over one xGMI link
    order, assign, ov = L.moe_block_dw_schedule(op_ms, a2a_ms)
    log(f"  all-to-all {a2a_ms:.4f} ms each; planner order {order.tolist()}, overlap {ov:.4f} ms")
    assert assign[6] == 1, "dWg should overlap the first all-to-all"
    base = backward(None)
    planned = backward(order.tolist())
    reverse = backward(list(range(13, 7, -1)))
    grads = ("dx", "dWqkv", "dWo", "dln1_g", "dln1_b", "dln2_g", "dln2_b", "dWg", "dW1", "dW2", "dm", "dh", "dqkv")
    _assert_bitwise(base, timed, m.E, "timed single stream vs default", grads)
    _assert_bitwise(base, planned, m.E, "planner order vs default", grads)
    _assert_bitwise(base, reverse, m.E, "reverse order vs default", grads)


def test_prepacked_expert_weights_give_the_same_block(L):
    """moe.wpacked = 1: the block takes W1, W2 already packed (moe_pack_weights)
    and writes dW1, dW2 packed; every output and gradient is bitwise the one
    of the block that packs the row-major weights itself."""
    spec = SMALL["B2_S200_d256_f256_E8_2chunks"]
    inp = block_inputs(spec)
    w, x, dy = _upload(L, inp)
    m = spec.moe
    C = O.capacity(spec.B * spec.S, m.E, m.k, m.cf_num, m.cf_den)
    cfg0 = L.make_block_cfg(spec.B, spec.S, spec.heads, m.f, m.E, m.k, C, m.G, m.act, m.renorm)
    cfg1 = L.make_block_cfg(spec.B, spec.S, spec.heads, m.f, m.E, m.k, C, m.G, m.act, m.renorm, wpacked=1)
    wp = dict(w)
    wp["W1"], wp["W2"] = torch.empty_like(w["W1"]), torch.empty_like(w["W2"])
    L.moe_pack_weights(cfg1.moe, w["W1"], w["W2"], wp["W1"], wp["W2"])
    res = []
    for cfg, weights in ((cfg0, w), (cfg1, wp)):
        b = L.alloc_block(cfg, 2)
        out, dx = torch.empty_like(x), torch.empty_like(x)
        s = torch.cuda.current_stream()
        L.moe_block_chunked(cfg, weights, b, x, out, dy, dx, b, L.MOE_BLOCK_FWD | L.MOE_BLOCK_BWD, 2, [s] * 3,
                            b["ws"])
        torch.cuda.synchronize()
        b["out"], b["dx"] = out, dx
        res.append(b)
    b0, b1 = res
    _assert_bitwise(b0, b1, m.E, "prepacked vs row-major weights", tuple(n for n in _COMPARED if n not in ("dW1", "dW2")))
    E, f, d = m.E, m.f, spec.d
    unpack = lambda t, R, X: host(t).reshape(E, R // 16, X // 32, 16, 32).transpose(0, 1, 3, 2, 4).reshape(E, R, X)
    np.testing.assert_array_equal(unpack(b1["dW1"], f, d), host(b0["dW1"]).reshape(E, f, d))
    np.testing.assert_array_equal(unpack(b1["dW2"], d, f), host(b0["dW2"]).reshape(E, d, f))
