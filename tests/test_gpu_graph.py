"""The layer step (forward + backward, six C-ABI calls) captured once in a
HIP graph and replayed: every replay, with eager work on the same stream
between replays, reproduces the eager step's outputs bit for bit (the
library records no memset nodes; all kernels are deterministic)."""
import numpy as np
import pytest

from synth import LayerSpec, layer_inputs
from tests.gpu_harness import host, log, spec_C, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

OUTS = ("logits", "idx", "w", "slot", "fill", "send_buf", "H", "A", "O", "y", "dO", "dH", "dXe", "dlogits", "dx",
        "dW1", "dW2", "dWg")


@pytest.fixture(scope="module")
def L():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    from paper_2404_19429_amd import lancet_moe
    return lancet_moe


@pytest.mark.parametrize("routing", ["token", "bpr"])
def test_graph_replays_equal_eager(L, routing):
    spec = LayerSpec(name="g", T=1500, d=256, f=512, E=16, k=2, cf_num=1, cf_den=1, dtype="bf16", act="gelu_tanh",
                     renorm=1, zipf_s=0.8, seed=31)
    inp = layer_inputs(spec)
    C = spec_C(spec)
    log(f"[graph] T={spec.T} E={spec.E} C={C} routing={routing}")
    cfg = L.make_cfg(spec.T, spec.d, spec.f, spec.E, spec.k, C, 1, "bf16", "gelu_tanh", 1, wpacked=1)
    b = L.alloc_layer(cfg)
    other = L.alloc_layer(cfg)
    dev = {n: to_dev(inp[n], torch.bfloat16) for n in ("x", "Wg", "W1", "W2", "dy")}
    bias = torch.as_tensor(inp["bias"], dtype=torch.float32).cuda()

    def step(bb):
        L.moe_gate_topk(cfg, dev["x"], dev["Wg"], bias, bb.logits, bb.idx, bb.w)
        if routing == "bpr":
            L.moe_dispatch_bpr(cfg, dev["x"], bb.logits, bb.idx, bb.fill, bb.slot, bb.send_buf, bb.order, bb.ws_bpr)
        else:
            L.moe_dispatch(cfg, dev["x"], bb.idx, bb.carry, bb.fill, bb.slot, bb.send_buf, bb.ws_dispatch)
        L.moe_expert_ffn_fwd(cfg, bb.send_buf, bb.carry, bb.fill, bb.W1p, bb.W2p, bb.H, bb.A, bb.O, bb.ws_ffn)
        L.moe_combine(cfg, bb.O, bb.idx, bb.slot, bb.w, bb.y)
        L.moe_bwd_dx(cfg, dev["Wg"], bb.logits, bb.idx, bb.w, bb.slot, bb.carry, bb.fill, bb.H, bb.O, bb.W1p, bb.W2p,
                     dev["dy"], bb.dO, bb.dH, bb.dXe, bb.dlogits, bb.dx, bb.ws_dx)
        L.moe_bwd_dw(cfg, dev["x"], bb.dlogits, bb.carry, bb.fill, bb.send_buf, bb.A, bb.dO, bb.dH, bb.dW1, bb.dW2,
                     bb.dWg, bb.ws_dw)

    for bb in (b, other):
        L.moe_pack_weights(cfg, dev["W1"], dev["W2"], bb.W1p, bb.W2p)
    step(other)                                   # eager reference
    torch.cuda.synchronize()
    ref = {n: host(getattr(other, n)) for n in OUTS}
    fill = ref["fill"]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(b)
    torch.cuda.synchronize()
    for rep in range(3):
        for n in OUTS:                            # poison the graph's outputs
            t = getattr(b, n)
            t.fill_(float("nan") if t.is_floating_point() else -3)
        graph.replay()
        step(other)                               # eager work between replays
        torch.cuda.synchronize()
        for n in OUTS:
            got, want = host(getattr(b, n)), ref[n]
            if n in ("send_buf", "H", "A", "O", "dO", "dH", "dXe"):
                X = spec.d if n in ("send_buf", "O", "dO", "dXe") else spec.f
                rows = L.rows_alloc(cfg)
                got = got.reshape(spec.E, rows * X // 512, 512) if n not in ("O", "dXe") else got.reshape(spec.E, rows, X)
                want = want.reshape(got.shape)
                # kept rows only (the others are never written)
                for e in range(spec.E):
                    nrow = int(fill[e])
                    if n in ("O", "dXe"):
                        np.testing.assert_array_equal(got[e, :nrow], want[e, :nrow], err_msg=f"{n} replay {rep}")
                    else:   # blocked layout: compare whole 16-row blocks of kept rows
                        nb = (nrow // 16) * (X // 32)
                        np.testing.assert_array_equal(got[e, :nb], want[e, :nb], err_msg=f"{n} replay {rep}")
            else:
                np.testing.assert_array_equal(got, want, err_msg=f"{n} replay {rep}")


def test_graph_replay_full_size_equals_eager(L):
    """The configuration bench.py times: the 8192-token layer (d_model 1024,
    d_ff 4096, 16 experts, top-2), packed weights, the step as one HIP graph.
    Two replays reproduce the eager step's outputs bit for bit."""
    from synth import layer_spec
    spec = layer_spec(2)
    inp = layer_inputs(spec)
    C = spec_C(spec)
    log(f"[graph full] {spec.name} C={C}")
    cfg = L.make_cfg(spec.T, spec.d, spec.f, spec.E, spec.k, C, spec.G, spec.dtype, spec.act, spec.renorm,
                     wpacked=1)
    b, ref_b = L.alloc_layer(cfg), L.alloc_layer(cfg)
    dev = {n: to_dev(inp[n], torch.bfloat16) for n in ("x", "Wg", "W1", "W2", "dy")}

    def step(bb):
        L.moe_gate_topk(cfg, dev["x"], dev["Wg"], None, bb.logits, bb.idx, bb.w)
        L.moe_dispatch(cfg, dev["x"], bb.idx, bb.carry, bb.fill, bb.slot, bb.send_buf, bb.ws_dispatch)
        L.moe_expert_ffn_fwd(cfg, bb.send_buf, bb.carry, bb.fill, bb.W1p, bb.W2p, bb.H, bb.A, bb.O, bb.ws_ffn)
        L.moe_combine(cfg, bb.O, bb.idx, bb.slot, bb.w, bb.y)
        L.moe_bwd_dx(cfg, dev["Wg"], bb.logits, bb.idx, bb.w, bb.slot, bb.carry, bb.fill, bb.H, bb.O, bb.W1p, bb.W2p,
                     dev["dy"], bb.dO, bb.dH, bb.dXe, bb.dlogits, bb.dx, bb.ws_dx)
        L.moe_bwd_dw(cfg, dev["x"], bb.dlogits, bb.carry, bb.fill, bb.send_buf, bb.A, bb.dO, bb.dH, bb.dW1, bb.dW2,
                     bb.dWg, bb.ws_dw)

    for bb in (b, ref_b):
        L.moe_pack_weights(cfg, dev["W1"], dev["W2"], bb.W1p, bb.W2p)
    step(ref_b)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(b)
    names = ("logits", "idx", "w", "slot", "fill", "y", "dlogits", "dx", "dW1", "dW2", "dWg")
    for rep in range(2):
        for n in names:
            t = getattr(b, n)
            t.fill_(float("nan") if t.is_floating_point() else -3)
        graph.replay()
        torch.cuda.synchronize()
        for n in names:
            assert torch.equal(getattr(b, n), getattr(ref_b, n)), f"{n} differs on replay {rep}"
