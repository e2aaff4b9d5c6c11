"""moe_dispatch_noalloc (the dispatch with the library's fixed workspace, for
callers that cannot allocate) against moe_dispatch through the C ABI: two
calls in a row, the second with a smaller input and a carry-in, each equal
bit for bit to moe_dispatch on the same input (slots, fills and every kept
row of the send buffer)."""
import numpy as np
import pytest

from oracle import moe_oracle as O
from synth import LayerSpec, layer_inputs
from tests.gpu_harness import ebuf, host, kept_rows, log, nan_fill, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def L():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    from paper_2404_19429_amd import lancet_moe
    return lancet_moe


def _one_call(L, spec, C, carry):
    inp = layer_inputs(spec)
    log(f"[noalloc] T={spec.T} d={spec.d} E={spec.E} k={spec.k} C={C} carry={'yes' if carry is not None else 'no'}")
    cfg = L.make_cfg(spec.T, spec.d, spec.f, spec.E, spec.k, C, spec.G, spec.dtype, spec.act, spec.renorm)
    ref, got = L.alloc_layer(cfg), L.alloc_layer(cfg)
    nan_fill(ref)
    nan_fill(got)
    x, Wg = to_dev(inp["x"], torch.bfloat16), to_dev(inp["Wg"], torch.bfloat16)
    L.moe_gate_topk(cfg, x, Wg, None, ref.logits, ref.idx, ref.w)
    cin = None if carry is None else torch.as_tensor(np.asarray(carry, np.int32)).cuda()
    L.moe_dispatch(cfg, x, ref.idx, cin, ref.fill, ref.slot, ref.send_buf, ref.ws_dispatch)
    L.moe_dispatch_noalloc(cfg, x, ref.idx, cin, got.fill, got.slot, got.send_buf)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(got.slot), host(ref.slot))
    np.testing.assert_array_equal(host(got.fill), host(ref.fill))
    fill = host(ref.fill)
    lo = np.zeros(spec.E, np.int64) if carry is None else np.asarray(carry, np.int64)
    np.testing.assert_array_equal(kept_rows(ebuf(got, "send_buf"), fill, lo), kept_rows(ebuf(ref, "send_buf"), fill, lo))
    # the capacity rule itself, against the oracle on the same choices
    slot_o, fill_o = O.assign_slots(host(ref.idx), spec.E, C, lo)
    np.testing.assert_array_equal(host(got.slot), slot_o)
    np.testing.assert_array_equal(fill, fill_o)
    return int(fill.sum() - lo.sum())


def test_noalloc_dispatch_equals_dispatch_twice_second_smaller(L):
    big = LayerSpec(name="na1", T=20000, d=256, f=256, E=16, k=2, cf_num=5, cf_den=4, dtype="bf16",
                    act="gelu_tanh", renorm=1, seed=61)
    small = LayerSpec(name="na2", T=777, d=512, f=128, E=8, k=2, cf_num=1, cf_den=1, dtype="bf16",
                      act="gelu_tanh", renorm=1, zipf_s=1.2, seed=62)
    C1 = O.capacity(big.T, big.E, big.k, big.cf_num, big.cf_den)
    assert _one_call(L, big, C1, None) > 0
    C2 = O.capacity(small.T, small.E, small.k, small.cf_num, small.cf_den)
    carry = [0, 5, C2, 17, 1, 0, 30, 2]
    assert _one_call(L, small, C2, carry) > 0


def test_noalloc_dispatch_rejects_a_call_above_its_workspace(L):
    cfg = L.make_cfg(1 << 17, 128, 128, 64, 2, 4096, 1, "bf16", "gelu_tanh", 1)
    with pytest.raises(L.MoeError) as ei:
        L._check(L._lib.moe_dispatch_noalloc(L.ctypes.byref(cfg), 16, 16, None, 16, 16, 16, None))
    assert ei.value.status == L.MOE_ESHAPE
