"""C-ABI tests that need no GPU: the library loads, exports every symbol the
header declares, and rejects invalid arguments on the host before launching."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lancet_moe.h")

L = pytest.importorskip("paper_2404_19429_amd.lancet_moe", reason="library not built")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(moe_[a-z_0-9]+)\s*\(", src)))


def test_header_declares_and_library_exports_every_symbol():
    names = _declared()
    assert set(names) == set(L.EXPORTS), names
    lib = ctypes.CDLL(L.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


@pytest.mark.parametrize("T,E,k,num,den,expect", [(8192, 16, 2, 5, 4, 1280), (16384, 8, 2, 5, 4, 5120),
                                                  (32768, 64, 2, 2, 1, 2048), (256, 4, 1, 5, 4, 80),
                                                  (0, 4, 1, 5, 4, 0), (10, 3, 1, 1, 1, 4)])
def test_capacity(T, E, k, num, den, expect):
    assert L.moe_capacity(T, E, k, num, den) == expect


@pytest.mark.parametrize("args", [(-1, 4, 1, 1, 1), (10, 0, 1, 1, 1), (10, 4, 0, 1, 1), (10, 4, 1, 0, 1),
                                  (10, 4, 1, 1, 0), (1 << 40, 1, 8, 8, 1)])
def test_capacity_invalid(args):
    assert L.moe_capacity(*args) == -1


def _cfg(**kw):
    base = dict(T=1024, d_model=256, d_ff=512, E=8, k=2, C=320, G=1, dtype="bf16", act="gelu_tanh", renorm=1)
    base.update(kw)
    return L.make_cfg(**base)


GOOD = 4096  # a fake, 16-byte aligned address: validation never dereferences it


def _gate(cfg, x=GOOD, Wg=GOOD, bias=None, logits=GOOD, idx=GOOD, w=GOOD):
    return L._lib.moe_gate_topk(ctypes.byref(cfg) if cfg is not None else None, x, Wg, bias, logits, idx, w, None)


@pytest.mark.parametrize("kw,status", [
    (dict(k=0), L.MOE_EINVAL), (dict(k=9, E=16), L.MOE_EINVAL), (dict(k=5, E=4), L.MOE_EINVAL),
    (dict(E=0), L.MOE_ESHAPE), (dict(E=65), L.MOE_ESHAPE), (dict(C=0), L.MOE_EINVAL),
    (dict(G=3), L.MOE_EINVAL), (dict(G=0), L.MOE_EINVAL), (dict(d_model=100), L.MOE_ESHAPE),
    (dict(d_ff=4), L.MOE_ESHAPE), (dict(T=-1), L.MOE_EINVAL), (dict(act=7), L.MOE_EINVAL),
    (dict(renorm=2), L.MOE_EINVAL), (dict(dtype=5), L.MOE_EDTYPE),
])
def test_invalid_cfg_rejected_before_launch(kw, status):
    assert _gate(_cfg(**kw)) == status
    assert L.moe_last_error()


def test_null_and_misaligned_pointers():
    c = _cfg()
    assert L._lib.moe_gate_topk(None, GOOD, GOOD, None, GOOD, GOOD, GOOD, None) == L.MOE_EINVAL
    assert _gate(c, x=None) == L.MOE_EINVAL and "x is NULL" in L.moe_last_error()
    assert _gate(c, idx=None) == L.MOE_EINVAL
    assert _gate(c, w=GOOD + 4) == L.MOE_EALIGN
    assert _gate(c, bias=GOOD + 8) == L.MOE_EALIGN


def test_valid_call_without_gpu_reports_device_error():
    assert _gate(_cfg()) == L.MOE_EDEVICE
    assert "device" in L.moe_last_error()


def test_dispatch_workspace_and_alias_checks():
    c = _cfg()
    need = L.moe_workspace_bytes(c, L.MOE_CALL_DISPATCH)
    assert need > 0
    lib = L._lib
    assert lib.moe_dispatch(ctypes.byref(c), GOOD, GOOD, None, GOOD, GOOD, GOOD, None, 0, None) == L.MOE_EWORKSPACE
    assert lib.moe_dispatch(ctypes.byref(c), GOOD, GOOD, None, GOOD, GOOD, GOOD, GOOD, need - 1, None) == L.MOE_EWORKSPACE
    assert lib.moe_dispatch(ctypes.byref(c), GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, need, None) == L.MOE_EINVAL
    assert "alias" in L.moe_last_error()
    assert lib.moe_dispatch(ctypes.byref(c), GOOD, GOOD, GOOD, GOOD * 2, GOOD, GOOD, GOOD, need, None) == L.MOE_EDEVICE


def test_bf16_gemm_shape_rule():
    c = _cfg(d_model=72)         # multiple of 8 (gate/dispatch fine) but not of 64
    lib = L._lib
    assert lib.moe_expert_ffn_fwd(ctypes.byref(c), *([GOOD] * 8), GOOD, 1 << 40, None) == L.MOE_ESHAPE
    assert _gate(c) == L.MOE_EDEVICE
    c32 = _cfg(d_model=72, dtype="f32")
    assert lib.moe_expert_ffn_fwd(ctypes.byref(c32), *([GOOD] * 8), GOOD, 1 << 40, None) == L.MOE_EDEVICE


def test_workspace_bytes_invalid_cfg_is_zero():
    assert L.moe_workspace_bytes(_cfg(k=0), 0) == 0
    assert L.moe_workspace_bytes(_cfg(), 9) == 0


def test_binding_rejects_host_tensors_and_short_buffers():
    import torch
    c = _cfg(T=4, d_model=8, d_ff=8, E=2, k=1, C=4)
    with pytest.raises(ValueError, match="device tensor"):
        L.moe_gate_topk(c, torch.zeros(4, 8, dtype=torch.bfloat16), None, None, None, None, None, stream=0)


def test_isa_check_flags_use_before_wait():
    from paper_2404_19429_amd.isa_check import check_text
    clean = """_ZN4lmoe16gemm_wide_kernelX:
\t;;#ASMSTART
\tds_read_b128 v[4:7], v1
\ts_waitcnt lgkmcnt(0)
\t;;#ASMEND
\tv_mfma_f32_16x16x32_bf16 a[0:3], v[4:7], v[8:11], a[0:3]
"""
    bad = clean.replace("\ts_waitcnt lgkmcnt(0)\n", "").replace(";;#ASMEND\n", ";;#ASMEND\n\tv_mov_b32 v20, v5\n")
    assert check_text(clean) == {}
    hits = check_text(bad)
    assert list(hits) == ["_ZN4lmoe16gemm_wide_kernelX"] and any("v_mov_b32" in h for h in hits["_ZN4lmoe16gemm_wide_kernelX"])


def _block_call(cfg, n_chunks=2, passes=3, grads=True, ws_bytes=None, **acts_over):
    w = L.moe_block_weights(*([GOOD] * len(L.BLOCK_WEIGHTS)))
    g = L.moe_block_grads(*([GOOD] * len(L.BLOCK_GRADS))) if grads else None
    names = L.BLOCK_ACTS_FWD + L.BLOCK_ACTS_BWD
    a = L.moe_block_acts(*[acts_over.get(n, GOOD) for n in names])
    st = (ctypes.c_void_p * 3)(None, None, None)
    need = L.moe_block_workspace_bytes(cfg, n_chunks)
    ws = need if ws_bytes is None else ws_bytes
    return L._lib.moe_block_chunked(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(g) if g else None, GOOD,
                                    GOOD, GOOD, GOOD, ctypes.byref(a), passes, n_chunks, st, GOOD, ws)


def _bcfg(**kw):
    base = dict(B=8, S=2048, heads=16, d_ff=8192, E=16, k=2, C=2560)
    base.update(kw)
    return L.make_block_cfg(**base)


def test_block_workspace_bytes():
    assert L.moe_block_workspace_bytes(_bcfg(), 4) > 0
    assert L.moe_block_workspace_bytes(_bcfg(), 3) == 0 and "n_chunks" in L.moe_last_error()


def test_block_valid_call_without_gpu_reports_device_error():
    assert _block_call(_bcfg(), 4) == L.MOE_EDEVICE


@pytest.mark.parametrize("mutate,status", [
    (lambda c: setattr(c, "heads", 15), L.MOE_ESHAPE),              # d_model != 128 * heads
    (lambda c: setattr(c.moe, "T", 100), L.MOE_EINVAL),             # T != B * S
    (lambda c: setattr(c.moe, "dtype", L.MOE_F32), L.MOE_EDTYPE),   # bf16 only
    (lambda c: setattr(c.moe, "d_ff", 8200), L.MOE_ESHAPE),         # d_ff not a multiple of 64
    (lambda c: setattr(c, "B", 0), L.MOE_ESHAPE),
])
def test_block_invalid_cfg(mutate, status):
    c = _bcfg()
    mutate(c)
    assert _block_call(c, 4) == status
    assert L.moe_last_error()


def test_block_invalid_arguments():
    c = _bcfg()
    assert _block_call(c, 3) == L.MOE_EINVAL                         # 3 does not divide B = 8
    assert _block_call(c, 4, passes=0) == L.MOE_EINVAL
    assert _block_call(c, 4, grads=False) == L.MOE_EINVAL             # backward without gradients
    assert _block_call(c, 4, passes=L.MOE_BLOCK_FWD, grads=False) == L.MOE_EDEVICE
    assert _block_call(c, 4, ws_bytes=16) == L.MOE_EWORKSPACE
    assert _block_call(c, 4, qkv=None) == L.MOE_EINVAL and "qkv" in L.moe_last_error()
    assert _block_call(c, 4, lse=GOOD + 4) == L.MOE_EALIGN
    assert _block_call(c, 4, passes=L.MOE_BLOCK_FWD, dqkv=None) == L.MOE_EDEVICE   # backward buffers unused


def test_pack_weights_validation():
    c = _cfg()
    lib = L._lib
    assert lib.moe_pack_weights(ctypes.byref(c), GOOD, GOOD * 2, GOOD * 3, GOOD * 4, None) == L.MOE_EDEVICE
    assert lib.moe_pack_weights(ctypes.byref(c), GOOD, GOOD * 2, GOOD, GOOD * 4, None) == L.MOE_EINVAL
    assert lib.moe_pack_weights(ctypes.byref(c), GOOD, GOOD * 2, None, GOOD * 4, None) == L.MOE_EINVAL
    assert lib.moe_pack_weights(ctypes.byref(_cfg(d_model=72)), GOOD, GOOD * 2, GOOD * 3, GOOD * 4, None) == L.MOE_ESHAPE


def test_expert_buffer_sizes_pad_bf16_rows_to_16():
    assert L.rows_alloc(_cfg(C=320)) == 320 and L.rows_alloc(_cfg(C=321)) == 336
    assert L.rows_alloc(_cfg(C=321, dtype="f32")) == 321
    assert L.expert_numel(_cfg(C=100, E=3), 64) == 3 * 112 * 64


def test_ffn_fwd_workspace_rule():
    """bf16 expert products need the K-split workspace the library reports; float needs none."""
    c = _cfg()
    lib = L._lib
    need = L.moe_workspace_bytes(c, L.MOE_CALL_FFN_FWD)
    assert need > 0 and need == L.moe_workspace_bytes(c, L.MOE_CALL_BWD_DX)
    assert lib.moe_expert_ffn_fwd(ctypes.byref(c), *([GOOD] * 8), None, 0, None) == L.MOE_EWORKSPACE
    assert lib.moe_expert_ffn_fwd(ctypes.byref(c), *([GOOD] * 8), GOOD, need - 1, None) == L.MOE_EWORKSPACE
    assert lib.moe_expert_ffn_fwd(ctypes.byref(c), *([GOOD] * 8), GOOD, need, None) == L.MOE_EDEVICE
    c32 = _cfg(dtype="f32")
    assert L.moe_workspace_bytes(c32, L.MOE_CALL_FFN_FWD) == 0
    assert lib.moe_expert_ffn_fwd(ctypes.byref(c32), *([GOOD] * 8), None, 0, None) == L.MOE_EDEVICE


def test_wpacked_flag_validation():
    assert _gate(_cfg(wpacked=2)) == L.MOE_EINVAL
    assert "wpacked" in L.moe_last_error()
    assert _gate(_cfg(wpacked=1)) == L.MOE_EDEVICE   # valid; no GPU here


def test_ksplit_flag_validation_and_struct_layout():
    assert _gate(_cfg(ksplit=2)) == L.MOE_EINVAL
    assert "ksplit" in L.moe_last_error()
    assert _gate(_cfg(ksplit=-1)) == L.MOE_EINVAL
    assert _gate(_cfg(ksplit=0)) == L.MOE_EDEVICE     # valid; no GPU here
    # int64 T, ten int32 fields, ksplit, padded to the int64 alignment
    assert ctypes.sizeof(L.moe_cfg) == 56
    assert L.moe_cfg.ksplit.offset == 48
    assert L.moe_block_cfg.moe.offset == 16


def test_dispatch_bpr_validation():
    c = _cfg()
    need = L.moe_workspace_bytes(c, L.MOE_CALL_DISPATCH_BPR)
    # the dispatch workspace plus two token-sized 64-bit element arrays and the order
    assert need >= L.moe_workspace_bytes(c, L.MOE_CALL_DISPATCH) + 16 * c.T
    lib = L._lib
    f = lib.moe_dispatch_bpr
    assert f(ctypes.byref(c), GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, None, None, 0, None) == L.MOE_EWORKSPACE
    assert f(ctypes.byref(c), GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, None, GOOD, need - 1, None) == L.MOE_EWORKSPACE
    assert f(ctypes.byref(c), GOOD, None, GOOD, GOOD, GOOD, GOOD, None, GOOD, need, None) == L.MOE_EINVAL
    assert "logits" in L.moe_last_error()
    assert f(ctypes.byref(c), GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD + 4, GOOD, need, None) == L.MOE_EALIGN
    assert f(ctypes.byref(c), GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, None, GOOD, need, None) == L.MOE_EDEVICE
    assert f(ctypes.byref(c), GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, need, None) == L.MOE_EDEVICE


def test_dispatch_noalloc_validation():
    """The fixed-workspace dispatch validates like moe_dispatch and rejects a
    call whose workspace would exceed the library's fixed 1 MiB, on the host."""
    lib = L._lib
    f = lib.moe_dispatch_noalloc
    c = _cfg()
    assert f(ctypes.byref(c), GOOD, GOOD, None, GOOD, GOOD, GOOD, None) == L.MOE_EDEVICE   # valid; no GPU here
    assert f(ctypes.byref(c), GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, None) == L.MOE_EINVAL    # carry aliases fill
    assert "alias" in L.moe_last_error()
    assert f(ctypes.byref(c), GOOD, None, None, GOOD, GOOD, GOOD, None) == L.MOE_EINVAL
    assert f(ctypes.byref(c), GOOD + 8, GOOD, None, GOOD, GOOD, GOOD, None) == L.MOE_EALIGN
    # 4 * (2 * ceil(T / 256) * E + T * k) bytes: T = 65536, E = 64, k = 2 fits exactly below 1 MiB ...
    fits = _cfg(T=65536, E=64, k=2, C=4096, d_model=128, d_ff=128)
    assert 4 * (2 * 256 * 64 + 65536 * 2) <= 1 << 20
    assert f(ctypes.byref(fits), GOOD, GOOD, None, GOOD, GOOD, GOOD, None) == L.MOE_EDEVICE
    # ... twice the tokens do not
    big = _cfg(T=131072, E=64, k=2, C=4096, d_model=128, d_ff=128)
    assert f(ctypes.byref(big), GOOD, GOOD, None, GOOD, GOOD, GOOD, None) == L.MOE_ESHAPE
    assert "moe_dispatch" in L.moe_last_error()
    # T = 0 is a valid no-op with null token arrays
    z = _cfg(T=0)
    assert f(ctypes.byref(z), None, None, None, GOOD, None, GOOD, None) == L.MOE_EDEVICE


def test_block_cfg_layout_and_dw_order_validation():
    assert ctypes.sizeof(L.moe_block_cfg) == 96 and L.moe_block_cfg.dw_order.offset == 72
    bad = L.make_block_cfg(2, 64, 2, 512, 8, 2, 40, dw_order=[8, 9, 10, 11, 12, 12])
    assert L.moe_block_workspace_bytes(bad, 1) == 0
    assert "dw_order" in L.moe_last_error()
    bad2 = L.make_block_cfg(2, 64, 2, 512, 8, 2, 40, dw_order=[7, 9, 10, 11, 12, 13])
    assert L.moe_block_workspace_bytes(bad2, 1) == 0
    good = L.make_block_cfg(2, 64, 2, 512, 8, 2, 40, dw_order=[13, 12, 11, 10, 9, 8])
    assert L.moe_block_workspace_bytes(good, 1) > 0
    assert L.moe_block_workspace_bytes(L.make_block_cfg(2, 64, 2, 512, 8, 2, 40), 1) > 0


def test_product_times_rejects_null_and_timing_needs_a_device():
    ms = (ctypes.c_double * 6)()
    counts = (ctypes.c_int32 * 6)()
    assert L._lib.moe_product_times(None, counts) == L.MOE_EINVAL
    assert L._lib.moe_product_times(ms, None) == L.MOE_EINVAL
    # no device in this container: starting the record fails cleanly
    assert L._lib.moe_product_timing(1) in (L.MOE_OK, L.MOE_EDEVICE)
    L._lib.moe_product_timing(0)


def test_block_op_times_without_a_timed_call():
    ms = (ctypes.c_double * 14)()
    assert L._lib.moe_block_op_times(ms) in (L.MOE_EINVAL, L.MOE_ELAUNCH)
