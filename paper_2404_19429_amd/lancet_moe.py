"""Python binding of liblancet_moe.so (ctypes).

Argument marshalling only: every function here has the name of the C-ABI
entry point it calls, checks that each tensor is a contiguous device tensor
of the right dtype and at least the size the call will touch (the C ABI takes
bare pointers and cannot check sizes), and passes pointers and the current
HIP stream.  All computation happens in the HIP kernels.  There is no CPU
fallback: if the library is missing, importing this module raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
#: The in-tree build; LANCET_MOE_LIB may name another build of the same library.
LIB_PATH = os.environ.get("LANCET_MOE_LIB") or os.path.join(_HERE, "liblancet_moe.so")

MOE_OK, MOE_EINVAL, MOE_ESHAPE, MOE_EALIGN, MOE_EDTYPE, MOE_EDEVICE, MOE_ELAUNCH, MOE_EWORKSPACE = 0, -1, -2, -3, -4, -5, -6, -7
MOE_F32, MOE_BF16 = 0, 1
ACTS = {"identity": 0, "relu": 1, "gelu_tanh": 2, "gelu_erf": 3}
MOE_CALL_DISPATCH, MOE_CALL_BWD_DX, MOE_CALL_BWD_DW, MOE_CALL_FFN_FWD, MOE_CALL_DISPATCH_BPR = 0, 1, 2, 3, 4

#: Every symbol include/lancet_moe.h declares.
EXPORTS = ["moe_capacity", "moe_workspace_bytes", "moe_last_error", "moe_gate_topk", "moe_dispatch",
           "moe_dispatch_noalloc", "moe_dispatch_bpr", "moe_pack_weights", "moe_expert_ffn_fwd", "moe_combine", "moe_bwd_dx", "moe_bwd_dw",
           "moe_block_workspace_bytes", "moe_block_chunked", "moe_block_op_times", "moe_block_dw_schedule",
           "moe_dw_schedule", "moe_pipeline_plan", "moe_pipeline_range_cost", "moe_product_timing",
           "moe_product_times"]
#: The expert products moe_product_times reports, in its order.
PRODUCTS = ["fwd1", "fwd2", "dA", "dXe", "dW2", "dW1"]
MOE_BLOCK_FWD, MOE_BLOCK_BWD, MOE_BLOCK_TIMED = 1, 2, 4
#: The block backward's operations (moe_block_op): the chain 0..7, the weight-gradient groups 8..13.
BLOCK_OPS = ["combine_bwd", "expert_dx", "dispatch_bwd", "ln2_bwd", "dattn", "attn_bwd", "da", "ln1_bwd",
             "dw_expert", "dwg", "dln2", "dwo", "dwqkv", "dln1"]
MOE_BOP_DW_EXPERT = 8


class MoeError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"status {status}: {msg}")
        self.status = status


class moe_cfg(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int64), ("d_model", ctypes.c_int32), ("d_ff", ctypes.c_int32),
                ("E", ctypes.c_int32), ("k", ctypes.c_int32), ("C", ctypes.c_int32), ("G", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("act", ctypes.c_int32), ("renorm", ctypes.c_int32),
                ("wpacked", ctypes.c_int32), ("ksplit", ctypes.c_int32)]


class moe_block_cfg(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("S", ctypes.c_int32), ("heads", ctypes.c_int32), ("moe", moe_cfg),
                ("dw_order", ctypes.c_int32 * 6)]


BLOCK_WEIGHTS = ["ln1_g", "ln1_b", "Wqkv", "Wo", "ln2_g", "ln2_b", "Wg", "W1", "W2"]
BLOCK_GRADS = ["dln1_g", "dln1_b", "dWqkv", "dWo", "dln2_g", "dln2_b", "dWg", "dW1", "dW2"]
BLOCK_ACTS_FWD = ["a", "ln1_mean", "ln1_rstd", "qkv", "attn", "lse", "h", "ln2_mean", "ln2_rstd", "m", "logits",
                  "idx", "w", "slot", "fill", "send_buf", "H", "A", "expert_out", "W1p", "W2p"]
BLOCK_ACTS_BWD = ["dO", "dH", "dXe", "dlogits", "dm", "dh", "dattn", "delta", "dqkv", "da"]


class moe_block_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in BLOCK_WEIGHTS]


class moe_block_grads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in BLOCK_GRADS]


class moe_block_acts(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in BLOCK_ACTS_FWD + BLOCK_ACTS_BWD]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2404_19429_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    CFG = ctypes.POINTER(moe_cfg)
    sig = {
        "moe_capacity": (I32, [I64, I32, I32, I32, I32]),
        "moe_workspace_bytes": (SZ, [CFG, I32]),
        "moe_last_error": (ctypes.c_char_p, []),
        "moe_gate_topk": (I32, [CFG, P, P, P, P, P, P, P]),
        "moe_dispatch": (I32, [CFG, P, P, P, P, P, P, P, SZ, P]),
        "moe_dispatch_noalloc": (I32, [CFG, P, P, P, P, P, P, P]),
        "moe_dispatch_bpr": (I32, [CFG, P, P, P, P, P, P, P, P, SZ, P]),
        "moe_pack_weights": (I32, [CFG, P, P, P, P, P]),
        "moe_expert_ffn_fwd": (I32, [CFG, P, P, P, P, P, P, P, P, P, SZ, P]),
        "moe_combine": (I32, [CFG, P, P, P, P, P, P]),
        "moe_bwd_dx": (I32, [CFG] + [P] * 18 + [SZ, P]),
        "moe_bwd_dw": (I32, [CFG] + [P] * 12 + [SZ, P]),
        "moe_dw_schedule": (I32, [I32, P, P, I32, P, P, P, P, P]),
        "moe_block_op_times": (I32, [P]),
        "moe_product_timing": (I32, [I32]),
        "moe_product_times": (I32, [P, P]),
        "moe_block_dw_schedule": (I32, [P, ctypes.c_double, P, P, P]),
        "moe_pipeline_plan": (I32, [I32, I32, P, P, P, I32, P, P, P, P, P]),
        "moe_pipeline_range_cost": (I32, [I32, I32, P, P, P, I32, I32, I32, P]),
        "moe_block_workspace_bytes": (SZ, [ctypes.POINTER(moe_block_cfg), I32]),
        "moe_block_chunked": (I32, [ctypes.POINTER(moe_block_cfg), ctypes.POINTER(moe_block_weights),
                                    ctypes.POINTER(moe_block_grads), P, P, P, P, ctypes.POINTER(moe_block_acts),
                                    I32, I32, ctypes.POINTER(P), P, SZ]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype, fn.argtypes = res, args
    return lib


_lib = _load()


# ----------------------------------------------------------------------- helpers
def make_cfg(T, d_model, d_ff, E, k, C, G=1, dtype="bf16", act="gelu_tanh", renorm=1, wpacked=0,
             ksplit=1) -> moe_cfg:
    dt = {"bf16": MOE_BF16, "f32": MOE_F32}[dtype] if isinstance(dtype, str) else int(dtype)
    return moe_cfg(int(T), int(d_model), int(d_ff), int(E), int(k), int(C), int(G), dt,
                   ACTS[act] if isinstance(act, str) else int(act), int(renorm), int(wpacked), int(ksplit))


def torch_dtype(cfg: moe_cfg):
    return torch.bfloat16 if cfg.dtype == MOE_BF16 else torch.float32


def rows_alloc(cfg: moe_cfg) -> int:
    """Rows per expert of an [E][C][X] buffer: C rounded up to 16 for bf16 (blocked layout), C for float."""
    return (cfg.C + 15) // 16 * 16 if cfg.dtype == MOE_BF16 else cfg.C


def expert_numel(cfg: moe_cfg, X: int) -> int:
    """Elements of an [E][C][X] expert buffer (see the layout note in include/lancet_moe.h)."""
    return cfg.E * rows_alloc(cfg) * X


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _ptr(t: Optional[torch.Tensor], name: str, dtype, numel: int, nullable: bool = False):
    if t is None:
        if nullable:
            return None
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() < numel:
        raise ValueError(f"{name} has {t.numel()} elements, the call touches {numel}")
    return t.data_ptr() if t.numel() else None


def _check(st: int):
    if st != MOE_OK:
        raise MoeError(st, _lib.moe_last_error().decode())


# ------------------------------------------------------------------- entry points
def moe_capacity(T: int, E: int, k: int, cf_num: int, cf_den: int) -> int:
    return int(_lib.moe_capacity(T, E, k, cf_num, cf_den))


def moe_workspace_bytes(cfg: moe_cfg, call: int) -> int:
    return int(_lib.moe_workspace_bytes(ctypes.byref(cfg), call))


def moe_last_error() -> str:
    return _lib.moe_last_error().decode()


def moe_gate_topk(cfg, x, Wg, bias, logits, idx, w, stream=None):
    dt = torch_dtype(cfg)
    T, d, E, k = cfg.T, cfg.d_model, cfg.E, cfg.k
    _check(_lib.moe_gate_topk(ctypes.byref(cfg), _ptr(x, "x", dt, T * d), _ptr(Wg, "Wg", dt, E * d),
                              _ptr(bias, "bias", torch.float32, E, nullable=True),
                              _ptr(logits, "logits", torch.float32, T * E), _ptr(idx, "idx", torch.int32, T * k),
                              _ptr(w, "w", torch.float32, T * k), _stream(stream)))


def moe_dispatch(cfg, x, idx, carry, fill, slot, send_buf, ws, stream=None):
    dt = torch_dtype(cfg)
    T, d, E, k = cfg.T, cfg.d_model, cfg.E, cfg.k
    need = moe_workspace_bytes(cfg, MOE_CALL_DISPATCH)
    _check(_lib.moe_dispatch(ctypes.byref(cfg), _ptr(x, "x", dt, T * d), _ptr(idx, "idx", torch.int32, T * k),
                             _ptr(carry, "carry", torch.int32, E, nullable=True), _ptr(fill, "fill", torch.int32, E),
                             _ptr(slot, "slot", torch.int32, T * k), _ptr(send_buf, "send_buf", dt, expert_numel(cfg, d)),
                             _ptr(ws, "ws", torch.uint8, need, nullable=need == 0),
                             ws.numel() if ws is not None else 0, _stream(stream)))


def moe_dispatch_noalloc(cfg, x, idx, carry, fill, slot, send_buf, stream=None):
    dt = torch_dtype(cfg)
    T, d, E, k = cfg.T, cfg.d_model, cfg.E, cfg.k
    _check(_lib.moe_dispatch_noalloc(ctypes.byref(cfg), _ptr(x, "x", dt, T * d), _ptr(idx, "idx", torch.int32, T * k),
                                     _ptr(carry, "carry", torch.int32, E, nullable=True),
                                     _ptr(fill, "fill", torch.int32, E), _ptr(slot, "slot", torch.int32, T * k),
                                     _ptr(send_buf, "send_buf", dt, expert_numel(cfg, d)), _stream(stream)))


def moe_dispatch_bpr(cfg, x, logits, idx, fill, slot, send_buf, order, ws, stream=None):
    dt = torch_dtype(cfg)
    T, d, E, k = cfg.T, cfg.d_model, cfg.E, cfg.k
    need = moe_workspace_bytes(cfg, MOE_CALL_DISPATCH_BPR)
    _check(_lib.moe_dispatch_bpr(ctypes.byref(cfg), _ptr(x, "x", dt, T * d),
                                 _ptr(logits, "logits", torch.float32, T * E), _ptr(idx, "idx", torch.int32, T * k),
                                 _ptr(fill, "fill", torch.int32, E), _ptr(slot, "slot", torch.int32, T * k),
                                 _ptr(send_buf, "send_buf", dt, expert_numel(cfg, d)),
                                 _ptr(order, "order", torch.int32, T, nullable=True),
                                 _ptr(ws, "ws", torch.uint8, need, nullable=need == 0),
                                 ws.numel() if ws is not None else 0,
                                 _stream(stream)))


def moe_dw_schedule(kinds, times, edges):
    """Weight-gradient schedule pass on the host (see include/lancet_moe.h).
    kinds: 0 other / 1 all-to-all / 2 weight gradient; times: per instruction;
    edges: (src, dst) pairs.  Returns (assign [n] int32, order [n] int32, overlap)."""
    import numpy as np
    kinds = np.ascontiguousarray(kinds, np.int32)
    times = np.ascontiguousarray(times, np.float64)
    e = np.ascontiguousarray(np.asarray(edges, np.int32).reshape(-1, 2))
    src, dst = np.ascontiguousarray(e[:, 0]), np.ascontiguousarray(e[:, 1])
    n = int(kinds.size)
    assign = np.empty(n, np.int32)
    order = np.empty(n, np.int32)
    ov = ctypes.c_double(0.0)
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p) if a.size else None
    _check(_lib.moe_dw_schedule(n, p(kinds), p(times), int(src.size), p(src), p(dst), p(assign), p(order),
                                ctypes.byref(ov)))
    return assign, order, ov.value


def _pipeline_args(kinds, times, join):
    import numpy as np
    kinds = np.ascontiguousarray(kinds, np.int32)
    times = np.ascontiguousarray(times, np.float64).reshape(kinds.size, -1)
    join = np.ascontiguousarray(join, np.float64)
    assert times.shape[1] == join.size, "times needs one column per k = 1..K"
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p) if a.size else None
    return kinds, times, join, p


def moe_pipeline_plan(kinds, times, join, G=0):
    """Partition-range plan on the host (see include/lancet_moe.h).  times [N][K],
    join [K].  Returns (T(N), [(begin, end, k), ...] 1-based inclusive)."""
    import numpy as np
    kinds, times, join, p = _pipeline_args(kinds, times, join)
    N, K = int(kinds.size), int(join.size)
    b, e, k = (np.zeros(max(N, 1), np.int32) for _ in range(3))
    n_seg, total = ctypes.c_int32(0), ctypes.c_double(0.0)
    _check(_lib.moe_pipeline_plan(N, K, p(kinds), p(times), p(join), int(G), p(b), p(e), p(k), ctypes.byref(n_seg),
                                  ctypes.byref(total)))
    return total.value, [(int(b[q]), int(e[q]), int(k[q])) for q in range(n_seg.value)]


def moe_pipeline_range_cost(kinds, times, join, i, n, k):
    kinds, times, join, p = _pipeline_args(kinds, times, join)
    c = ctypes.c_double(0.0)
    _check(_lib.moe_pipeline_range_cost(int(kinds.size), int(join.size), p(kinds), p(times), p(join), int(i), int(n),
                                        int(k), ctypes.byref(c)))
    return c.value


def moe_pack_weights(cfg, W1, W2, W1p, W2p, stream=None):
    dt = torch_dtype(cfg)
    n = cfg.E * cfg.d_ff * cfg.d_model
    _check(_lib.moe_pack_weights(ctypes.byref(cfg), _ptr(W1, "W1", dt, n), _ptr(W2, "W2", dt, n),
                                 _ptr(W1p, "W1p", dt, n), _ptr(W2p, "W2p", dt, n), _stream(stream)))


def moe_expert_ffn_fwd(cfg, send_buf, row_begin, row_end, W1p, W2p, H, A, expert_out, ws=None, stream=None):
    dt = torch_dtype(cfg)
    d, f, E = cfg.d_model, cfg.d_ff, cfg.E
    need = moe_workspace_bytes(cfg, MOE_CALL_FFN_FWD)
    _check(_lib.moe_expert_ffn_fwd(ctypes.byref(cfg), _ptr(send_buf, "send_buf", dt, expert_numel(cfg, d)),
                                   _ptr(row_begin, "row_begin", torch.int32, E, nullable=True),
                                   _ptr(row_end, "row_end", torch.int32, E), _ptr(W1p, "W1p", dt, E * f * d),
                                   _ptr(W2p, "W2p", dt, E * d * f), _ptr(H, "H", dt, expert_numel(cfg, f)),
                                   _ptr(A, "A", dt, expert_numel(cfg, f)),
                                   _ptr(expert_out, "expert_out", dt, expert_numel(cfg, d)),
                                   _ptr(ws, "ws", torch.uint8, need, nullable=need == 0),
                                   ws.numel() if ws is not None else 0, _stream(stream)))


def moe_combine(cfg, expert_out, idx, slot, w, y, stream=None):
    dt = torch_dtype(cfg)
    T, d, k = cfg.T, cfg.d_model, cfg.k
    _check(_lib.moe_combine(ctypes.byref(cfg), _ptr(expert_out, "expert_out", dt, expert_numel(cfg, d)),
                            _ptr(idx, "idx", torch.int32, T * k), _ptr(slot, "slot", torch.int32, T * k),
                            _ptr(w, "w", torch.float32, T * k), _ptr(y, "y", dt, T * d), _stream(stream)))


def moe_bwd_dx(cfg, Wg, logits, idx, w, slot, row_begin, row_end, H, expert_out, W1p, W2p, dy, dO, dH, dXe,
               dlogits, dx, ws=None, stream=None):
    dt = torch_dtype(cfg)
    T, d, f, E, k = cfg.T, cfg.d_model, cfg.d_ff, cfg.E, cfg.k
    nd, nf = expert_numel(cfg, d), expert_numel(cfg, f)
    need = moe_workspace_bytes(cfg, MOE_CALL_BWD_DX)
    _check(_lib.moe_bwd_dx(ctypes.byref(cfg), _ptr(Wg, "Wg", dt, E * d), _ptr(logits, "logits", torch.float32, T * E),
                           _ptr(idx, "idx", torch.int32, T * k), _ptr(w, "w", torch.float32, T * k),
                           _ptr(slot, "slot", torch.int32, T * k),
                           _ptr(row_begin, "row_begin", torch.int32, E, nullable=True),
                           _ptr(row_end, "row_end", torch.int32, E), _ptr(H, "H", dt, nf),
                           _ptr(expert_out, "expert_out", dt, nd), _ptr(W1p, "W1p", dt, E * f * d),
                           _ptr(W2p, "W2p", dt, E * d * f), _ptr(dy, "dy", dt, T * d), _ptr(dO, "dO", dt, nd),
                           _ptr(dH, "dH", dt, nf), _ptr(dXe, "dXe", dt, nd),
                           _ptr(dlogits, "dlogits", torch.float32, T * E), _ptr(dx, "dx", dt, T * d),
                           _ptr(ws, "ws", torch.uint8, need, nullable=need == 0),
                           ws.numel() if ws is not None else 0, _stream(stream)))


def moe_bwd_dw(cfg, x, dlogits, row_begin, row_end, send_buf, A, dO, dH, dW1, dW2, dWg, ws, stream=None):
    dt = torch_dtype(cfg)
    T, d, f, E = cfg.T, cfg.d_model, cfg.d_ff, cfg.E
    nd, nf = expert_numel(cfg, d), expert_numel(cfg, f)
    need = moe_workspace_bytes(cfg, MOE_CALL_BWD_DW)
    _check(_lib.moe_bwd_dw(ctypes.byref(cfg), _ptr(x, "x", dt, T * d, nullable=T == 0),
                           _ptr(dlogits, "dlogits", torch.float32, T * E),
                           _ptr(row_begin, "row_begin", torch.int32, E, nullable=True),
                           _ptr(row_end, "row_end", torch.int32, E), _ptr(send_buf, "send_buf", dt, nd),
                           _ptr(A, "A", dt, nf), _ptr(dO, "dO", dt, nd), _ptr(dH, "dH", dt, nf),
                           _ptr(dW1, "dW1", dt, E * f * d), _ptr(dW2, "dW2", dt, E * d * f),
                           _ptr(dWg, "dWg", torch.float32, E * d),
                           _ptr(ws, "ws", torch.uint8, need, nullable=need == 0),
                           ws.numel() if ws is not None else 0, _stream(stream)))


# ------------------------------------------------------------- layer step driver
@dataclass
class LayerBuffers:
    """Device tensors of one MoE layer step (allocated once, reused every step)."""
    cfg: moe_cfg
    logits: torch.Tensor
    idx: torch.Tensor
    w: torch.Tensor
    carry: torch.Tensor
    fill: torch.Tensor
    slot: torch.Tensor
    send_buf: torch.Tensor
    H: torch.Tensor
    A: torch.Tensor
    O: torch.Tensor
    y: torch.Tensor
    dO: torch.Tensor
    dH: torch.Tensor
    dXe: torch.Tensor
    dlogits: torch.Tensor
    dx: torch.Tensor
    dW1: torch.Tensor
    dW2: torch.Tensor
    dWg: torch.Tensor
    W1p: torch.Tensor
    W2p: torch.Tensor
    ws_dispatch: torch.Tensor
    ws_ffn: torch.Tensor
    ws_dx: torch.Tensor
    ws_dw: torch.Tensor
    order: torch.Tensor       # batch-prioritized routing: the visiting order
    ws_bpr: torch.Tensor


def alloc_layer(cfg: moe_cfg, device="cuda") -> LayerBuffers:
    dt = torch_dtype(cfg)
    T, d, f, E, k, C = cfg.T, cfg.d_model, cfg.d_ff, cfg.E, cfg.k, cfg.C
    e = lambda *s, dtype=dt: torch.empty(*s, dtype=dtype, device=device)
    nd, nf = expert_numel(cfg, d), expert_numel(cfg, f)
    return LayerBuffers(
        cfg=cfg, logits=e(T, E, dtype=torch.float32), idx=e(T, k, dtype=torch.int32), w=e(T, k, dtype=torch.float32),
        carry=torch.zeros(E, dtype=torch.int32, device=device), fill=e(E, dtype=torch.int32),
        slot=e(T, k, dtype=torch.int32), send_buf=e(nd), H=e(nf), A=e(nf), O=e(nd), y=e(T, d),
        dO=e(nd), dH=e(nf), dXe=e(nd), dlogits=e(T, E, dtype=torch.float32), dx=e(T, d),
        dW1=e(E, f, d), dW2=e(E, d, f), dWg=e(E, d, dtype=torch.float32), W1p=e(E * f * d), W2p=e(E * d * f),
        ws_dispatch=e(max(16, moe_workspace_bytes(cfg, MOE_CALL_DISPATCH)), dtype=torch.uint8),
        ws_ffn=e(max(16, moe_workspace_bytes(cfg, MOE_CALL_FFN_FWD)), dtype=torch.uint8),
        ws_dx=e(max(16, moe_workspace_bytes(cfg, MOE_CALL_BWD_DX)), dtype=torch.uint8),
        ws_dw=e(max(16, moe_workspace_bytes(cfg, MOE_CALL_BWD_DW)), dtype=torch.uint8),
        order=e(max(1, T), dtype=torch.int32),
        ws_bpr=e(max(16, moe_workspace_bytes(cfg, MOE_CALL_DISPATCH_BPR)), dtype=torch.uint8),
    )


def layer_forward(b: LayerBuffers, x, Wg, bias, W1, W2, stream=None, routing="token"):
    """weight packing -> gate -> dispatch -> experts -> combine, all on one stream.
    routing "bpr": batch-prioritized capacity order (no carry-in; b.carry must be zero)."""
    c = b.cfg
    moe_pack_weights(c, W1, W2, b.W1p, b.W2p, stream)
    moe_gate_topk(c, x, Wg, bias, b.logits, b.idx, b.w, stream)
    if routing == "bpr":
        moe_dispatch_bpr(c, x, b.logits, b.idx, b.fill, b.slot, b.send_buf, b.order, b.ws_bpr, stream)
    else:
        moe_dispatch(c, x, b.idx, b.carry, b.fill, b.slot, b.send_buf, b.ws_dispatch, stream)
    moe_expert_ffn_fwd(c, b.send_buf, b.carry, b.fill, b.W1p, b.W2p, b.H, b.A, b.O, b.ws_ffn, stream)
    moe_combine(c, b.O, b.idx, b.slot, b.w, b.y, stream)


def layer_backward(b: LayerBuffers, x, Wg, dy, stream=None, dw_stream=None):
    """dX chain on `stream` (with the weights packed by layer_forward); the dW
    products on `dw_stream` (default: same stream), ordered after the dX chain by an event."""
    c = b.cfg
    moe_bwd_dx(c, Wg, b.logits, b.idx, b.w, b.slot, b.carry, b.fill, b.H, b.O, b.W1p, b.W2p, dy, b.dO, b.dH, b.dXe,
               b.dlogits, b.dx, b.ws_dx, stream)
    if dw_stream is not None:
        ev = torch.cuda.Event()
        ev.record(stream if isinstance(stream, torch.cuda.Stream) else torch.cuda.current_stream())
        dw_stream.wait_event(ev)
    moe_bwd_dw(c, x, b.dlogits, b.carry, b.fill, b.send_buf, b.A, b.dO, b.dH, b.dW1, b.dW2, b.dWg, b.ws_dw,
               dw_stream if dw_stream is not None else stream)


# ------------------------------------------------------------------------ block
def make_block_cfg(B, S, heads, d_ff, E, k, C, G=1, act="gelu_tanh", renorm=1, dw_order=None,
                   wpacked=0) -> moe_block_cfg:
    """dw_order: the weight-gradient groups (8..13) in launch order; None = the default order.
    wpacked: 1 = the block's W1, W2 are the packed copies and dW1, dW2 come packed."""
    d = 128 * heads
    order = (ctypes.c_int32 * 6)(*([-1] * 6 if dw_order is None else [int(v) for v in dw_order]))
    return moe_block_cfg(int(B), int(S), int(heads),
                         make_cfg(B * S, d, d_ff, E, k, C, G, "bf16", act, renorm, wpacked=wpacked), order)


def moe_product_timing(on):
    """Start (True) or stop (False) recording per-product events on this thread; either clears the record."""
    _check(_lib.moe_product_timing(1 if on else 0))


def moe_product_times():
    """(ms, counts) per expert product (PRODUCTS order) since the last clear; clears the record."""
    import numpy as np
    ms = np.zeros(len(PRODUCTS), np.float64)
    counts = np.zeros(len(PRODUCTS), np.int32)
    _check(_lib.moe_product_times(ms.ctypes.data, counts.ctypes.data))
    return ms, counts


def moe_block_op_times():
    """Durations (ms) of the backward operations of this thread's last timed block call (BLOCK_OPS order)."""
    import numpy as np
    ms = np.zeros(len(BLOCK_OPS), np.float64)
    _check(_lib.moe_block_op_times(ms.ctypes.data))
    return ms


def moe_block_dw_schedule(op_ms, a2a_ms):
    """The block backward's weight-gradient schedule: (dw_order [6], assign [16], overlap)."""
    import numpy as np
    t = np.ascontiguousarray(op_ms, np.float64)
    assert t.size == len(BLOCK_OPS)
    order = np.empty(6, np.int32)
    assign = np.empty(16, np.int32)
    ov = ctypes.c_double(0.0)
    _check(_lib.moe_block_dw_schedule(t.ctypes.data, float(a2a_ms), order.ctypes.data, assign.ctypes.data,
                                      ctypes.byref(ov)))
    return order, assign, ov.value


def block_shapes(cfg: moe_block_cfg, n_chunks: int):
    """{name: (numel, dtype)} of every weight, gradient and activation of the block."""
    m = cfg.moe
    T, d, f, E, k = m.T, m.d_model, m.d_ff, m.E, m.k
    nd, nf = expert_numel(m, d), expert_numel(m, f)
    Sp = (cfg.S + 63) // 64 * 64
    st = cfg.B * cfg.heads * Sp
    bf, f32, i32 = torch.bfloat16, torch.float32, torch.int32
    return {
        "ln1_g": (d, bf), "ln1_b": (d, bf), "Wqkv": (3 * d * d, bf), "Wo": (d * d, bf), "ln2_g": (d, bf),
        "ln2_b": (d, bf), "Wg": (E * d, bf), "W1": (E * f * d, bf), "W2": (E * d * f, bf),
        "dln1_g": (d, f32), "dln1_b": (d, f32), "dWqkv": (3 * d * d, bf), "dWo": (d * d, bf), "dln2_g": (d, f32),
        "dln2_b": (d, f32), "dWg": (E * d, f32), "dW1": (E * f * d, bf), "dW2": (E * d * f, bf),
        "a": (T * d, bf), "ln1_mean": (T, f32), "ln1_rstd": (T, f32), "qkv": (T * 3 * d, bf), "attn": (T * d, bf),
        "lse": (st, f32), "h": (T * d, bf), "ln2_mean": (T, f32), "ln2_rstd": (T, f32), "m": (T * d, bf),
        "logits": (T * E, f32), "idx": (T * k, i32), "w": (T * k, f32), "slot": (T * k, i32),
        "fill": (n_chunks * E, i32), "send_buf": (nd, bf), "H": (nf, bf), "A": (nf, bf),
        "expert_out": (nd, bf), "W1p": (E * f * d, bf), "W2p": (E * d * f, bf), "dO": (nd, bf), "dH": (nf, bf),
        "dXe": (nd, bf),
        "dlogits": (T * E, f32), "dm": (T * d, bf), "dh": (T * d, bf), "dattn": (T * d, bf), "delta": (st, f32),
        "dqkv": (T * 3 * d, bf), "da": (T * d, bf),
    }


def moe_block_workspace_bytes(cfg: moe_block_cfg, n_chunks: int) -> int:
    return int(_lib.moe_block_workspace_bytes(ctypes.byref(cfg), n_chunks))


def moe_block_chunked(cfg: moe_block_cfg, weights: dict, grads: Optional[dict], x, out, dy, dx, acts: dict,
                      passes: int, n_chunks: int, streams, ws):
    """streams: three torch.cuda.Stream (or raw handles) -- compute, data movement, weight gradients."""
    shp = block_shapes(cfg, n_chunks)
    T, d = cfg.moe.T, cfg.moe.d_model
    bwd = bool(passes & MOE_BLOCK_BWD)
    fwd = bool(passes & MOE_BLOCK_FWD)
    w = moe_block_weights(*[_ptr(weights[n], n, shp[n][1], shp[n][0]) for n in BLOCK_WEIGHTS])
    g = None
    if bwd:
        g = moe_block_grads(*[_ptr(grads[n], n, shp[n][1], shp[n][0]) for n in BLOCK_GRADS])
    names = BLOCK_ACTS_FWD + (BLOCK_ACTS_BWD if bwd else [])
    a = moe_block_acts(*[_ptr(acts[n], n, shp[n][1], shp[n][0]) if n in names else None
                         for n in BLOCK_ACTS_FWD + BLOCK_ACTS_BWD])
    need = moe_block_workspace_bytes(cfg, n_chunks)
    st = (ctypes.c_void_p * 3)(*[_stream(s) for s in streams])
    _check(_lib.moe_block_chunked(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(g) if g is not None else None,
                                  _ptr(x, "x", torch.bfloat16, T * d),
                                  _ptr(out, "out", torch.bfloat16, T * d) if fwd else None,
                                  _ptr(dy, "dy", torch.bfloat16, T * d) if bwd else None,
                                  _ptr(dx, "dx", torch.bfloat16, T * d) if bwd else None,
                                  ctypes.byref(a), int(passes), int(n_chunks), st,
                                  _ptr(ws, "ws", torch.uint8, need), ws.numel(), ))


def alloc_block(cfg: moe_block_cfg, n_chunks: int, device="cuda", names=None) -> dict:
    """Empty device tensors for the block's gradients and activations (and its
    workspace under "ws"); weights are the caller's."""
    shp = block_shapes(cfg, n_chunks)
    out = {}
    for n in BLOCK_GRADS + BLOCK_ACTS_FWD + BLOCK_ACTS_BWD:
        if names is None or n in names:
            numel, dt = shp[n]
            out[n] = torch.empty(numel, dtype=dt, device=device)
    out["ws"] = torch.empty(max(16, moe_block_workspace_bytes(cfg, n_chunks)), dtype=torch.uint8, device=device)
    return out
