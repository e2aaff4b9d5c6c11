"""Helpers for the GPU parity tests: upload seeded inputs, run the HIP layer
through the C ABI, download results, and compare against the oracle.

Float metric (per tensor): max|gpu - ref| / max|ref| <= tol, with tol 1e-5 for
float32 workloads and 2e-2 for bf16 ones.  Integer results are compared
bit-exactly.  Rows of [E][C][*] buffers past an expert's fill are never
compared; the harness fills those buffers with NaN before the run so a kernel
that read an unspecified row would poison its outputs and fail the test.
"""
from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import moe_oracle as O

TOL = {"f32": 1e-5, "bf16": 2e-2}


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def normwise(gpu, ref) -> float:
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    if gpu.size == 0:
        return 0.0
    assert np.all(np.isfinite(gpu)), "non-finite values in GPU output"
    scale = np.max(np.abs(ref))
    err = np.max(np.abs(gpu - ref))
    return float(err / scale) if scale > 0 else float(err)


def assert_close(name, gpu, ref, tol):
    e = normwise(gpu, ref)
    assert e <= tol, f"{name}: normwise error {e:.3e} > {tol:.1e}"
    return e


def to_dev(a, dtype):
    if a is None:
        return None
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to("cuda").to(dtype).contiguous()


def host(t):
    return t.detach().float().cpu().numpy() if t.is_floating_point() else t.detach().cpu().numpy()


EXPERT_X = {"send_buf": "d", "H": "f", "A": "f", "O": "d", "expert_out": "d", "dO": "d", "dH": "f", "dXe": "d"}


ROW_MAJOR_BUFFERS = ("O", "expert_out", "dXe")   # product outputs only the gathers read


def expert_host(t, cfg, X, blocked=True):
    """An [E][C][X] expert buffer as a row-major numpy array (bf16 buffers
    have C padded to a multiple of 16 and, if `blocked`, are stored in
    16 x 32 blocks)."""
    a = host(t)
    E, C = cfg.E, cfg.C
    if cfg.dtype == 1:  # bf16
        Cp = (C + 15) // 16 * 16
        if not blocked:
            return a.reshape(E, Cp, X)[:, :C]
        return a.reshape(E, Cp // 16, X // 32, 16, 32).transpose(0, 1, 3, 2, 4).reshape(E, Cp, X)[:, :C]
    return a.reshape(E, C, X)


def ebuf(b, name):
    """Expert buffer `name` of LayerBuffers b, row-major [E][C][X]."""
    c = b.cfg
    X = c.d_model if EXPERT_X[name] == "d" else c.d_ff
    return expert_host(getattr(b, name), c, X, blocked=name not in ROW_MAJOR_BUFFERS)


def kept_rows(buf, fill, lo=None):
    """Concatenate rows [lo_e, fill_e) of every expert block."""
    E = buf.shape[0]
    lo = np.zeros(E, np.int64) if lo is None else lo
    return np.concatenate([buf[e, int(lo[e]):int(fill[e])] for e in range(E)], axis=0)


def nan_fill(b):
    """Poison every output, so a value a kernel fails to write shows up."""
    for name in ("send_buf", "H", "A", "O", "dO", "dH", "dXe", "dW1", "dW2", "dWg"):
        getattr(b, name).fill_(float("nan"))


def run_layer(L, spec, inp, C, backward=True, dw_stream=None, carry=None, routing="token", ksplit=1):
    """Run gate -> dispatch -> experts -> combine (and the backward) on cuda:0."""
    dt = torch.bfloat16 if spec.dtype == "bf16" else torch.float32
    cfg = L.make_cfg(inp["x"].shape[0], spec.d, spec.f, spec.E, spec.k, C, spec.G, spec.dtype, spec.act,
                     spec.renorm, ksplit=ksplit)
    b = L.alloc_layer(cfg)
    nan_fill(b)
    if carry is not None:
        b.carry.copy_(torch.as_tensor(np.asarray(carry), dtype=torch.int32))
    dev = {n: to_dev(inp[n], dt) for n in ("x", "Wg", "W1", "W2", "dy")}
    bias = None if inp.get("bias") is None else torch.as_tensor(inp["bias"], dtype=torch.float32).cuda()
    L.layer_forward(b, dev["x"], dev["Wg"], bias, dev["W1"], dev["W2"], routing=routing)
    if backward:
        L.layer_backward(b, dev["x"], dev["Wg"], dev["dy"], dw_stream=dw_stream)
    torch.cuda.synchronize()
    return b, dev


def spec_C(spec, T=None):
    return O.capacity(spec.T if T is None else T, spec.E, spec.k, spec.cf_num, spec.cf_den)


def ksplit_xcds(lo, hi, C, ncols, cus=256, tile=256):
    """How many XCDs split the K sums of their last round in a plain-store
    ragged-M expert product (expert_out, dXe) with ksplit = 1: a mirror of the
    product's schedule (256 x 256 tiles; full M-tiles of every expert, then
    its short last M-tile, dealt to 8 XCDs in even contiguous shares; rounds of
    nslot = blocks / 8 tiles; a last round of r tiles is split when
    0 < 4 r <= nslot).  Used to check that a test case exercises the split."""
    tn = -(-ncols // tile)
    tm = -(-(C + 15) // tile)
    blocks = min(cus, 256, tm * tn * len(lo))
    blocks = -(-blocks // 8) * 8
    nslot = blocks // 8
    NF = NP = 0
    for a, b in zip(lo, hi):
        a, b = int(a), int(b)
        span = b - a
        if span <= 0:
            continue
        span += a & 15
        t = -(-span // tile)
        sh = 1 if span % tile else 0
        NF += (t - sh) * tn
        NP += sh * tn
    perF, perP = -(-NF // 8), -(-NP // 8)
    n_split = 0
    for x in range(8):
        nf = max(min(NF, x * perF + perF) - x * perF, 0)
        npp = max(min(NP, x * perP + perP) - x * perP, 0)
        r = (nf + npp) % nslot
        n_split += int(nslot >= 4 and 0 < r and 4 * r <= nslot)
    return n_split


def bf16_ulp(a):
    """Spacing of bfloat16 numbers at |a| (the ulp of a bf16 value of that magnitude)."""
    a = np.abs(np.asarray(a, np.float64))
    e = np.floor(np.log2(np.maximum(a, np.finfo(np.float32).tiny)))
    return np.exp2(e - 7)
