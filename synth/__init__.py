"""Seeded synthetic inputs for the MoE-layer training step.

This module is shared by the CPU oracle and by the HIP path's tests and
benchmark.  It holds workload shapes and random number generation only: no
step of the method (gating, capacity, dispatch, experts, combine, gradients)
is computed here.

The paper trains GPT-2 MoE models on WikiText (Evaluation, "Benchmark Models
and Datasets").  The MoE layer consumes hidden states, not token ids, so
seeded Gaussian activations stand in for the dataset; layer widths, expert
counts and per-GPU token counts follow the paper's workloads.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Optional

import numpy as np

__all__ = ["LayerSpec", "BlockSpec", "CONFIGS", "layer_spec", "block_spec",
           "round_bf16", "layer_inputs", "block_inputs", "routing_logits"]


@dataclass(frozen=True)
class LayerSpec:
    """Shape and numerics of one MoE layer workload (one GPU's share)."""
    name: str
    T: int                 # tokens on this GPU
    d: int                 # d_model
    f: int                 # d_ff (expert FFN inner width)
    E: int                 # experts
    k: int                 # top-k
    cf_num: int            # capacity factor as a rational cf_num / cf_den
    cf_den: int
    dtype: str             # "f32" or "bf16": storage type of activations/weights
    act: str               # "relu" | "gelu_tanh" | "gelu_erf" | "identity"
    renorm: int            # 1: top-k weights renormalised over the selected experts
    G: int = 1             # destination slices of the send buffer (E % G == 0)
    x_std: float = 1.0
    wg_std: float = 0.02
    w_std: float = 0.02
    zipf_s: float = 0.0    # >0: per-expert logit offset -s*ln(rank), seeded rank permutation
    seed: int = 0


@dataclass(frozen=True)
class BlockSpec:
    """Pre-LN transformer block whose FFN is an MoE layer."""
    name: str
    B: int
    S: int
    d: int
    heads: int
    moe: LayerSpec = field(repr=False)
    n_chunks: int = 4
    seed: int = 0


def _cfg(**kw) -> LayerSpec:
    return LayerSpec(**kw)


#: The five workloads.  Numbers are the sizes; nothing else.
CONFIGS = {
    1: _cfg(name="tiny_fp32", T=256, d=64, f=256, E=4, k=1, cf_num=5, cf_den=4,
            dtype="f32", act="relu", renorm=0, seed=1001),
    2: _cfg(name="layer_bf16_T8192_d1024_f4096_E16", T=8192, d=1024, f=4096, E=16, k=2,
            cf_num=5, cf_den=4, dtype="bf16", act="gelu_tanh", renorm=1, seed=1002),
    3: _cfg(name="ep_share_bf16_T16384_d2048_f8192_E8", T=16384, d=2048, f=8192, E=8, k=2,
            cf_num=5, cf_den=4, dtype="bf16", act="gelu_tanh", renorm=1, G=8, seed=1003),
    4: _cfg(name="zipf_skew_bf16_T32768_d1024_f4096_E64", T=32768, d=1024, f=4096, E=64, k=2,
            cf_num=2, cf_den=1, dtype="bf16", act="gelu_tanh", renorm=1, zipf_s=1.2,
            seed=1004),
}

_BLOCK5_MOE = _cfg(name="block_moe_bf16", T=16384, d=2048, f=8192, E=16, k=2, cf_num=5,
                   cf_den=4, dtype="bf16", act="gelu_tanh", renorm=1, seed=1005)
BLOCK5 = BlockSpec(name="block_bf16_B8_S2048_d2048_h16_E16", B=8, S=2048, d=2048, heads=16,
                   moe=_BLOCK5_MOE, n_chunks=4, seed=1005)


def layer_spec(n: int, **overrides) -> LayerSpec:
    """Config n (1-4), optionally with fields overridden (smaller parity cases)."""
    return replace(CONFIGS[n], **overrides)


def block_spec(**overrides) -> BlockSpec:
    moe_over = {k[4:]: v for k, v in overrides.items() if k.startswith("moe_")}
    rest = {k: v for k, v in overrides.items() if not k.startswith("moe_")}
    b = replace(BLOCK5, **rest)
    moe = replace(b.moe, T=b.B * b.S, d=b.d, **moe_over)
    return replace(b, moe=moe)


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); result stays float32.

    Input generation only: the generated values are exactly representable in
    bfloat16, so the GPU path and the oracle consume identical numbers.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    u = ((u + np.uint64(0x7FFF) + lsb) & np.uint64(0xFFFF0000)).astype(np.uint32)
    return u.view(np.float32)


def _normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    out = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        out *= np.float32(std)
    return out


def _finish(a: np.ndarray, dtype: str) -> np.ndarray:
    return round_bf16(a) if dtype == "bf16" else np.ascontiguousarray(a, dtype=np.float32)


def layer_inputs(spec: LayerSpec, seed: Optional[int] = None, with_weights: bool = True):
    """Seeded inputs of one MoE layer, as float32 numpy arrays.

    Streams are spawned from SeedSequence(seed) in a fixed order: x, Wg, W1, W2,
    dy, zipf-permutation.  For bf16 workloads every array except the gate
    offset is rounded to bfloat16 values.  Layouts are nn.Linear [out][in]:
    Wg [E][d], W1 [E][f][d], W2 [E][d][f]; activations row-major [T][d].
    ``bias`` is None unless the workload has a Zipf skew: then it is the
    per-expert offset -s*ln(rank_e) with rank a seeded permutation of 1..E
    (the log of the Zipf pmf with its constant dropped), float32.
    """
    seed = spec.seed if seed is None else seed
    ss = np.random.SeedSequence(seed)
    s_x, s_wg, s_w1, s_w2, s_dy, s_zipf = ss.spawn(6)
    T, d, f, E = spec.T, spec.d, spec.f, spec.E
    out = {}
    out["x"] = _finish(_normal(np.random.default_rng(s_x), (T, d), spec.x_std), spec.dtype)
    out["Wg"] = _finish(_normal(np.random.default_rng(s_wg), (E, d), spec.wg_std), spec.dtype)
    if with_weights:
        out["W1"] = _finish(_normal(np.random.default_rng(s_w1), (E, f, d), spec.w_std), spec.dtype)
        out["W2"] = _finish(_normal(np.random.default_rng(s_w2), (E, d, f), spec.w_std), spec.dtype)
    out["dy"] = _finish(_normal(np.random.default_rng(s_dy), (T, d), 1.0), spec.dtype)
    if spec.zipf_s > 0:
        rank = np.random.default_rng(s_zipf).permutation(E) + 1
        out["bias"] = (-spec.zipf_s * np.log(rank.astype(np.float64))).astype(np.float32)
    else:
        out["bias"] = None
    return out


def routing_logits(T: int, E: int, seed: int, ties: float = 0.0, scale: float = 1.0):
    """Float32 logits for routing-only tests.

    With ``ties`` > 0 a fraction of tokens get exactly equal values planted on
    a random pair (or all) of experts, so that tie-breaking is exercised.
    """
    rng = np.random.default_rng(np.random.SeedSequence(seed))
    l = (rng.standard_normal((T, E)) * scale).astype(np.float32)
    if ties > 0:
        n_tie = int(T * ties)
        rows = rng.choice(T, size=n_tie, replace=False)
        for i, t in enumerate(rows):
            if i % 3 == 0:
                l[t, :] = l[t, 0]                      # all equal
            else:
                a, b = rng.choice(E, size=2, replace=False)
                l[t, b] = l[t, a]                      # one planted pair
    return l


def block_inputs(spec: BlockSpec, seed: Optional[int] = None):
    """Seeded inputs of the pre-LN MoE transformer block (float32 arrays, bf16 values).

    Streams from SeedSequence(seed) in the order: x, Wg, W1, W2, dy, zipf, LN,
    Wqkv, Wo.  LN gains are 1 + N(0, 0.02), biases N(0, 0.02).
    """
    seed = spec.seed if seed is None else seed
    m = spec.moe
    ss = np.random.SeedSequence(seed)
    s_x, s_wg, s_w1, s_w2, s_dy, _s_zipf, s_ln, s_qkv, s_o = ss.spawn(9)
    B, S, d, E, f = spec.B, spec.S, spec.d, m.E, m.f
    T = B * S
    dt = m.dtype
    out = {
        "x": _finish(_normal(np.random.default_rng(s_x), (T, d), 1.0), dt),
        "Wg": _finish(_normal(np.random.default_rng(s_wg), (E, d), m.wg_std), dt),
        "W1": _finish(_normal(np.random.default_rng(s_w1), (E, f, d), m.w_std), dt),
        "W2": _finish(_normal(np.random.default_rng(s_w2), (E, d, f), m.w_std), dt),
        "dy": _finish(_normal(np.random.default_rng(s_dy), (T, d), 1.0), dt),
    }
    rng_ln = np.random.default_rng(s_ln)
    out["ln1_g"] = _finish(1.0 + _normal(rng_ln, (d,), 0.02), dt)
    out["ln1_b"] = _finish(_normal(rng_ln, (d,), 0.02), dt)
    out["ln2_g"] = _finish(1.0 + _normal(rng_ln, (d,), 0.02), dt)
    out["ln2_b"] = _finish(_normal(rng_ln, (d,), 0.02), dt)
    out["Wqkv"] = _finish(_normal(np.random.default_rng(s_qkv), (3 * d, d), 0.02), dt)
    out["Wo"] = _finish(_normal(np.random.default_rng(s_o), (d, d), 0.02), dt)
    return out
