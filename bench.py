"""Benchmark: MoE layer forward + backward on one MI355X.

One step = top-k gate -> capacity-bounded dispatch -> expert FFN grouped GEMMs
-> weighted combine -> dX chain -> dW products, over one batch of seeded
synthetic input already resident in HBM.  The default workload is one GPU's
expert-parallel share (16384 tokens, d_model 2048, d_ff 8192, 8 local experts
in 8 destination slices, top-2, capacity factor 1.25, bf16), the largest
single-GPU MoE-layer workload; --config 2 and 4 select the 8192-token,
16-expert layer and the Zipf-skewed 64-expert layer.  Prints ONE JSON line.

The expert weights are held in the packed layout the GEMMs read, as a
training loop on this library keeps them: they are packed once before the
timed steps, and the dW products write their gradients in the same packed
layout (cfg.wpacked = 1), so an optimizer updates the packed copies in place.
The cost of one re-pack (moe_pack_weights) is measured separately and
reported as pack_weights_ms, with ms_per_step_with_repack for a caller that
keeps row-major weights and re-packs every step.

The timed steps are replays of one HIP graph that captures the six calls of
the step (the launches go out together, without per-kernel host gaps; graph
replays reproduce the eager step bit for bit, tests/test_gpu_graph.py); the
eager step is timed too (eager_ms_per_step).  Per-call durations come from
HIP events recorded around every C-ABI call on the stream the kernels run on,
over the eager steps.  Those steps run over the same buffers (hot caches:
the 256 MiB Infinity Cache may hold what the previous call wrote); the cold
variant reads a 512 MiB scratch buffer before every step and before every
call, outside the timed events, so each call starts from HBM
(cold_ms_per_step, cold_per_call_ms, cold_hbm_frac_per_call).  The roofline
object reports the expert-GEMM kernel with the largest time per step: its algorithmic
2 N d f flops per launch over its average launch duration, timed by HIP events
that the library records around each expert product on the kernels' own
stream during the eager steps (moe_product_timing), against the dense bf16
MFMA peak; traffic is the HBM-side bytes per launch from the committed PMC
summary for the current GEMM sources.  roofline_kernels lists every product
kernel, roofline_calls the three GEMM calls (4 N d f flops each over the
call's event time, gathers included).  The CPU
baseline is the float64 oracle on a bounded sample of the same workload.

With --workload block: one step = forward + backward of the pre-LN MoE block
(8 sequences x 2048 tokens, d_model 2048, 16 heads, 16 experts, d_ff 8192,
top-2) through moe_block_chunked with 4 batch partitions on three streams;
the line also reports forward and backward times with 1 partition and with
all work on a single stream, which isolate the pipelining and the deferred
weight gradients.

With --routing bpr the step's dispatch is the batch-prioritized one
(moe_dispatch_bpr: tokens visited by importance); either way the line reports
the other order's dispatch time on the same gate output (dispatch_*_ms).

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 2|3|4] [--workload layer|block]
                       [--routing token|bpr] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

MI355X_PEAK_BF16_TFLOPS = 2500.0   # dense bf16 MFMA
MI355X_PEAK_HBM_GBPS = 8000.0
ROOT = os.path.dirname(os.path.abspath(__file__))
#: HBM bytes per call from PMC counters (profiles/*_pmc_traffic.md), each valid for the
#: workload, call and GEMM sources it names.
PROFILES = os.path.join(ROOT, "profiles")
GEMM_SOURCES = ["paper_2404_19429_amd/csrc/gemm.hip", "paper_2404_19429_amd/csrc/lds_ops.h",
                "paper_2404_19429_amd/csrc/common.h"]


def gemm_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in GEMM_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_records():
    """Every `traffic_record:` line of the committed PMC summaries, as dicts
    (workload, call, gemm_source_hash, traffic_bytes_per_call,
    algorithmic_bytes_per_call) with the file they came from."""
    import glob
    out = []
    for path in sorted(glob.glob(os.path.join(PROFILES, "*_pmc*.md"))):
        for line in open(path).read().splitlines():
            if line.startswith("traffic_record:"):
                kv = dict(f.split("=", 1) for f in line.split(":", 1)[1].split())
                kv["file"] = path
                out.append(kv)
    return out


def measured_traffic(workload: str, call: str):
    """HBM-side bytes per call of `call` recorded in a committed PMC summary, or
    None if none was taken on this workload with the current GEMM sources."""
    h = gemm_source_hash()
    for kv in traffic_records():
        if kv.get("workload") == workload and kv.get("call") == call and kv.get("gemm_source_hash") == h:
            return float(kv["traffic_bytes_per_call"])
    return None


METRIC = "MoE layer fwd+bwd tokens/s on 1 MI355X; expert GEMM MFMA util; dispatch GB/s"
CALLS = ["gate", "dispatch", "expert_ffn_fwd", "combine", "bwd_dx", "bwd_dw"]


def _args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=3, choices=[2, 3, 4])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true", help="skip the HIP-graph replay of the layer step")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="run one plain device copy of this many MiB first (calibrates HBM byte counters)")
    ap.add_argument("--cpu-sample-tokens", type=int, default=0,
                    help="tokens of the oracle's CPU sample (0: 2^36 / (d_model d_ff) tokens, at most T: "
                         "about 10-20 s on the GPU machine's host)")
    ap.add_argument("--no-cold", action="store_true", help="skip the cold-cache steps")
    ap.add_argument("--workload", default="layer", choices=["layer", "block"])
    ap.add_argument("--pipeline-check", action="store_true",
                    help="block workload: predict the partitioned forward's time for 1, 2, 4, 8 partitions with the "
                         "library's pipeline simulator from measured stage times, and compare with the measured time")
    ap.add_argument("--block-one-stream", action="store_true",
                    help="block workload: run the timed steps with all work on one stream and skip the variants "
                         "(a kernel trace of it shows each kernel's own time, without concurrent kernels)")
    ap.add_argument("--routing", default="token", choices=["token", "bpr"],
                    help="capacity order of the layer step: token order, or batch-prioritized (importance order)")
    return ap.parse_args()


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(spec, inp, n_tokens):
    """The oracle, as it stands, on the first n_tokens tokens of the workload."""
    from dataclasses import replace
    from oracle import moe_oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    sub = {k: (v[:n_tokens] if k in ("x", "dy") else v) for k, v in inp.items()}
    s = replace(spec, T=n_tokens)
    t0 = time.perf_counter()
    fw = O.layer_forward(s, sub)
    O.layer_backward(s, sub, fw)
    dt = time.perf_counter() - t0
    return {"value": n_tokens / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle", "cpu": cpu_model(),
            "sample": f"float64 oracle layer forward+backward on the first {n_tokens} tokens of the same "
                      f"workload (capacity recomputed for {n_tokens} tokens), {dt:.1f} s wall"}


def block_cpu_baseline(spec, inp, S_sample):
    """The block oracle, as it stands, on the first S_sample tokens of sequence 0."""
    from dataclasses import replace
    from oracle import block_oracle as BO
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    sub = dict(inp)
    sub["x"], sub["dy"] = inp["x"][:S_sample], inp["dy"][:S_sample]
    s = replace(spec, B=1, S=S_sample, moe=replace(spec.moe, T=S_sample))
    t0 = time.perf_counter()
    fw = BO.block_forward(s, sub)
    BO.block_backward(s, sub, fw)
    dt = time.perf_counter() - t0
    return {"value": S_sample / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle", "cpu": cpu_model(),
            "sample": f"float64 oracle block forward+backward on the first {S_sample} tokens of sequence 0 "
                      f"(one sequence of {S_sample}; capacity recomputed), {dt:.1f} s wall"}


def block_flops(spec, kept):
    """Algorithmic MFMA flops of one block step: projections, causal attention, experts."""
    T, d, f, S, B = spec.B * spec.S, spec.d, spec.moe.f, spec.S, spec.B
    proj = 2.0 * T * d * (3 * d) + 2.0 * T * d * d                  # QKV + output projection
    attn_fwd = 2 * 2.0 * B * S * (S + 1) / 2 * d                   # QK^T and PV over the causal half
    experts = 4.0 * kept * d * f
    fwd = proj + attn_fwd + experts
    bwd = 2 * proj + 2 * attn_fwd + 2 * experts                    # dX + dW; attention dQ, dK, dV, dP
    return fwd, bwd


def main_block(a):
    import torch
    from paper_2404_19429_amd import lancet_moe as L
    from synth import BLOCK5, block_inputs

    spec = BLOCK5
    inp = block_inputs(spec)
    m = spec.moe
    T = spec.B * spec.S
    C = L.moe_capacity(T, m.E, m.k, m.cf_num, m.cf_den)
    # The expert weights are kept packed, as a training loop on this library keeps
    # them (packed once here; dW1, dW2 come back packed), like the layer step.
    cfg = L.make_block_cfg(spec.B, spec.S, spec.heads, m.f, m.E, m.k, C, m.G, m.act, m.renorm, wpacked=1)
    bf = torch.bfloat16
    w = {n: torch.from_numpy(inp[n]).cuda().to(bf).reshape(-1) for n in L.BLOCK_WEIGHTS}
    for n in ("W1", "W2"):
        packed = torch.empty_like(w[n])
        w[n + "_rowmajor"] = w[n]
        w[n] = packed
    L.moe_pack_weights(cfg.moe, w["W1_rowmajor"], w["W2_rowmajor"], w["W1"], w["W2"])
    del w["W1_rowmajor"], w["W2_rowmajor"]
    x = torch.from_numpy(inp["x"]).cuda().to(bf).reshape(-1)
    dy = torch.from_numpy(inp["dy"]).cuda().to(bf).reshape(-1)
    out, dx = torch.empty_like(x), torch.empty_like(x)
    n = spec.n_chunks
    bufs = {nc: L.alloc_block(cfg, nc) for nc in (n, 1)}
    main = torch.cuda.current_stream()
    three = [main, torch.cuda.Stream(), torch.cuda.Stream()]
    one = [main] * 3

    def run(passes, nc, streams, c=None):
        b = bufs[nc]
        L.moe_block_chunked(cfg if c is None else c, w, b, x, out, dy, dx, b, passes, nc, streams, b["ws"])

    def timed(passes, nc, streams, steps, warm, c=None):
        if passes == L.MOE_BLOCK_BWD:
            run(L.MOE_BLOCK_FWD, nc, streams, c)         # activations for the backward
        for _ in range(warm):
            run(passes, nc, streams, c)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(main)
        for _ in range(steps):
            run(passes, nc, streams, c)
        e1.record(main)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    FB = L.MOE_BLOCK_FWD | L.MOE_BLOCK_BWD
    main_streams = one if a.block_one_stream else three
    for _ in range(a.warmup):
        run(FB, n, main_streams)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(a.steps):
        run(FB, n, main_streams)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_s = wall / a.steps
    if a.block_one_stream:
        kept = int(bufs[n]["fill"].view(n, m.E)[-1].sum().item())
        fwd_fl, bwd_fl = block_flops(spec, kept)
        print(json.dumps({"metric": "MoE block fwd+bwd tokens/s on 1 MI355X (4 partitions, one stream)",
                          "value": T / step_s, "unit": "tokens/s", "ms_per_step": step_s * 1e3,
                          "steps": a.steps, "warmup": a.warmup, "step_tflop": (fwd_fl + bwd_fl) / 1e12,
                          "config": {"workload": spec.name, "streams": 1}}), flush=True)
        return
    k = max(3, a.steps // 2)
    variants = {
        "fwd_4part_3streams": timed(L.MOE_BLOCK_FWD, n, three, k, 2),
        "fwd_4part_1stream": timed(L.MOE_BLOCK_FWD, n, one, k, 2),
        "fwd_1part_3streams": timed(L.MOE_BLOCK_FWD, 1, three, k, 2),
        "bwd_3streams": timed(L.MOE_BLOCK_BWD, n, three, k, 2),
        "bwd_1stream": timed(L.MOE_BLOCK_BWD, n, one, k, 2),
    }
    kept = int(bufs[n]["fill"].view(n, m.E)[-1].sum().item())
    # Ablation analogue (whole forward + backward steps): batch partitioning with
    # the dispatch/combine stream, and the deferred weight-gradient stream, each
    # on and off.
    sx, sw = three[1], three[2]
    ablation = {
        "neither (1 partition, 1 stream)": timed(FB, 1, one, k, 2),
        "partitioning only (4 partitions, dispatch/combine stream, no weight stream)": timed(FB, n, [main, sx, main],
                                                                                               k, 2),
        "weight-gradient deferral only (1 partition, weight stream)": timed(FB, 1, [main, main, sw], k, 2),
        "both (4 partitions, 3 streams)": timed(FB, n, three, k, 2),
    }
    # The weight-gradient schedule pass on this run's own operation times
    # (one stream, MOE_BLOCK_TIMED), the all-to-alls costed as the slice to
    # one of 7 peers over one 153 GB/s xGMI link.
    run(L.MOE_BLOCK_FWD, n, one)
    run(L.MOE_BLOCK_BWD | L.MOE_BLOCK_TIMED, n, one)
    torch.cuda.synchronize()
    op_ms = L.moe_block_op_times()
    a2a_ms = kept * spec.d * 2 / 8 / 153e9 * 1e3
    dw_order, dw_assign, dw_ov = L.moe_block_dw_schedule(op_ms, a2a_ms)
    cfg_planned = L.make_block_cfg(spec.B, spec.S, spec.heads, m.f, m.E, m.k, C, m.G, m.act, m.renorm,
                                   dw_order=dw_order.tolist(), wpacked=1)
    variants["bwd_3streams_planned_dw_order"] = timed(L.MOE_BLOCK_BWD, n, three, k, 2, cfg_planned)
    dw_schedule = {"op_ms": {o: float(t) for o, t in zip(L.BLOCK_OPS, op_ms)}, "a2a_ms_model": a2a_ms,
                   "planned_order": [L.BLOCK_OPS[i] for i in dw_order],
                   "default_order": L.BLOCK_OPS[8:], "overlap_ms": dw_ov}
    fwd_fl, bwd_fl = block_flops(spec, kept)
    achieved = (fwd_fl + bwd_fl) / step_s / 1e12
    res = {
        "metric": "MoE block fwd+bwd tokens/s on 1 MI355X (batch-partitioned, 3 HIP streams)",
        "value": T / step_s,
        "unit": "tokens/s",
        "n_gpus": 1, "steps": a.steps, "warmup": a.warmup, "ms_per_step": step_s * 1e3,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded Gaussian hidden states and weights; no dataset)",
        "weights": "expert weights packed once before the timed steps; dW1/dW2 written packed (moe.wpacked=1)",
        "config": {"workload": spec.name, "B": spec.B, "S": spec.S, "d_model": spec.d, "heads": spec.heads,
                   "E": m.E, "k": m.k, "d_ff": m.f, "C": C, "n_chunks": n, "kept_rows": kept,
                   "parallelism": "single GPU (one GPU's share; all-to-all not run)"},
        "roofline": {"kernel": "whole block step (all MFMA work: projections, attention, experts)",
                     "bound": "mfma", "achieved": achieved, "peak": MI355X_PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / MI355X_PEAK_BF16_TFLOPS, "traffic": None},
        "step_tflop": (fwd_fl + bwd_fl) / 1e12,
        "variant_ms": variants,
        "pipelining_gain_fwd_ms": variants["fwd_4part_1stream"] - variants["fwd_4part_3streams"],
        "deferred_dw_gain_bwd_ms": variants["bwd_1stream"] - variants["bwd_3streams"],
        "ablation_step_ms": ablation,
        "dw_schedule": dw_schedule,
    }
    if a.pipeline_check:
        del bufs
        res["pipeline_check"] = pipeline_check(L, torch, spec, cfg, w, x, out, dy, dx, main, three, one)
    if not a.no_cpu_baseline:
        res["cpu_baseline"] = block_cpu_baseline(spec, inp, 512)
    print(json.dumps(res), flush=True)


def pipeline_check(L, torch, spec, cfg, w, x, out, dy, dx, main, three, one):
    """The block forward split into k = 1, 2, 4, 8 batch partitions: stage times
    of one partition (pre-MoE computation up to the gate; dispatch; experts;
    combine) measured at T / k tokens (the expert weights stay packed, so the
    forward's packing stage is empty), the pipelined time the library's
    simulator predicts from them (moe_pipeline_range_cost: compute stages on
    one resource, dispatch/combine on another), and the measured time of the
    partitioned forward on three streams.  On one GPU the dispatch/combine
    stream shares the compute units, which the simulator does not model."""
    m = spec.moe
    ks = [k for k in (1, 2, 4, 8) if spec.B % k == 0]
    ev = lambda: torch.cuda.Event(enable_timing=True)

    def avg_ms(fn, reps=5, warm=2):
        for _ in range(warm):
            fn()
        torch.cuda.synchronize()
        e0, e1 = ev(), ev()
        e0.record(main)
        for _ in range(reps):
            fn()
        e1.record(main)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    stage = {}
    for k in ks:
        B1 = spec.B // k
        T1 = B1 * spec.S
        C1 = L.moe_capacity(T1, m.E, m.k, m.cf_num, m.cf_den)
        c1 = L.make_block_cfg(B1, spec.S, spec.heads, m.f, m.E, m.k, C1, m.G, m.act, m.renorm, wpacked=1)
        b = L.alloc_block(c1, 1)
        n1 = T1 * spec.d
        xs, outs = x[:n1], out[:n1]
        fwd = avg_ms(lambda: L.moe_block_chunked(c1, w, b, xs, outs, None, None, b, L.MOE_BLOCK_FWD, 1, one, b["ws"]))
        mc = c1.moe
        ws_d = torch.empty(max(16, L.moe_workspace_bytes(mc, L.MOE_CALL_DISPATCH)), dtype=torch.uint8, device="cuda")
        ws_f = torch.empty(max(16, L.moe_workspace_bytes(mc, L.MOE_CALL_FFN_FWD)), dtype=torch.uint8, device="cuda")
        y = b["dm"][:n1]
        disp = avg_ms(lambda: L.moe_dispatch(mc, b["m"], b["idx"], None, b["fill"], b["slot"], b["send_buf"], ws_d))
        ffn = avg_ms(lambda: L.moe_expert_ffn_fwd(mc, b["send_buf"], None, b["fill"], w["W1"], w["W2"], b["H"],
                                                  b["A"], b["expert_out"], ws_f))
        comb = avg_ms(lambda: L.moe_combine(mc, b["expert_out"], b["idx"], b["slot"], b["w"], y))
        pack = 0.0   # the weights stay packed (moe.wpacked = 1): the forward packs nothing
        stage[k] = [pack, max(0.0, fwd - pack - disp - ffn - comb), disp, ffn, comb]
        if k == 1:
            kept_rows = int(b["fill"].sum().item())
        del b, ws_d, ws_f
        torch.cuda.empty_cache()
    # expert weight packing (once per forward, not split), then per partition:
    # computation up to the gate, dispatch, experts, combine
    kinds = [0, 0, 1, 0, 1]
    K = max(ks)
    inf = float("inf")
    times = [[stage[1][0]] + [inf] * (K - 1)]
    times += [[stage[k][j] if k in stage else inf for k in range(1, K + 1)] for j in range(1, 5)]
    join = [0.0] * K                         # partitions are contiguous slices of the batch: no split/join work
    outk = {}
    for k in ks:
        bk = L.alloc_block(cfg, k)

        def fwd_k(streams, bk=bk, k=k):
            L.moe_block_chunked(cfg, w, bk, x, out, None, None, bk, L.MOE_BLOCK_FWD, k, streams, bk["ws"])
        meas = avg_ms(lambda: fwd_k(three), reps=5)
        meas1 = avg_ms(lambda: fwd_k(one), reps=5)
        pred = times[0][0] + L.moe_pipeline_range_cost(kinds, times, join, 2, 5, k)
        outk[str(k)] = {"stage_ms": [round(v, 4) for v in stage[k]], "predicted_ms": pred,
                        "measured_3streams_ms": meas, "measured_1stream_ms": meas1,
                        "error": (pred - meas) / meas}
        del bk
        torch.cuda.empty_cache()
    total, segs = L.moe_pipeline_plan(kinds, times, join)
    # What the same plan does when dispatch and combine are real all-to-alls
    # between 8 GPUs (2 experts each): a GPU sends 7/8 of its kept rows, over 7
    # xGMI links of 153 GB/s, or over one 100 Gb/s network port.
    a2a_mb = kept_rows * spec.d * 2 * 7 / 8 / 1e6
    what_if = {}
    for net, gbps in (("xgmi_7x153GBps", 7 * 153.0), ("nic_100Gbps", 12.5)):
        tw = [row[:] for row in times]
        for j in (2, 4):
            for k in range(1, K + 1):
                if tw[j][k - 1] != inf:
                    tw[j][k - 1] = a2a_mb / k / gbps       # ms: MB / (GB/s)
        tot_w, segs_w = L.moe_pipeline_plan(kinds, tw, join)
        what_if[net] = {"a2a_ms_unsplit": a2a_mb / gbps,
                        "predicted_ms": {str(k): tw[0][0] + L.moe_pipeline_range_cost(kinds, tw, join, 2, 5, k)
                                         for k in ks},
                        "dp_plan": {"predicted_ms": tot_w, "ranges": segs_w}}
    return {"per_partitions": outk, "dp_plan": {"predicted_ms": total, "ranges": segs},
            "what_if_all_to_all": what_if,
            "stages": ["weight packing", "pre-MoE computation + gate", "dispatch", "experts", "combine"]}


def main():
    a = _args()
    if a.gpus != 1:
        print(f"bench.py measures one GPU's share of the MoE layer step; --gpus {a.gpus} is not supported "
              f"(the all-to-all between GPUs is not implemented by this library).", file=sys.stderr)
        sys.exit(2)
    if a.workload == "block":
        return main_block(a)
    import torch
    from paper_2404_19429_amd import lancet_moe as L
    from synth import layer_inputs, layer_spec

    spec = layer_spec(a.config)
    inp = layer_inputs(spec)
    C = L.moe_capacity(spec.T, spec.E, spec.k, spec.cf_num, spec.cf_den)
    cfg = L.make_cfg(spec.T, spec.d, spec.f, spec.E, spec.k, C, spec.G, spec.dtype, spec.act, spec.renorm,
                     wpacked=1)
    dt = torch.bfloat16 if spec.dtype == "bf16" else torch.float32
    dev = {n: torch.from_numpy(inp[n]).cuda().to(dt).contiguous() for n in ("x", "Wg", "W1", "W2", "dy")}
    bias = None if inp["bias"] is None else torch.from_numpy(inp["bias"]).cuda()
    b = L.alloc_layer(cfg)
    stream = torch.cuda.current_stream()

    def step(evs=None):
        def mark(i):
            if evs is not None:
                evs[i].record(stream)
        mark(0)
        L.moe_gate_topk(cfg, dev["x"], dev["Wg"], bias, b.logits, b.idx, b.w)
        mark(1)
        if a.routing == "bpr":
            L.moe_dispatch_bpr(cfg, dev["x"], b.logits, b.idx, b.fill, b.slot, b.send_buf, None, b.ws_bpr)
        else:
            L.moe_dispatch(cfg, dev["x"], b.idx, b.carry, b.fill, b.slot, b.send_buf, b.ws_dispatch)
        mark(2)
        L.moe_expert_ffn_fwd(cfg, b.send_buf, b.carry, b.fill, b.W1p, b.W2p, b.H, b.A, b.O, b.ws_ffn)
        mark(3)
        L.moe_combine(cfg, b.O, b.idx, b.slot, b.w, b.y)
        mark(4)
        L.moe_bwd_dx(cfg, dev["Wg"], b.logits, b.idx, b.w, b.slot, b.carry, b.fill, b.H, b.O, b.W1p,
                     b.W2p, dev["dy"], b.dO, b.dH, b.dXe, b.dlogits, b.dx, b.ws_dx)
        mark(5)
        L.moe_bwd_dw(cfg, dev["x"], b.dlogits, b.carry, b.fill, b.send_buf, b.A, b.dO, b.dH, b.dW1, b.dW2,
                     b.dWg, b.ws_dw)
        mark(6)

    def step_calls():
        """The step's six calls as separate callables (the cold-cache variant flushes between them)."""
        disp = ((lambda: L.moe_dispatch_bpr(cfg, dev["x"], b.logits, b.idx, b.fill, b.slot, b.send_buf, None,
                                            b.ws_bpr)) if a.routing == "bpr" else
                (lambda: L.moe_dispatch(cfg, dev["x"], b.idx, b.carry, b.fill, b.slot, b.send_buf, b.ws_dispatch)))
        return [lambda: L.moe_gate_topk(cfg, dev["x"], dev["Wg"], bias, b.logits, b.idx, b.w), disp,
                lambda: L.moe_expert_ffn_fwd(cfg, b.send_buf, b.carry, b.fill, b.W1p, b.W2p, b.H, b.A, b.O,
                                             b.ws_ffn),
                lambda: L.moe_combine(cfg, b.O, b.idx, b.slot, b.w, b.y),
                lambda: L.moe_bwd_dx(cfg, dev["Wg"], b.logits, b.idx, b.w, b.slot, b.carry, b.fill, b.H, b.O,
                                     b.W1p, b.W2p, dev["dy"], b.dO, b.dH, b.dXe, b.dlogits, b.dx, b.ws_dx),
                lambda: L.moe_bwd_dw(cfg, dev["x"], b.dlogits, b.carry, b.fill, b.send_buf, b.A, b.dO, b.dH,
                                     b.dW1, b.dW2, b.dWg, b.ws_dw)]

    def pack():
        L.moe_pack_weights(cfg, dev["W1"], dev["W2"], b.W1p, b.W2p)

    if a.copy_probe_mib > 0:   # a plain copy of known size: the counter scale for HBM bytes
        src = torch.empty(a.copy_probe_mib * (1 << 20) // 2, dtype=torch.bfloat16, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    pack()                       # once: the weights then stay packed
    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(CALLS) + 1)] for _ in range(a.steps)]
    torch.cuda.synchronize()
    L.moe_product_timing(True)   # each expert product's own duration, from events on the kernels' stream
    t0 = time.perf_counter()
    for i in range(a.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    prod_ms, prod_n = L.moe_product_times()
    L.moe_product_timing(False)
    per_call = {c: 0.0 for c in CALLS}
    for e in evs:
        for j, c in enumerate(CALLS):
            per_call[c] += e[j].elapsed_time(e[j + 1])
    per_call = {c: v / a.steps for c, v in per_call.items()}       # ms per step

    # The same step captured once in a HIP graph and replayed: the launches
    # go out as one graph, without the host's per-kernel launch gaps.
    graph_ms = None
    if not a.no_graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
        for _ in range(a.warmup):
            graph.replay()
        torch.cuda.synchronize()
        g0 = time.perf_counter()
        for _ in range(a.steps):
            graph.replay()
        torch.cuda.synchronize()
        graph_ms = (time.perf_counter() - g0) / a.steps * 1e3
    step_ms = sum(evs[i][0].elapsed_time(evs[i][len(CALLS)]) for i in range(a.steps)) / a.steps

    # Cold caches: a 512 MiB scratch read (twice the Infinity Cache) before the
    # step and before each call, outside the events, so every call reads its
    # inputs from HBM.  A read leaves clean lines behind (a write would leave
    # dirty ones, whose write-back the next kernel would pay for).
    # cold_ms_per_step times whole steps flushed only before the step;
    # cold_per_call_ms the calls flushed one by one.
    cold = None
    if not a.no_cold:
        scratch = torch.ones(128 << 20, dtype=torch.float32, device="cuda")
        sink = torch.empty(1, dtype=torch.float32, device="cuda")
        flush = lambda: torch.sum(scratch, dim=0, keepdim=True, out=sink)
        cs = max(3, a.steps // 2)
        ev = lambda: torch.cuda.Event(enable_timing=True)
        cstep = [(ev(), ev()) for _ in range(cs)]
        ccall = [[(ev(), ev()) for _ in CALLS] for _ in range(cs)]   # own start and end per call
        for i in range(cs):
            flush()
            cstep[i][0].record(stream)
            step()
            cstep[i][1].record(stream)
        for i in range(cs):
            for j, fn in enumerate(step_calls()):
                flush()
                ccall[i][j][0].record(stream)
                fn()
                ccall[i][j][1].record(stream)
        torch.cuda.synchronize()
        del scratch
        cold = {"ms_per_step": sum(e0.elapsed_time(e1) for e0, e1 in cstep) / cs,
                "per_call_ms": {c: sum(ccall[i][j][0].elapsed_time(ccall[i][j][1]) for i in range(cs)) / cs
                                for j, c in enumerate(CALLS)}}

    # One re-pack of W1, W2 (not part of the step; reported for callers that re-pack every step).
    pe = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    pe[0].record(stream)
    for _ in range(5):
        pack()
    pe[1].record(stream)
    torch.cuda.synchronize()
    pack_ms = pe[0].elapsed_time(pe[1]) / 5

    # The other capacity order's dispatch on the same gate output (not part of the step).
    alt = {}
    for name in ("token", "bpr"):
        if name == a.routing:
            continue
        de = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        de[0].record(stream)
        for _ in range(10):
            if name == "bpr":
                L.moe_dispatch_bpr(cfg, dev["x"], b.logits, b.idx, b.fill, b.slot, b.send_buf, None, b.ws_bpr)
            else:
                L.moe_dispatch(cfg, dev["x"], b.idx, b.carry, b.fill, b.slot, b.send_buf, b.ws_dispatch)
        de[1].record(stream)
        torch.cuda.synchronize()
        alt[f"dispatch_{name}_ms"] = de[0].elapsed_time(de[1]) / 10
    step()                       # leave the buffers as the step's own routing left them
    torch.cuda.synchronize()

    fill = b.fill.cpu().numpy()
    N = int(fill.sum())                                           # kept (token, expert) rows
    d, f, T = spec.d, spec.f, spec.T
    eb = 2 if spec.dtype == "bf16" else 4
    gemm_call_flop = 4.0 * N * d * f                              # each of the three GEMM calls: two products
    # Algorithmic HBM bytes per call: gate reads x and Wg, writes logits, idx, w; dispatch reads x, writes
    # the kept rows, idx + slot; combine reads the kept expert rows, idx, slot, w and writes y.
    disp_bytes = (T * d + N * d) * eb + T * spec.k * 4 * 2
    gate_bytes = (T * d + spec.E * d) * eb + T * spec.E * 4 + T * spec.k * 8
    comb_bytes = (N * d + T * d) * eb + T * spec.k * 12
    call_bytes = {"gate": gate_bytes, "dispatch": disp_bytes, "combine": comb_bytes}

    def hbm_fracs(pc):
        return {c: call_bytes[c] / (pc[c] * 1e-3) / 1e9 / MI355X_PEAK_HBM_GBPS for c in call_bytes}

    dispatch_gbps = disp_bytes / (per_call["dispatch"] * 1e-3) / 1e9
    gemm_calls = {
        "expert_ffn_fwd": "moe_expert_ffn_fwd: FWD1 H = X W1^T with (H, act(H)) epilogue + FWD2 O = act(H) W2^T "
                          "(gemm_wide_kernel, + the K-split fix-up launch when a last round is split)",
        "bwd_dx": "moe_bwd_dx: dA = dO W2 with dA * act'(H) epilogue + dXe = dH W1 (gemm_wide_kernel, + fix-up), "
                  "plus its combine-backward and dispatch-backward gathers",
        "bwd_dw": "moe_bwd_dw: ragged-K dW2 = dO^T A + dW1 = dH^T X (gemm_wide_kernel), plus the dWg reduction",
    }
    rl_calls = {}
    for c, what in gemm_calls.items():
        ach = gemm_call_flop / (per_call[c] * 1e-3) / 1e12
        rl_calls[c] = {"kernel": what, "bound": "mfma", "achieved": ach, "peak": MI355X_PEAK_BF16_TFLOPS,
                       "unit": "TFLOP/s", "frac": ach / MI355X_PEAK_BF16_TFLOPS,
                       "ms": per_call[c], "traffic": measured_traffic(spec.name, c)}
    dominant = max(gemm_calls, key=lambda c: per_call[c])
    # Per kernel: each expert product is 2 N d f flops per launch.  The two dW
    # products are launches of one kernel instantiation; the kernel with the
    # largest time per step is the roofline's.
    prod_flop = 2.0 * N * d * f
    kernels = {
        "fwd1": ("FWD1 H = X W1^T with the (H, act(H)) epilogue", ["fwd1"]),
        "fwd2": ("FWD2 O = act(H) W2^T (+ K-split fix-up)", ["fwd2"]),
        "dA": ("dA = dO W2 with the dH = dA act'(H) epilogue", ["dA"]),
        "dXe": ("dXe = dH W1 (+ K-split fix-up)", ["dXe"]),
        "dW": ("ragged-K dW2 = dO^T A and dW1 = dH^T X, two launches per step", ["dW2", "dW1"]),
    }
    pi = {p: i for i, p in enumerate(L.PRODUCTS)}
    rl_kernels = {}
    for kname, (what, prods) in kernels.items():
        n_launch = int(sum(prod_n[pi[p]] for p in prods))
        if n_launch == 0:
            continue
        avg_ms = float(sum(prod_ms[pi[p]] for p in prods)) / n_launch
        ach = prod_flop / (avg_ms * 1e-3) / 1e12
        rl_kernels[kname] = {"kernel": f"gemm_wide_kernel: {what}", "bound": "mfma", "achieved": ach,
                             "peak": MI355X_PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": ach / MI355X_PEAK_BF16_TFLOPS,
                             "launch_ms": avg_ms, "launches_per_step": n_launch / a.steps,
                             "traffic": measured_traffic(spec.name, "kernel:" + kname)}
    dom_kernel = max(rl_kernels, key=lambda k: rl_kernels[k]["launch_ms"] * rl_kernels[k]["launches_per_step"])
    eager_ms = wall / a.steps * 1e3
    working_set = sum(t.numel() * t.element_size() for t in vars(b).values() if isinstance(t, torch.Tensor))
    working_set += sum(t.numel() * t.element_size() for t in dev.values())
    step_ms_timed = graph_ms if graph_ms is not None else eager_ms
    tokens_per_s = T / (step_ms_timed * 1e-3)
    all_gemm_ms = sum(per_call[c] for c in gemm_calls)

    out = {
        "metric": METRIC,
        "value": tokens_per_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": step_ms_timed,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec.dtype,
        "data": "synthetic (seeded Gaussian hidden states and weights; no dataset)",
        "cache": f"timed steps repeat over the same buffers (hot: the layer's buffers total "
                 f"{working_set / 2**30:.2f} GiB, above the 256 MiB Infinity Cache, but a call may find what "
                 f"the previous call wrote there); 'cold' reads 512 MiB of scratch first",
        "config": {"workload": spec.name, "T": T, "d_model": d, "d_ff": f, "E": spec.E, "k": spec.k,
                   "C": C, "G": spec.G, "capacity_factor": f"{spec.cf_num}/{spec.cf_den}", "act": spec.act,
                   "routing": a.routing,
                   "kept_rows": N, "parallelism": "single GPU (one GPU's share; all-to-all not run)"},
        "roofline": {k: v for k, v in rl_kernels[dom_kernel].items() if k not in ("launch_ms", "launches_per_step")},
        "roofline_kernel": dom_kernel,
        "roofline_kernels": rl_kernels,
        "roofline_calls": rl_calls,
        "expert_gemm_mfma_frac": 3 * gemm_call_flop / (all_gemm_ms * 1e-3) / 1e12 / MI355X_PEAK_BF16_TFLOPS,
        "dispatch_GBps": dispatch_gbps,
        "dispatch_hbm_frac": dispatch_gbps / MI355X_PEAK_HBM_GBPS,
        "hbm_frac_per_call": hbm_fracs(per_call),
        "per_call_ms": per_call,
        "step_mode": "hip_graph_replay" if graph_ms is not None else "eager",
        "eager_ms_per_step": eager_ms,
        "event_ms_per_step": step_ms,
        "weights": "packed once before the timed steps; dW1/dW2 written packed (wpacked=1)",
        "pack_weights_ms": pack_ms,
        **alt,
        "ms_per_step_with_repack": step_ms_timed + pack_ms,
    }
    if cold is not None:
        out["cold_ms_per_step"] = cold["ms_per_step"]
        out["cold_per_call_ms"] = cold["per_call_ms"]
        out["cold_hbm_frac_per_call"] = hbm_fracs(cold["per_call_ms"])
    if not a.no_cpu_baseline:
        n_cpu = a.cpu_sample_tokens or min(T, max(256, int(2 ** 36 // (d * f)) // 256 * 256))
        out["cpu_baseline"] = cpu_baseline(spec, inp, n_cpu)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
