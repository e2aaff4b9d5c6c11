// Orchestration of the partitioned pre-LN MoE block on three HIP streams.
//
// Forward (Sec. 2.3 "Challenge 1", Fig. "part_all"; Sec. 5.3): the batch is
// cut into n partitions of whole sequences.  Following the stage-ordered
// pipeline schedule, the compute stream runs the pre-MoE stage of every
// partition in index order (LN1, QKV projection, attention, output projection
// + residual, LN2, gate), then the expert stage of every partition; the
// data-movement stream runs partition i's dispatch once its gate is done and
// its combine once its experts are done.  Partition i's dispatch starts from
// the capacity partition i-1 left (fill[i-1]) and its experts work on rows
// [fill[i-1], fill[i]) of the shared [E][C][*] buffers, so partitions touch
// disjoint rows; the expert products take every K sum whole and in order
// (moe.ksplit = 0), so the result equals the unpartitioned block bit for bit.
//
// Backward (unpartitioned): the activation-gradient chain runs on the compute
// stream; each weight gradient goes to the weight stream as soon as the
// tensors it reads exist (Sec. 2.3 "Opportunity 1"; Sec. 4).
//
// Cross-stream order uses events from a per-thread, per-device pool, recorded
// before any wait on them is enqueued.  No host synchronisation.
#include <vector>

#include "internal.h"

namespace lmoe {

namespace {

struct EventPool {
  int dev = -1;
  std::vector<hipEvent_t> ev;
  size_t next = 0;
};
thread_local EventPool g_events;

// Event number i of this call (created on first use, reused by later calls on this thread).
hipError_t event(hipEvent_t* out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (g_events.dev != dev) {  // a different device: events belong to the device they were made on
    g_events.ev.clear();      // (the old ones are leaked rather than destroyed on the wrong device)
    g_events.dev = dev;
  }
  if (g_events.next == g_events.ev.size()) {
    hipEvent_t ev;
    e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
    if (e != hipSuccess) return e;
    g_events.ev.push_back(ev);
  }
  *out = g_events.ev[g_events.next++];
  return hipSuccess;
}

// b waits for everything enqueued on a so far.
hipError_t order(hipStream_t a, hipStream_t b) {
  if (a == b) return hipSuccess;
  hipEvent_t ev;
  hipError_t e = event(&ev);
  if (e != hipSuccess) return e;
  e = hipEventRecord(ev, a);
  if (e != hipSuccess) return e;
  return hipStreamWaitEvent(b, ev, 0);
}

#define HIP_TRY(expr)                      \
  do {                                     \
    const hipError_t _e = (expr);          \
    if (_e != hipSuccess) return _e;       \
  } while (0)

size_t align256(size_t n) { return (n + 255) / 256 * 256; }

struct WsLayout {
  size_t disp, dw, ln2, ln1, sk, total;
};

WsLayout ws_layout(const moe_block_cfg& c, int n) {
  const int64_t T = c.moe.T;
  const int d = c.moe.d_model;
  moe_cfg part = c.moe;
  part.T = T / n;
  WsLayout L;
  size_t off = 0;
  L.disp = off; off += align256(dispatch_ws_bytes(part));
  L.dw = off;   off += align256(bwd_dw_ws_bytes(c.moe));
  L.ln2 = off;  off += align256((size_t)ln_bwd_blocks(T) * 2 * d * sizeof(float));
  L.ln1 = off;  off += align256((size_t)ln_bwd_blocks(T) * 2 * d * sizeof(float));
  L.sk = off;   off += align256(expert_sk_ws_bytes(c.moe));   // expert products on the compute stream
  L.total = off;
  return L;
}

}  // namespace

size_t block_ws_bytes(const moe_block_cfg& c, int n_chunks) { return ws_layout(c, n_chunks).total; }

hipError_t run_block(const moe_block_cfg& c, const moe_block_weights& W, const moe_block_grads* G, const void* x,
                     void* out, const void* dy, void* dx, const moe_block_acts& A, int passes, int n,
                     const hipStream_t st[3], void* ws) {
  g_events.next = 0;
  const hipStream_t Sc = st[0], Sx = st[1], Sw = st[2];
  moe_cfg mc = c.moe;
  mc.ksplit = 0;   // one in-order K sum per output element: results independent of the partitioning
  const int64_t T = mc.T;
  const int d = mc.d_model, E = mc.E, k = mc.k, H = c.heads, S = c.S;
  const int64_t d3 = 3 * (int64_t)d;
  const int Sp = attn_stat_stride(S);
  const WsLayout L = ws_layout(c, n);
  char* wsb = (char*)ws;
  auto bf = [](const void* p, int64_t off) { return (const void*)((const uint16_t*)p + off); };
  auto bfm = [](void* p, int64_t off) { return (void*)((uint16_t*)p + off); };

  if (passes & MOE_BLOCK_FWD) {
    const int nseq = c.B / n;
    const int64_t Tc = (int64_t)nseq * S;
    moe_cfg pc = mc;
    pc.T = Tc;
    HIP_TRY(order(Sc, Sx));  // the data-movement stream starts after the caller's earlier work
    launch_pack_weights(mc, W.W1, W.W2, A.W1p, A.W2p, Sc);  // expert weights as the GEMMs read them
    std::vector<hipEvent_t> ev_disp(n);
    for (int i = 0; i < n; ++i) {  // pre-MoE stage, partitions in order
      const int64_t t0 = Tc * i;
      launch_ln_fwd(bf(x, t0 * d), W.ln1_g, W.ln1_b, bfm(A.a, t0 * d), A.ln1_mean + t0, A.ln1_rstd + t0, Tc, d, Sc);
      launch_dense(Tc, (int)d3, d, bf(A.a, t0 * d), d, W.Wqkv, d, true, bfm(A.qkv, t0 * d3), d3, nullptr, Sc);
      launch_attn_fwd(bf(A.qkv, t0 * d3), bfm(A.attn, t0 * d), A.lse + (int64_t)i * nseq * H * Sp, nseq, S, H, Sc);
      launch_dense(Tc, d, d, bf(A.attn, t0 * d), d, W.Wo, d, true, bfm(A.h, t0 * d), d, bf(x, t0 * d), Sc);
      launch_ln_fwd(bf(A.h, t0 * d), W.ln2_g, W.ln2_b, bfm(A.m, t0 * d), A.ln2_mean + t0, A.ln2_rstd + t0, Tc, d, Sc);
      launch_gate(pc, bf(A.m, t0 * d), W.Wg, nullptr, A.logits + t0 * E, A.idx + t0 * k, A.w + t0 * k, Sc);
      HIP_TRY(hipGetLastError());
      HIP_TRY(order(Sc, Sx));
      launch_dispatch(pc, bf(A.m, t0 * d), A.idx + t0 * k, i == 0 ? nullptr : A.fill + (int64_t)(i - 1) * E,
                      A.fill + (int64_t)i * E, A.slot + t0 * k, A.send_buf, wsb + L.disp, Sx);
      HIP_TRY(hipGetLastError());
      HIP_TRY(event(&ev_disp[i]));
      HIP_TRY(hipEventRecord(ev_disp[i], Sx));
    }
    for (int i = 0; i < n; ++i) {  // expert stage, partitions in order; each combine follows on Sx
      const int64_t t0 = Tc * i;
      HIP_TRY(hipStreamWaitEvent(Sc, ev_disp[i], 0));
      const int32_t* rb = i == 0 ? nullptr : A.fill + (int64_t)(i - 1) * E;
      launch_expert_fwd(mc, A.send_buf, rb, A.fill + (int64_t)i * E, A.W1p, A.W2p, A.H, A.A, A.expert_out, wsb + L.sk, Sc);
      HIP_TRY(hipGetLastError());
      HIP_TRY(order(Sc, Sx));
      launch_combine(pc, A.expert_out, A.idx + t0 * k, A.slot + t0 * k, A.w + t0 * k, bfm(out, t0 * d), Sx,
                     bf(A.h, t0 * d));
      HIP_TRY(hipGetLastError());
    }
    HIP_TRY(order(Sx, Sc));
  }

  if (passes & MOE_BLOCK_BWD) {
    const int32_t* fill_end = A.fill + (int64_t)(n - 1) * E;
    HIP_TRY(order(Sc, Sw));  // the weight stream starts after the caller's earlier work
    // MoE layer: combine/gate backward, expert dX, dispatch backward -> dm
    launch_combine_bwd(mc, A.logits, A.idx, A.w, A.slot, A.expert_out, dy, A.dO, A.dlogits, Sc);
    launch_expert_bwd_dx(mc, A.dO, nullptr, fill_end, A.H, A.W1p, A.W2p, A.dH, A.dXe, wsb + L.sk, Sc);
    launch_dispatch_bwd(mc, W.Wg, A.dlogits, A.idx, A.slot, A.dXe, A.dm, Sc);
    HIP_TRY(hipGetLastError());
    HIP_TRY(order(Sc, Sw));
    launch_expert_bwd_dw(mc, A.send_buf, A.A, A.dO, A.dH, nullptr, fill_end, G->dW1, G->dW2, Sw);
    launch_dwg(mc, A.m, A.dlogits, G->dWg, wsb + L.dw, Sw);
    // LN2 backward with the residual: dh = dy + LN2'(dm)
    launch_ln_bwd(A.dm, A.h, A.ln2_mean, A.ln2_rstd, W.ln2_g, dy, A.dh, (float*)(wsb + L.ln2), T, d, Sc);
    HIP_TRY(hipGetLastError());
    HIP_TRY(order(Sc, Sw));
    launch_ln_gain_reduce((const float*)(wsb + L.ln2), T, d, G->dln2_g, G->dln2_b, Sw);
    launch_dense_wgrad(d, d, T, A.dh, d, A.attn, d, G->dWo, d, Sw);  // dWo = dh^T o
    // attention backward
    launch_dense(T, d, d, A.dh, d, W.Wo, d, false, A.dattn, d, nullptr, Sc);  // do = dh Wo
    launch_attn_bwd(A.qkv, A.attn, A.dattn, A.lse, A.delta, A.dqkv, c.B, S, H, Sc);
    HIP_TRY(hipGetLastError());
    HIP_TRY(order(Sc, Sw));
    launch_dense_wgrad((int)d3, d, T, A.dqkv, d3, A.a, d, G->dWqkv, d, Sw);  // dWqkv = dqkv^T a
    // QKV projection and LN1 backward with the residual: dx = dh + LN1'(dqkv Wqkv)
    launch_dense(T, d, (int)d3, A.dqkv, d3, W.Wqkv, d, false, A.da, d, nullptr, Sc);
    launch_ln_bwd(A.da, x, A.ln1_mean, A.ln1_rstd, W.ln1_g, A.dh, dx, (float*)(wsb + L.ln1), T, d, Sc);
    HIP_TRY(hipGetLastError());
    HIP_TRY(order(Sc, Sw));
    launch_ln_gain_reduce((const float*)(wsb + L.ln1), T, d, G->dln1_g, G->dln1_b, Sw);
    HIP_TRY(hipGetLastError());
    HIP_TRY(order(Sw, Sc));
  }
  return hipGetLastError();
}

}  // namespace lmoe
