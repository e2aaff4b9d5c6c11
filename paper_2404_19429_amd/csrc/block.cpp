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

#define HIP_TRY(expr)                      \
  do {                                     \
    const hipError_t _e = (expr);          \
    if (_e != hipSuccess) return _e;       \
  } while (0)

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

size_t align256(size_t n) { return (n + 255) / 256 * 256; }

// Timing events of this thread's last timed backward: start and end of each
// operation.
struct TimingEvents {
  int dev = -1;
  hipEvent_t ev[2 * MOE_BOP_COUNT] = {};
  bool valid = false;
};
thread_local TimingEvents g_timing;

hipError_t timing_begin() {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (g_timing.dev != dev) {   // events belong to the device they were made on
    for (auto& e : g_timing.ev) {
      e = nullptr;
      HIP_TRY(hipEventCreate(&e));
    }
    g_timing.dev = dev;
  }
  g_timing.valid = false;
  return hipSuccess;
}

// The chain operation whose output a weight-gradient group reads.
int dw_producer(int op) {
  switch (op) {
    case MOE_BOP_DW_EXPERT: return MOE_BOP_EXPERT_DX;
    case MOE_BOP_DWG: return MOE_BOP_COMBINE_BWD;
    case MOE_BOP_DLN2:
    case MOE_BOP_DWO: return MOE_BOP_LN2_BWD;
    case MOE_BOP_DWQKV: return MOE_BOP_ATTN_BWD;
    default: return MOE_BOP_LN1_BWD;
  }
}

struct WsLayout {
  size_t disp, dw, ln2, ln1, sk, wqkv, wo, act, wgp, total;
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
  // Blocked copies for the dense products on the wide kernel: Wqkv, Wo, and
  // one activation operand at a time (used in turn on the compute stream).
  L.wqkv = off; off += align256((size_t)3 * d * d * 2);
  L.wo = off;   off += align256((size_t)d * d * 2);
  L.act = off;  off += align256((size_t)pad16(T) * 3 * d * 2);
  // Float partials of the dense weight gradients (dWo, then dWqkv, on the
  // weight stream).
  L.wgp = off;  off += align256(wgrad_ws_bytes(3 * d, d));
  L.total = off;
  return L;
}

}  // namespace

// The weight-gradient launch order of cfg (the default when dw_order[0] < 0).
void dw_launch_order(const moe_block_cfg& c, int32_t out[6]) {
  for (int q = 0; q < 6; ++q) out[q] = c.dw_order[0] < 0 ? MOE_BOP_DW_EXPERT + q : c.dw_order[q];
}

hipError_t block_op_times(double* ms) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (!g_timing.valid || g_timing.dev != dev) return hipErrorNotReady;
  for (int op = 0; op < MOE_BOP_COUNT; ++op) {
    HIP_TRY(hipEventSynchronize(g_timing.ev[2 * op + 1]));
    float t = 0.f;
    HIP_TRY(hipEventElapsedTime(&t, g_timing.ev[2 * op], g_timing.ev[2 * op + 1]));
    ms[op] = t;
  }
  return hipSuccess;
}

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
  // moe.wpacked = 1: the caller's W1, W2 are already the packed copies (and
  // dW1, dW2 are written packed); else the forward packs them into acts.
  const void* W1p = mc.wpacked ? W.W1 : A.W1p;
  const void* W2p = mc.wpacked ? W.W2 : A.W2p;
  void* Wqkv_b = wsb + L.wqkv;   // blocked copies for the wide dense products
  void* Wo_b = wsb + L.wo;
  void* act_b = wsb + L.act;

  if (passes & MOE_BLOCK_FWD) {
    const int nseq = c.B / n;
    const int64_t Tc = (int64_t)nseq * S;
    moe_cfg pc = mc;
    pc.T = Tc;
    HIP_TRY(order(Sc, Sx));  // the data-movement stream starts after the caller's earlier work
    if (!mc.wpacked) launch_pack_weights(mc, W.W1, W.W2, A.W1p, A.W2p, Sc);  // expert weights as the GEMMs read them
    launch_pack_rows(W.Wqkv, Wqkv_b, d3, d, Sc);
    launch_pack_rows(W.Wo, Wo_b, d, d, Sc);
    std::vector<hipEvent_t> ev_disp(n);
    for (int i = 0; i < n; ++i) {  // pre-MoE stage, partitions in order
      const int64_t t0 = Tc * i;
      // LN1 and attention write their outputs' blocked copies (act_b) for the
      // projections that follow; each copy is used before the next is written.
      launch_ln_fwd(bf(x, t0 * d), W.ln1_g, W.ln1_b, bfm(A.a, t0 * d), A.ln1_mean + t0, A.ln1_rstd + t0, Tc, d, Sc,
                    act_b);
      launch_dense_wide(Tc, (int)d3, d, act_b, Wqkv_b, true, bfm(A.qkv, t0 * d3), d3, nullptr, Sc);
      launch_attn_fwd(bf(A.qkv, t0 * d3), bfm(A.attn, t0 * d), A.lse + (int64_t)i * nseq * H * Sp, nseq, S, H, Sc,
                      act_b);
      launch_dense_wide(Tc, d, d, act_b, Wo_b, true, bfm(A.h, t0 * d), d, bf(x, t0 * d), Sc);
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
      launch_expert_fwd(mc, A.send_buf, rb, A.fill + (int64_t)i * E, W1p, W2p, A.H, A.A, A.expert_out, wsb + L.sk, Sc);
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
    const bool timed = (passes & MOE_BLOCK_TIMED) != 0;
    if (timed) HIP_TRY(timing_begin());
    auto mark = [&](int op, int which, hipStream_t s) -> hipError_t {
      return timed ? hipEventRecord(g_timing.ev[2 * op + which], s) : hipSuccess;
    };
    HIP_TRY(order(Sc, Sw));  // the weight stream starts after the caller's earlier work
    if (!(passes & MOE_BLOCK_FWD)) {   // a forward in the same call has packed them already
      launch_pack_rows(W.Wqkv, Wqkv_b, d3, d, Sc);
      launch_pack_rows(W.Wo, Wo_b, d, d, Sc);
    }
    // The activation-gradient chain on Sc, recording after each operation
    // whose output a weight gradient reads the event that gradient waits for.
    hipEvent_t after[MOE_BOP_COUNT] = {};
    auto produced = [&](int op) -> hipError_t {
      HIP_TRY(event(&after[op]));
      return hipEventRecord(after[op], Sc);
    };
    // MoE layer: combine/gate backward, expert dX, dispatch backward -> dm
    HIP_TRY(mark(MOE_BOP_COMBINE_BWD, 0, Sc));
    launch_combine_bwd(mc, A.logits, A.idx, A.w, A.slot, A.expert_out, dy, A.dO, A.dlogits, Sc);
    HIP_TRY(mark(MOE_BOP_COMBINE_BWD, 1, Sc));
    HIP_TRY(produced(MOE_BOP_COMBINE_BWD));
    HIP_TRY(mark(MOE_BOP_EXPERT_DX, 0, Sc));
    launch_expert_bwd_dx(mc, A.dO, nullptr, fill_end, A.H, W1p, W2p, A.dH, A.dXe, wsb + L.sk, Sc);
    HIP_TRY(mark(MOE_BOP_EXPERT_DX, 1, Sc));
    HIP_TRY(produced(MOE_BOP_EXPERT_DX));
    HIP_TRY(mark(MOE_BOP_DISPATCH_BWD, 0, Sc));
    launch_dispatch_bwd(mc, W.Wg, A.dlogits, A.idx, A.slot, A.dXe, A.dm, Sc);
    HIP_TRY(mark(MOE_BOP_DISPATCH_BWD, 1, Sc));
    // LN2 backward with the residual: dh = dy + LN2'(dm)
    HIP_TRY(mark(MOE_BOP_LN2_BWD, 0, Sc));
    launch_ln_bwd(A.dm, A.h, A.ln2_mean, A.ln2_rstd, W.ln2_g, dy, A.dh, (float*)(wsb + L.ln2), T, d, Sc,
                  act_b);   // dh, and its blocked copy for d(attn out) = dh Wo
    HIP_TRY(mark(MOE_BOP_LN2_BWD, 1, Sc));
    HIP_TRY(produced(MOE_BOP_LN2_BWD));
    // attention backward
    HIP_TRY(mark(MOE_BOP_DATTN, 0, Sc));
    launch_dense_wide(T, d, d, act_b, Wo_b, false, A.dattn, d, nullptr, Sc);  // do = dh Wo
    HIP_TRY(mark(MOE_BOP_DATTN, 1, Sc));
    HIP_TRY(mark(MOE_BOP_ATTN_BWD, 0, Sc));
    launch_attn_bwd(A.qkv, A.attn, A.dattn, A.lse, A.delta, A.dqkv, c.B, S, H, Sc, act_b);  // + blocked dqkv
    HIP_TRY(mark(MOE_BOP_ATTN_BWD, 1, Sc));
    HIP_TRY(produced(MOE_BOP_ATTN_BWD));
    // QKV projection and LN1 backward with the residual: dx = dh + LN1'(dqkv Wqkv)
    HIP_TRY(mark(MOE_BOP_DA, 0, Sc));
    launch_dense_wide(T, d, (int)d3, act_b, Wqkv_b, false, A.da, d, nullptr, Sc);
    HIP_TRY(mark(MOE_BOP_DA, 1, Sc));
    HIP_TRY(mark(MOE_BOP_LN1_BWD, 0, Sc));
    launch_ln_bwd(A.da, x, A.ln1_mean, A.ln1_rstd, W.ln1_g, A.dh, dx, (float*)(wsb + L.ln1), T, d, Sc);
    HIP_TRY(mark(MOE_BOP_LN1_BWD, 1, Sc));
    HIP_TRY(produced(MOE_BOP_LN1_BWD));
    HIP_TRY(hipGetLastError());
    // The weight gradients on Sw in the configured order, each after the
    // chain operation whose output it reads (every event above is recorded
    // before any wait on it is enqueued).
    int32_t dwo[6];
    dw_launch_order(c, dwo);
    for (int q = 0; q < 6; ++q) {
      const int op = dwo[q];
      HIP_TRY(hipStreamWaitEvent(Sw, after[dw_producer(op)], 0));
      HIP_TRY(mark(op, 0, Sw));
      switch (op) {
        case MOE_BOP_DW_EXPERT:
          launch_expert_bwd_dw(mc, A.send_buf, A.A, A.dO, A.dH, nullptr, fill_end, G->dW1, G->dW2, Sw);
          break;
        case MOE_BOP_DWG: launch_dwg(mc, A.m, A.dlogits, G->dWg, wsb + L.dw, Sw); break;
        case MOE_BOP_DLN2:
          launch_ln_gain_reduce((float*)(wsb + L.ln2), T, d, G->dln2_g, G->dln2_b, Sw);
          break;
        case MOE_BOP_DWO: launch_dense_wgrad(d, d, T, A.dh, A.attn, G->dWo, wsb + L.wgp, Sw); break;  // dh^T o
        case MOE_BOP_DWQKV:
          launch_dense_wgrad((int)d3, d, T, A.dqkv, A.a, G->dWqkv, wsb + L.wgp, Sw);  // dWqkv = dqkv^T a
          break;
        default:
          launch_ln_gain_reduce((float*)(wsb + L.ln1), T, d, G->dln1_g, G->dln1_b, Sw);
          break;
      }
      HIP_TRY(mark(op, 1, Sw));
    }
    HIP_TRY(hipGetLastError());
    HIP_TRY(order(Sw, Sc));
    if (timed) g_timing.valid = true;
  }
  return hipGetLastError();
}

}  // namespace lmoe
