// C ABI of the MoE-layer library: host-side validation, then kernel launches.
// Validation needs no GPU, so every error path can be exercised on a host
// without one; only a call that passes validation touches the HIP runtime.
#include <cstddef>
#include <cstdio>
#include <cstdarg>
#include <cstring>
#include <string>

#include "internal.h"

// The Python binding and other callers lay these structs out by hand.
static_assert(sizeof(moe_cfg) == 56 && offsetof(moe_cfg, ksplit) == 48, "moe_cfg layout");
static_assert(sizeof(moe_block_cfg) == 96 && offsetof(moe_block_cfg, moe) == 16 &&
                  offsetof(moe_block_cfg, dw_order) == 72,
              "moe_block_cfg layout");

namespace {

thread_local std::string g_err;

moe_status fail(moe_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

moe_status ok() {
  g_err.clear();
  return MOE_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

#define REQUIRE_PTR(p)                                                            \
  do {                                                                            \
    if ((p) == nullptr) return fail(MOE_EINVAL, "%s: " #p " is NULL", fn);        \
    if (!aligned16(p)) return fail(MOE_EALIGN, "%s: " #p " is not 16-byte aligned", fn); \
  } while (0)
// Token-sized arrays (T rows) may be NULL when T == 0.
#define REQUIRE_TPTR(p)                                                           \
  do {                                                                            \
    if (cfg->T > 0) REQUIRE_PTR(p); else OPTIONAL_PTR(p);                         \
  } while (0)
#define OPTIONAL_PTR(p)                                                           \
  do {                                                                            \
    if ((p) != nullptr && !aligned16(p))                                          \
      return fail(MOE_EALIGN, "%s: " #p " is not 16-byte aligned", fn);           \
  } while (0)

moe_status check_cfg(const moe_cfg* c, const char* fn, bool need_gemm_shape) {
  if (!c) return fail(MOE_EINVAL, "%s: cfg is NULL", fn);
  if (c->dtype != MOE_F32 && c->dtype != MOE_BF16) return fail(MOE_EDTYPE, "%s: unknown dtype %d", fn, c->dtype);
  if (c->act < MOE_ACT_IDENTITY || c->act > MOE_ACT_GELU_ERF) return fail(MOE_EINVAL, "%s: unknown act %d", fn, c->act);
  if (c->renorm != 0 && c->renorm != 1) return fail(MOE_EINVAL, "%s: renorm must be 0 or 1", fn);
  if (c->wpacked != 0 && c->wpacked != 1) return fail(MOE_EINVAL, "%s: wpacked must be 0 or 1", fn);
  if (c->ksplit != 0 && c->ksplit != 1) return fail(MOE_EINVAL, "%s: ksplit must be 0 or 1", fn);
  if (c->T < 0) return fail(MOE_EINVAL, "%s: T < 0", fn);
  if (c->T > (int64_t)1 << 31) return fail(MOE_ESHAPE, "%s: T > 2^31 unsupported", fn);
  if (c->E < 1 || c->E > lmoe::kMaxE) return fail(MOE_ESHAPE, "%s: E=%d outside 1..%d", fn, c->E, lmoe::kMaxE);
  if (c->k < 1 || c->k > c->E || c->k > lmoe::kMaxK)
    return fail(MOE_EINVAL, "%s: k=%d outside 1..min(E, %d)", fn, c->k, lmoe::kMaxK);
  if (c->C < 1) return fail(MOE_EINVAL, "%s: C=%d < 1", fn, c->C);
  if (c->G < 1 || c->E % c->G != 0) return fail(MOE_EINVAL, "%s: G=%d does not divide E=%d", fn, c->G, c->E);
  if (c->d_model < 8 || c->d_model % 8 != 0) return fail(MOE_ESHAPE, "%s: d_model=%d not a positive multiple of 8", fn, c->d_model);
  if (c->d_ff < 8 || c->d_ff % 8 != 0) return fail(MOE_ESHAPE, "%s: d_ff=%d not a positive multiple of 8", fn, c->d_ff);
  if ((int64_t)c->C * c->E * (int64_t)(c->d_model > c->d_ff ? c->d_model : c->d_ff) > ((int64_t)1 << 40))
    return fail(MOE_ESHAPE, "%s: E*C*max(d, f) too large", fn);
  if (need_gemm_shape && c->dtype == MOE_BF16 && (c->d_model % 64 != 0 || c->d_ff % 64 != 0))
    return fail(MOE_ESHAPE, "%s: bf16 expert GEMMs need d_model and d_ff multiples of 64", fn);
  // The bf16 expert GEMMs address one expert's operand with 32-bit byte offsets.
  const int64_t xmax = c->d_model > c->d_ff ? c->d_model : c->d_ff;
  if (need_gemm_shape && c->dtype == MOE_BF16 &&
      (((int64_t)c->C + 15) * xmax * 2 >= ((int64_t)1 << 31) || (int64_t)c->d_model * c->d_ff * 2 >= ((int64_t)1 << 31)))
    return fail(MOE_ESHAPE, "%s: one expert's bf16 operand must stay under 2 GiB", fn);
  return MOE_OK;
}

// One gfx950 check per device, then cached.
moe_status check_device(const char* fn) {
  static thread_local int checked_dev = -1;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return fail(MOE_EDEVICE, "%s: no HIP device", fn);
  if (dev == checked_dev) return MOE_OK;
  hipDeviceProp_t prop;
  if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return fail(MOE_EDEVICE, "%s: cannot query device %d", fn, dev);
  if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
    return fail(MOE_EDEVICE, "%s: device %d is %s, this library is built for gfx950", fn, dev, prop.gcnArchName);
  checked_dev = dev;
  return MOE_OK;
}

moe_status check_launch(const char* fn) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(MOE_ELAUNCH, "%s: %s", fn, hipGetErrorString(e));
  return ok();
}

#define CHECK(expr)                        \
  do {                                     \
    const moe_status _st = (expr);         \
    if (_st != MOE_OK) return _st;         \
  } while (0)

}  // namespace

extern "C" {

int32_t moe_capacity(int64_t T, int32_t E, int32_t k, int32_t cf_num, int32_t cf_den) {
  if (T < 0 || E < 1 || k < 1 || cf_num < 1 || cf_den < 1) return -1;
  if (T == 0) return 0;
  const __int128 num = (__int128)k * T * cf_num;
  const __int128 den = (__int128)E * cf_den;
  const __int128 c = (num + den - 1) / den;
  if (c > INT32_MAX) return -1;
  return (int32_t)c;
}

size_t moe_workspace_bytes(const moe_cfg* cfg, int32_t call) {
  const char* fn = "moe_workspace_bytes";
  if (check_cfg(cfg, fn, false) != MOE_OK) return 0;
  switch (call) {
    case MOE_CALL_DISPATCH: return lmoe::dispatch_ws_bytes(*cfg);
    case MOE_CALL_BWD_DX: return lmoe::bwd_dx_ws_bytes(*cfg);
    case MOE_CALL_BWD_DW: return lmoe::bwd_dw_ws_bytes(*cfg);
    case MOE_CALL_FFN_FWD: return lmoe::expert_sk_ws_bytes(*cfg);
    case MOE_CALL_DISPATCH_BPR: return lmoe::dispatch_bpr_ws_bytes(*cfg);
    default: fail(MOE_EINVAL, "%s: unknown call %d", fn, call); return 0;
  }
}

const char* moe_last_error(void) { return g_err.c_str(); }

moe_status moe_gate_topk(const moe_cfg* cfg, const void* x, const void* Wg, const float* bias, float* logits,
                         int32_t* idx, float* w, moe_stream_t stream) {
  const char* fn = "moe_gate_topk";
  CHECK(check_cfg(cfg, fn, false));
  REQUIRE_TPTR(x); REQUIRE_PTR(Wg); OPTIONAL_PTR(bias);
  REQUIRE_TPTR(logits); REQUIRE_TPTR(idx); REQUIRE_TPTR(w);
  CHECK(check_device(fn));
  lmoe::launch_gate(*cfg, x, Wg, bias, logits, idx, w, (hipStream_t)stream);
  return check_launch(fn);
}

moe_status moe_dispatch(const moe_cfg* cfg, const void* x, const int32_t* idx, const int32_t* carry, int32_t* fill,
                        int32_t* slot, void* send_buf, void* ws, size_t ws_bytes, moe_stream_t stream) {
  const char* fn = "moe_dispatch";
  CHECK(check_cfg(cfg, fn, false));
  REQUIRE_TPTR(x); REQUIRE_TPTR(idx); OPTIONAL_PTR(carry); REQUIRE_PTR(fill);
  REQUIRE_TPTR(slot); REQUIRE_PTR(send_buf);
  if (carry != nullptr && (const void*)carry == (const void*)fill)
    return fail(MOE_EINVAL, "%s: carry and fill may not alias", fn);
  const size_t need = lmoe::dispatch_ws_bytes(*cfg);
  if (need > 0) {
    if (ws == nullptr || ws_bytes < need)
      return fail(MOE_EWORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, need, ws ? ws_bytes : 0);
    REQUIRE_PTR(ws);
  }
  CHECK(check_device(fn));
  lmoe::launch_dispatch(*cfg, x, idx, carry, fill, slot, send_buf, ws, (hipStream_t)stream);
  return check_launch(fn);
}

moe_status moe_dispatch_noalloc(const moe_cfg* cfg, const void* x, const int32_t* idx, const int32_t* carry,
                                int32_t* fill, int32_t* slot, void* send_buf, moe_stream_t stream) {
  const char* fn = "moe_dispatch_noalloc";
  CHECK(check_cfg(cfg, fn, false));
  REQUIRE_TPTR(x); REQUIRE_TPTR(idx); OPTIONAL_PTR(carry); REQUIRE_PTR(fill);
  REQUIRE_TPTR(slot); REQUIRE_PTR(send_buf);
  if (carry != nullptr && (const void*)carry == (const void*)fill)
    return fail(MOE_EINVAL, "%s: carry and fill may not alias", fn);
  const size_t need = lmoe::dispatch_ws_bytes(*cfg);
  if (need > lmoe::kNoAllocScratchBytes)
    return fail(MOE_ESHAPE, "%s: this call needs %zu bytes of workspace, above the library's fixed %zu "
                "(4 * (2 * ceil(T / 256) * E + T * k) must not exceed it); use moe_dispatch", fn, need,
                lmoe::kNoAllocScratchBytes);
  CHECK(check_device(fn));
  void* ws = nullptr;
  const hipError_t e = lmoe::noalloc_scratch(&ws);
  if (e != hipSuccess) return fail(MOE_ELAUNCH, "%s: no device address for the fixed workspace: %s", fn,
                                   hipGetErrorString(e));
  lmoe::launch_dispatch(*cfg, x, idx, carry, fill, slot, send_buf, ws, (hipStream_t)stream);
  return check_launch(fn);
}

moe_status moe_dispatch_bpr(const moe_cfg* cfg, const void* x, const float* logits, const int32_t* idx,
                            int32_t* fill, int32_t* slot, void* send_buf, int32_t* order, void* ws, size_t ws_bytes,
                            moe_stream_t stream) {
  const char* fn = "moe_dispatch_bpr";
  CHECK(check_cfg(cfg, fn, false));
  REQUIRE_TPTR(x); REQUIRE_TPTR(logits); REQUIRE_TPTR(idx); REQUIRE_PTR(fill);
  REQUIRE_TPTR(slot); REQUIRE_PTR(send_buf); OPTIONAL_PTR(order);
  const size_t need = lmoe::dispatch_bpr_ws_bytes(*cfg);
  if (need > 0) {
    if (ws == nullptr || ws_bytes < need)
      return fail(MOE_EWORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, need, ws ? ws_bytes : 0);
    REQUIRE_PTR(ws);
  }
  CHECK(check_device(fn));
  lmoe::launch_dispatch_bpr(*cfg, x, logits, idx, fill, slot, send_buf, order, ws, (hipStream_t)stream);
  return check_launch(fn);
}

moe_status moe_product_timing(int32_t on) {
  const char* fn = "moe_product_timing";
  const hipError_t e = lmoe::product_timing(on != 0);
  if (e != hipSuccess) return fail(MOE_EDEVICE, "%s: %s", fn, hipGetErrorString(e));
  return ok();
}

moe_status moe_product_times(double* ms, int32_t* counts) {
  const char* fn = "moe_product_times";
  if (ms == nullptr || counts == nullptr) return fail(MOE_EINVAL, "%s: ms and counts are required", fn);
  const hipError_t e = lmoe::product_times(ms, counts);
  if (e != hipSuccess) return fail(MOE_ELAUNCH, "%s: %s", fn, hipGetErrorString(e));
  return ok();
}

moe_status moe_block_op_times(double* ms) {
  const char* fn = "moe_block_op_times";
  if (ms == nullptr) return fail(MOE_EINVAL, "%s: ms is NULL", fn);
  const hipError_t e = lmoe::block_op_times(ms);
  if (e == hipErrorNotReady)
    return fail(MOE_EINVAL, "%s: no timed backward (MOE_BLOCK_TIMED) was issued on this thread and device", fn);
  if (e != hipSuccess) return fail(MOE_ELAUNCH, "%s: %s", fn, hipGetErrorString(e));
  return ok();
}

moe_status moe_block_dw_schedule(const double* op_ms, double a2a_ms, int32_t* dw_order, int32_t* assign,
                                 double* overlap) {
  const char* fn = "moe_block_dw_schedule";
  if (op_ms == nullptr || dw_order == nullptr || overlap == nullptr)
    return fail(MOE_EINVAL, "%s: op_ms, dw_order and overlap are required", fn);
  const std::string err = lmoe::block_dw_schedule(op_ms, a2a_ms, dw_order, assign, overlap);
  if (!err.empty()) return fail(MOE_EINVAL, "%s: %s", fn, err.c_str());
  return ok();
}

moe_status moe_dw_schedule(int32_t n, const int32_t* kind, const double* time, int32_t n_edges, const int32_t* src,
                           const int32_t* dst, int32_t* assign, int32_t* order, double* overlap) {
  const char* fn = "moe_dw_schedule";
  if (overlap == nullptr) return fail(MOE_EINVAL, "%s: overlap is NULL", fn);
  if (n > 0 && (kind == nullptr || time == nullptr || assign == nullptr || order == nullptr))
    return fail(MOE_EINVAL, "%s: kind, time, assign and order are required", fn);
  if (n_edges > 0 && (src == nullptr || dst == nullptr)) return fail(MOE_EINVAL, "%s: src and dst are required", fn);
  const std::string err = lmoe::dw_schedule(n, kind, time, n_edges, src, dst, assign, order, overlap);
  if (!err.empty()) return fail(MOE_EINVAL, "%s: %s", fn, err.c_str());
  return ok();
}

moe_status moe_pipeline_plan(int32_t N, int32_t K, const int32_t* kind, const double* times, const double* join,
                             int32_t G, int32_t* seg_begin, int32_t* seg_end, int32_t* seg_k, int32_t* n_seg,
                             double* total) {
  const char* fn = "moe_pipeline_plan";
  if (n_seg == nullptr || total == nullptr || join == nullptr) return fail(MOE_EINVAL, "%s: join, n_seg and total are required", fn);
  if (N > 0 && (kind == nullptr || times == nullptr || seg_begin == nullptr || seg_end == nullptr || seg_k == nullptr))
    return fail(MOE_EINVAL, "%s: kind, times and the segment arrays are required", fn);
  const std::string err = lmoe::pipeline_plan(N, K, kind, times, join, G, seg_begin, seg_end, seg_k, n_seg, total);
  if (!err.empty()) return fail(MOE_EINVAL, "%s: %s", fn, err.c_str());
  return ok();
}

moe_status moe_pipeline_range_cost(int32_t N, int32_t K, const int32_t* kind, const double* times,
                                   const double* join, int32_t i, int32_t n, int32_t k, double* cost) {
  const char* fn = "moe_pipeline_range_cost";
  if (cost == nullptr || kind == nullptr || times == nullptr || join == nullptr)
    return fail(MOE_EINVAL, "%s: kind, times, join and cost are required", fn);
  if (K < 1 || K > 64 || k < 1 || k > K || i < 1 || n < i || n > N)
    return fail(MOE_EINVAL, "%s: need 1 <= i <= n <= N and 1 <= k <= K <= 64", fn);
  *cost = lmoe::pipeline_range_cost(N, K, kind, times, join, i, n, k);
  return ok();
}

moe_status moe_pack_weights(const moe_cfg* cfg, const void* W1, const void* W2, void* W1p, void* W2p,
                            moe_stream_t stream) {
  const char* fn = "moe_pack_weights";
  CHECK(check_cfg(cfg, fn, true));
  REQUIRE_PTR(W1); REQUIRE_PTR(W2); REQUIRE_PTR(W1p); REQUIRE_PTR(W2p);
  if (W1 == W1p || W2 == W2p || W1p == W2p) return fail(MOE_EINVAL, "%s: packed and source weights may not alias", fn);
  CHECK(check_device(fn));
  lmoe::launch_pack_weights(*cfg, W1, W2, W1p, W2p, (hipStream_t)stream);
  return check_launch(fn);
}

moe_status moe_expert_ffn_fwd(const moe_cfg* cfg, const void* send_buf, const int32_t* row_begin,
                              const int32_t* row_end, const void* W1p, const void* W2p, void* H, void* A,
                              void* expert_out, void* ws, size_t ws_bytes, moe_stream_t stream) {
  const char* fn = "moe_expert_ffn_fwd";
  CHECK(check_cfg(cfg, fn, true));
  REQUIRE_PTR(send_buf); OPTIONAL_PTR(row_begin); REQUIRE_PTR(row_end);
  REQUIRE_PTR(W1p); REQUIRE_PTR(W2p); REQUIRE_PTR(H); REQUIRE_PTR(A); REQUIRE_PTR(expert_out);
  const size_t need = lmoe::expert_sk_ws_bytes(*cfg);
  if (need > 0) {
    if (ws == nullptr || ws_bytes < need)
      return fail(MOE_EWORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, need, ws ? ws_bytes : 0);
    REQUIRE_PTR(ws);
  }
  CHECK(check_device(fn));
  lmoe::launch_expert_fwd(*cfg, send_buf, row_begin, row_end, W1p, W2p, H, A, expert_out, ws, (hipStream_t)stream);
  return check_launch(fn);
}

moe_status moe_combine(const moe_cfg* cfg, const void* expert_out, const int32_t* idx, const int32_t* slot,
                       const float* w, void* y, moe_stream_t stream) {
  const char* fn = "moe_combine";
  CHECK(check_cfg(cfg, fn, false));
  REQUIRE_PTR(expert_out); REQUIRE_TPTR(idx); REQUIRE_TPTR(slot); REQUIRE_TPTR(w); REQUIRE_TPTR(y);
  CHECK(check_device(fn));
  lmoe::launch_combine(*cfg, expert_out, idx, slot, w, y, (hipStream_t)stream);
  return check_launch(fn);
}

moe_status moe_bwd_dx(const moe_cfg* cfg, const void* Wg, const float* logits, const int32_t* idx, const float* w,
                      const int32_t* slot, const int32_t* row_begin, const int32_t* row_end, const void* H,
                      const void* expert_out, const void* W1p, const void* W2p, const void* dy, void* dO, void* dH,
                      void* dXe, float* dlogits, void* dx, void* ws, size_t ws_bytes, moe_stream_t stream) {
  const char* fn = "moe_bwd_dx";
  CHECK(check_cfg(cfg, fn, true));
  REQUIRE_PTR(Wg); REQUIRE_TPTR(logits); REQUIRE_TPTR(idx); REQUIRE_TPTR(w); REQUIRE_TPTR(slot);
  OPTIONAL_PTR(row_begin); REQUIRE_PTR(row_end); REQUIRE_PTR(H); REQUIRE_PTR(expert_out);
  REQUIRE_PTR(W1p); REQUIRE_PTR(W2p); REQUIRE_TPTR(dy); REQUIRE_PTR(dO); REQUIRE_PTR(dH); REQUIRE_PTR(dXe);
  REQUIRE_TPTR(dlogits); REQUIRE_TPTR(dx);
  const size_t need = lmoe::bwd_dx_ws_bytes(*cfg);
  if (need > 0) {
    if (ws == nullptr || ws_bytes < need)
      return fail(MOE_EWORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, need, ws ? ws_bytes : 0);
    REQUIRE_PTR(ws);
  }
  CHECK(check_device(fn));
  hipStream_t s = (hipStream_t)stream;
  lmoe::launch_combine_bwd(*cfg, logits, idx, w, slot, expert_out, dy, dO, dlogits, s);
  lmoe::launch_expert_bwd_dx(*cfg, dO, row_begin, row_end, H, W1p, W2p, dH, dXe, ws, s);
  lmoe::launch_dispatch_bwd(*cfg, Wg, dlogits, idx, slot, dXe, dx, s);
  return check_launch(fn);
}

moe_status moe_bwd_dw(const moe_cfg* cfg, const void* x, const float* dlogits, const int32_t* row_begin,
                      const int32_t* row_end, const void* send_buf, const void* A, const void* dO, const void* dH,
                      void* dW1, void* dW2, float* dWg, void* ws, size_t ws_bytes, moe_stream_t stream) {
  const char* fn = "moe_bwd_dw";
  CHECK(check_cfg(cfg, fn, true));
  REQUIRE_TPTR(dlogits); OPTIONAL_PTR(row_begin); REQUIRE_PTR(row_end); REQUIRE_PTR(send_buf);
  REQUIRE_PTR(A); REQUIRE_PTR(dO); REQUIRE_PTR(dH); REQUIRE_PTR(dW1); REQUIRE_PTR(dW2); REQUIRE_PTR(dWg);
  REQUIRE_TPTR(x);
  const size_t need = lmoe::bwd_dw_ws_bytes(*cfg);
  if (need > 0) {
    if (ws == nullptr || ws_bytes < need)
      return fail(MOE_EWORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, need, ws ? ws_bytes : 0);
    REQUIRE_PTR(ws);
  }
  CHECK(check_device(fn));
  hipStream_t s = (hipStream_t)stream;
  lmoe::launch_expert_bwd_dw(*cfg, send_buf, A, dO, dH, row_begin, row_end, dW1, dW2, s);
  lmoe::launch_dwg(*cfg, x, dlogits, dWg, ws, s);
  return check_launch(fn);
}

// ------------------------------------------------------------------ block
namespace {

moe_status check_block(const moe_block_cfg* c, int32_t n_chunks, const char* fn) {
  if (!c) return fail(MOE_EINVAL, "%s: cfg is NULL", fn);
  CHECK(check_cfg(&c->moe, fn, true));
  if (c->moe.dtype != MOE_BF16) return fail(MOE_EDTYPE, "%s: the block is bf16 only", fn);
  if (c->B < 1 || c->S < 1 || c->heads < 1) return fail(MOE_ESHAPE, "%s: B, S and heads must be >= 1", fn);
  if ((int64_t)c->heads * 128 != c->moe.d_model)
    return fail(MOE_ESHAPE, "%s: d_model=%d is not 128 * heads (heads=%d)", fn, c->moe.d_model, c->heads);
  if (c->moe.d_model > 4096) return fail(MOE_ESHAPE, "%s: d_model=%d > 4096", fn, c->moe.d_model);
  if (c->moe.T != (int64_t)c->B * c->S) return fail(MOE_EINVAL, "%s: moe.T must equal B*S", fn);
  if (n_chunks < 1 || n_chunks > 64 || c->B % n_chunks != 0)
    return fail(MOE_EINVAL, "%s: n_chunks=%d must divide B=%d (1..64)", fn, n_chunks, c->B);
  if (c->dw_order[0] >= 0) {
    int seen = 0;
    for (int q = 0; q < 6; ++q) {
      const int op = c->dw_order[q];
      if (op < MOE_BOP_DW_EXPERT || op > MOE_BOP_DLN1 || (seen >> op) & 1)
        return fail(MOE_EINVAL, "%s: dw_order is not a permutation of MOE_BOP_DW_EXPERT..MOE_BOP_DLN1", fn);
      seen |= 1 << op;
    }
  }
  return MOE_OK;
}

}  // namespace

size_t moe_block_workspace_bytes(const moe_block_cfg* cfg, int32_t n_chunks) {
  if (check_block(cfg, n_chunks, "moe_block_workspace_bytes") != MOE_OK) return 0;
  return lmoe::block_ws_bytes(*cfg, n_chunks);
}

moe_status moe_block_chunked(const moe_block_cfg* cfg, const moe_block_weights* wts, const moe_block_grads* grads,
                             const void* x, void* out, const void* dy, void* dx, const moe_block_acts* acts,
                             int32_t passes, int32_t n_chunks, const moe_stream_t* streams, void* ws,
                             size_t ws_bytes) {
  const char* fn = "moe_block_chunked";
  CHECK(check_block(cfg, n_chunks, fn));
  if (passes < 1 || passes > 7 || passes == MOE_BLOCK_TIMED || passes == (MOE_BLOCK_TIMED | MOE_BLOCK_FWD))
    return fail(MOE_EINVAL, "%s: passes=%d (1 forward, 2 backward, 3 both; | 4 timed, with a backward)", fn, passes);
  if (!wts || !acts || !streams) return fail(MOE_EINVAL, "%s: weights, acts and streams are required", fn);
  REQUIRE_PTR(x);
  REQUIRE_PTR(wts->ln1_g); REQUIRE_PTR(wts->ln1_b); REQUIRE_PTR(wts->Wqkv); REQUIRE_PTR(wts->Wo);
  REQUIRE_PTR(wts->ln2_g); REQUIRE_PTR(wts->ln2_b); REQUIRE_PTR(wts->Wg); REQUIRE_PTR(wts->W1); REQUIRE_PTR(wts->W2);
  REQUIRE_PTR(acts->a); REQUIRE_PTR(acts->ln1_mean); REQUIRE_PTR(acts->ln1_rstd); REQUIRE_PTR(acts->qkv);
  REQUIRE_PTR(acts->attn); REQUIRE_PTR(acts->lse); REQUIRE_PTR(acts->h); REQUIRE_PTR(acts->ln2_mean);
  REQUIRE_PTR(acts->ln2_rstd); REQUIRE_PTR(acts->m); REQUIRE_PTR(acts->logits); REQUIRE_PTR(acts->idx);
  REQUIRE_PTR(acts->w); REQUIRE_PTR(acts->slot); REQUIRE_PTR(acts->fill); REQUIRE_PTR(acts->send_buf);
  REQUIRE_PTR(acts->H); REQUIRE_PTR(acts->A); REQUIRE_PTR(acts->expert_out);
  if (cfg->moe.wpacked) {
    OPTIONAL_PTR(acts->W1p); OPTIONAL_PTR(acts->W2p);
  } else {
    REQUIRE_PTR(acts->W1p); REQUIRE_PTR(acts->W2p);
  }
  if (passes & MOE_BLOCK_FWD) REQUIRE_PTR(out);
  if (passes & MOE_BLOCK_BWD) {
    REQUIRE_PTR(dy); REQUIRE_PTR(dx);
    if (!grads) return fail(MOE_EINVAL, "%s: grads is NULL for a backward pass", fn);
    REQUIRE_PTR(grads->dln1_g); REQUIRE_PTR(grads->dln1_b); REQUIRE_PTR(grads->dWqkv); REQUIRE_PTR(grads->dWo);
    REQUIRE_PTR(grads->dln2_g); REQUIRE_PTR(grads->dln2_b); REQUIRE_PTR(grads->dWg); REQUIRE_PTR(grads->dW1);
    REQUIRE_PTR(grads->dW2);
    REQUIRE_PTR(acts->dO); REQUIRE_PTR(acts->dH); REQUIRE_PTR(acts->dXe); REQUIRE_PTR(acts->dlogits);
    REQUIRE_PTR(acts->dm); REQUIRE_PTR(acts->dh); REQUIRE_PTR(acts->dattn); REQUIRE_PTR(acts->delta);
    REQUIRE_PTR(acts->dqkv); REQUIRE_PTR(acts->da);
  }
  const size_t need = lmoe::block_ws_bytes(*cfg, n_chunks);
  if (ws == nullptr || ws_bytes < need)
    return fail(MOE_EWORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, need, ws ? ws_bytes : 0);
  REQUIRE_PTR(ws);
  CHECK(check_device(fn));
  const hipStream_t st[3] = {(hipStream_t)streams[0], (hipStream_t)streams[1], (hipStream_t)streams[2]};
  const hipError_t e = lmoe::run_block(*cfg, *wts, grads, x, out, dy, dx, *acts, passes, n_chunks, st, ws);
  if (e != hipSuccess) return fail(MOE_ELAUNCH, "%s: %s", fn, hipGetErrorString(e));
  return ok();
}

}  // extern "C"
