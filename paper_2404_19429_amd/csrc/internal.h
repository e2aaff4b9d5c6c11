// Internal launchers shared between the kernel files and the C-ABI layer.
#pragma once

#include <algorithm>
#include <atomic>
#include <string>

#include "common.h"

namespace lmoe {

inline int current_device() {
  int d = 0;
  if (hipGetDevice(&d) != hipSuccess) d = 0;
  return d;
}

// A kernel that uses more dynamic LDS than the default limit must be allowed
// it once per device.  `mask` (one per kernel, zero-initialised) records the
// devices 0..63 done so far; two threads racing on a first call both set the
// attribute, which is harmless.  Devices past 63 set it on every call.
inline void allow_dyn_lds(const void* kern, int bytes, std::atomic<uint64_t>& mask) {
  const int dev = current_device();
  const uint64_t bit = dev < 64 ? (uint64_t)1 << dev : 0;
  if (bit && (mask.load(std::memory_order_acquire) & bit)) return;
  if (hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, bytes) == hipSuccess && bit)
    mask.fetch_or(bit, std::memory_order_release);
}

// Compute units of the current device (cached per device 0..63).
inline int num_cus() {
  static std::atomic<int> cache[64];
  const int dev = current_device();
  if (dev < 64) {
    const int n = cache[dev].load(std::memory_order_relaxed);
    if (n > 0) return n;
  }
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
  if (dev < 64) cache[dev].store(n, std::memory_order_relaxed);
  return n;
}

constexpr int kMaxK = 8;       // largest supported top-k
constexpr int kMaxE = 64;      // largest supported expert count (one lane per expert in the gate)
constexpr int kRouteChunk = 256;  // tokens per slot-assignment chunk

// plan.cpp (host only): the weight-gradient computation schedule pass.
constexpr int kMaxPlanInstr = 1 << 14;
std::string dw_schedule(int n, const int32_t* kind, const double* time, int n_edges, const int32_t* src,
                        const int32_t* dst, int32_t* assign, int32_t* order, double* overlap);

double pipeline_range_cost(int N, int K, const int32_t* kind, const double* times, const double* join, int i, int n,
                           int k);
// The block backward's weight-gradient schedule (the instance is described
// with moe_block_dw_schedule in lancet_moe.h).
std::string block_dw_schedule(const double* op_ms, double a2a_ms, int32_t* dw_order, int32_t* assign,
                              double* overlap);
std::string pipeline_plan(int N, int K, const int32_t* kind, const double* times, const double* join, int G,
                          int32_t* seg_begin, int32_t* seg_end, int32_t* seg_k, int32_t* n_seg, double* total);

// gate.hip
void launch_gate(const moe_cfg& c, const void* x, const void* Wg, const float* bias, float* logits,
                 int32_t* idx, float* w, hipStream_t s);

// route.hip
size_t dispatch_ws_bytes(const moe_cfg& c);
void launch_dispatch(const moe_cfg& c, const void* x, const int32_t* idx, const int32_t* carry, int32_t* fill,
                     int32_t* slot, void* send_buf, void* ws, hipStream_t s);
// moe_dispatch_noalloc: the device address, on the current device, of the
// library's fixed dispatch workspace (kNoAllocScratchBytes), looked up once per device.
constexpr size_t kNoAllocScratchBytes = (size_t)1 << 20;
hipError_t noalloc_scratch(void** out);
size_t dispatch_bpr_ws_bytes(const moe_cfg& c);
void launch_dispatch_bpr(const moe_cfg& c, const void* x, const float* logits, const int32_t* idx, int32_t* fill,
                         int32_t* slot, void* send_buf, int32_t* order, void* ws, hipStream_t s);
void launch_combine(const moe_cfg& c, const void* O, const int32_t* idx, const int32_t* slot, const float* w,
                    void* y, hipStream_t s, const void* resid = nullptr);
size_t bwd_dx_ws_bytes(const moe_cfg& c);
void launch_combine_bwd(const moe_cfg& c, const float* logits, const int32_t* idx, const float* w,
                        const int32_t* slot, const void* O, const void* dy, void* dO, float* dlogits, hipStream_t s);
void launch_dispatch_bwd(const moe_cfg& c, const void* Wg, const float* dlogits, const int32_t* idx,
                         const int32_t* slot, const void* dXe, void* dx, hipStream_t s);
size_t bwd_dw_ws_bytes(const moe_cfg& c);
void launch_dwg(const moe_cfg& c, const void* x, const float* dlogits, float* dWg, void* ws, hipStream_t s);

// Expert weights into the layout the expert GEMMs read (blocked for bf16, a copy for float).
void launch_pack_weights(const moe_cfg& c, const void* W1, const void* W2, void* W1p, void* W2p, hipStream_t s);

// gemm.hip: expert GEMMs over [E][C][*] buffers with per-expert row ranges.
// The row-ragged products take a workspace of expert_sk_ws_bytes(c) bytes
// (partial tiles and counters of their K-split schedule; unused for float).
size_t expert_sk_ws_bytes(const moe_cfg& c);
void launch_expert_fwd(const moe_cfg& c, const void* X, const int32_t* rb, const int32_t* re, const void* W1,
                       const void* W2, void* H, void* A, void* O, void* ws, hipStream_t s);
void launch_expert_bwd_dx(const moe_cfg& c, const void* dO, const int32_t* rb, const int32_t* re, const void* H,
                          const void* W1, const void* W2, void* dH, void* dXe, void* ws, hipStream_t s);
void launch_expert_bwd_dw(const moe_cfg& c, const void* X, const void* A, const void* dO, const void* dH,
                          const int32_t* rb, const int32_t* re, void* dW1, void* dW2, hipStream_t s);
// Per-product timing of the expert products on this thread (moe_product_timing):
// product_timing(on) starts (or stops) and clears the record on the current
// device; product_times sums the recorded durations (ms) and launch counts per
// product and clears the record (hipErrorUnknown if an event could not be made
// or recorded, or a launch came on another device).
enum { kProdFwd1 = 0, kProdFwd2, kProdDA, kProdDXe, kProdDW2, kProdDW1, kProducts };
hipError_t product_timing(bool on);
hipError_t product_times(double* ms, int32_t* counts);

// Dense bf16 products of the block (gemm.hip).
// launch_dense_wgrad: C[M][N] = A^T B with A [K][M], B [K][N] row-major bf16
// (sum over K rows), on the wide kernel with K split into token ranges whose
// float partials go to `part` (wgrad_ws_bytes(M, N) bytes).
size_t wgrad_ws_bytes(int M, int N);
void launch_dense_wgrad(int M, int N, int64_t K, const void* A, const void* B, void* C, void* part, hipStream_t s);
// Row-major [M][K] -> blocked [pad16(M)][K] (K a multiple of 32), and dense
// products on the wide kernel over blocked operands (see gemm.hip).
void launch_pack_rows(const void* src, void* dst, int64_t M, int K, hipStream_t s);
void launch_dense_wide(int64_t M, int N, int K, const void* A, const void* B, bool b_nk, void* C, int64_t ldc,
                       const void* resid, hipStream_t s);

// attn.hip: causal attention of the block (head dim 128).  Pointers are at
// the first token of nseq whole sequences of S tokens; lse and delta rows have
// stride attn_stat_stride(S).
inline int attn_stat_stride(int S) { return (S + 63) / 64 * 64; }
// o_blk / dqkv_blk non-null: the output is also written in the 16 x 32 blocked
// layout of the dense products ([pad16(nseq S)][d] / [..][3 d]; the padding
// rows are not written).
void launch_attn_fwd(const void* qkv, void* o, float* lse, int nseq, int S, int H, hipStream_t s,
                     void* o_blk = nullptr);
void launch_attn_bwd(const void* qkv, const void* o, const void* dout, const float* lse, float* delta, void* dqkv,
                     int nseq, int S, int H, hipStream_t s, void* dqkv_blk = nullptr);

// norm.hip: LayerNorm (eps 1e-5) of bf16 rows of width d (multiple of 8, <= 4096).
// The backward writes ln_bwd_blocks(T) x 2 x d float partials, reduced by
// launch_ln_gain_reduce into the gain and bias gradients (the reduction
// overwrites some partials: run it once per backward).
int ln_bwd_blocks(int64_t T);
// y_blk / dx_blk non-null (d a multiple of 32): the output is also written in
// the 16 x 32 blocked layout of the dense products (padding rows not written).
void launch_ln_fwd(const void* x, const void* g, const void* b, void* y, float* mean, float* rstd, int64_t T, int d,
                   hipStream_t s, void* y_blk = nullptr);
void launch_ln_bwd(const void* dyl, const void* x, const float* mean, const float* rstd, const void* g,
                   const void* dres, void* dx, float* part, int64_t T, int d, hipStream_t s, void* dx_blk = nullptr);
void launch_ln_gain_reduce(float* part, int64_t T, int d, float* dg, float* db, hipStream_t s);

// block.cpp: the partitioned block (arguments validated by the C ABI layer).
size_t block_ws_bytes(const moe_block_cfg& c, int n_chunks);
void dw_launch_order(const moe_block_cfg& c, int32_t out[6]);
hipError_t block_op_times(double* ms);   // hipErrorNotReady: no timed backward on this thread and device
hipError_t run_block(const moe_block_cfg& c, const moe_block_weights& W, const moe_block_grads* G, const void* x,
                     void* out, const void* dy, void* dx, const moe_block_acts& A, int passes, int n,
                     const hipStream_t st[3], void* ws);

}  // namespace lmoe
