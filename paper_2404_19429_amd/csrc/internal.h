// Internal launchers shared between the kernel files and the C-ABI layer.
#pragma once

#include "common.h"

namespace lmoe {

constexpr int kMaxK = 8;       // largest supported top-k
constexpr int kMaxE = 64;      // largest supported expert count (one lane per expert in the gate)
constexpr int kRouteChunk = 256;  // tokens per slot-assignment chunk

// gate.hip
void launch_gate(const moe_cfg& c, const void* x, const void* Wg, const float* bias, float* logits,
                 int32_t* idx, float* w, hipStream_t s);

// route.hip
size_t dispatch_ws_bytes(const moe_cfg& c);
void launch_dispatch(const moe_cfg& c, const void* x, const int32_t* idx, const int32_t* carry, int32_t* fill,
                     int32_t* slot, void* send_buf, void* ws, hipStream_t s);
void launch_combine(const moe_cfg& c, const void* O, const int32_t* idx, const int32_t* slot, const float* w,
                    void* y, hipStream_t s);
size_t bwd_dx_ws_bytes(const moe_cfg& c);
void launch_combine_bwd(const moe_cfg& c, const float* logits, const int32_t* idx, const float* w,
                        const int32_t* slot, const void* O, const void* dy, void* dO, float* dlogits, hipStream_t s);
void launch_dispatch_bwd(const moe_cfg& c, const void* Wg, const float* dlogits, const int32_t* idx,
                         const int32_t* slot, const void* dXe, void* dx, hipStream_t s);
size_t bwd_dw_ws_bytes(const moe_cfg& c);
void launch_dwg(const moe_cfg& c, const void* x, const float* dlogits, float* dWg, void* ws, hipStream_t s);

// gemm.hip: expert GEMMs over [E][C][*] buffers with per-expert row ranges.
void launch_expert_fwd(const moe_cfg& c, const void* X, const int32_t* rb, const int32_t* re, const void* W1,
                       const void* W2, void* H, void* A, void* O, hipStream_t s);
void launch_expert_bwd_dx(const moe_cfg& c, const void* dO, const int32_t* rb, const int32_t* re, const void* H,
                          const void* W1, const void* W2, void* dH, void* dXe, hipStream_t s);
void launch_expert_bwd_dw(const moe_cfg& c, const void* X, const void* A, const void* dO, const void* dH,
                          const int32_t* rb, const int32_t* re, void* dW1, void* dW2, hipStream_t s);

}  // namespace lmoe
