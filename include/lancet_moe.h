/*
 * lancet_moe.h -- C ABI of one GPU's share of the MoE-layer training step
 * whose all-to-all communication Lancet (arXiv 2404.19429) overlaps with
 * computation, built for AMD Instinct MI355X (gfx950).
 *
 * The layer (Background, "Mixture of Experts" and Fig. "moe_and_sharding"):
 * a trainable gate scores every expert and keeps the top k; tokens are
 * re-arranged into a fixed-shape E x C buffer (at most C rows per expert,
 * excess tokens dropped); every expert runs a two-layer FFN on its rows; the
 * outputs are gathered back to token order, weighted by the gate.  The
 * backward pass is split into the activation-gradient (dX) chain and the
 * weight-gradient (dW) products, which depend on nothing the dX chain has not
 * already produced (Sec. 2.2, Fig. "example_dw"; Sec. 4), so dW can run on any
 * stream once dX has been issued.  Batch partitions pass the experts' used
 * capacity to the next partition, so routing and drops equal the
 * unpartitioned layer (Sec. 2.3, "Challenge 1").
 *
 * Conventions for every call below:
 *   - All array pointers are DEVICE pointers owned by the caller, 16-byte
 *     aligned, row-major, densely packed.  The library allocates no device
 *     memory and keeps no state besides its compiled kernels and a
 *     thread-local error string.
 *   - "dtype" arrays hold float (MOE_F32) or bfloat16 (MOE_BF16) values as
 *     given by cfg->dtype; every other array has the type in its signature.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the null
 *     stream), never synchronise the host, and read expert row counts on the
 *     device.  Calls on different streams may run concurrently if their
 *     output buffers do not overlap.
 *   - Every call validates its arguments on the host before launching and
 *     returns a moe_status; on failure nothing is launched and
 *     moe_last_error() describes the problem.  T == 0 is valid.
 *   - Rows of an [E][C][*] buffer past an expert's filled range are
 *     unspecified: never read and never written by these calls.
 *   - A device other than gfx950 gives MOE_EDEVICE; a failed launch
 *     MOE_ELAUNCH.
 *
 * Layouts (nn.Linear [out][in]): Wg [E][d], W1 [E][f][d], W2 [E][d][f].
 * Symbols: T tokens, d = d_model, f = d_ff, E experts, k top-k, C capacity,
 * G destination slices of E/G experts each.
 */
#ifndef LANCET_MOE_H
#define LANCET_MOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef void* moe_stream_t; /* hipStream_t */

typedef enum {
  MOE_OK = 0,
  MOE_EINVAL = -1,     /* bad enum value, null pointer, k/E/C/G out of range */
  MOE_ESHAPE = -2,     /* a size outside what the kernels support */
  MOE_EALIGN = -3,     /* a pointer not 16-byte aligned */
  MOE_EDTYPE = -4,     /* unknown dtype */
  MOE_EDEVICE = -5,    /* no HIP device, or the current device is not gfx950 */
  MOE_ELAUNCH = -6,    /* the HIP runtime reported an error */
  MOE_EWORKSPACE = -7  /* workspace missing or smaller than moe_workspace_bytes() */
} moe_status;

typedef enum { MOE_F32 = 0, MOE_BF16 = 1 } moe_dtype;

/* Expert activation.  GELU_TANH is 0.5h(1+tanh(sqrt(2/pi)(h+0.044715h^3))). */
typedef enum { MOE_ACT_IDENTITY = 0, MOE_ACT_RELU = 1, MOE_ACT_GELU_TANH = 2, MOE_ACT_GELU_ERF = 3 } moe_act;

/* Which call a workspace is for (moe_workspace_bytes). */
typedef enum { MOE_CALL_DISPATCH = 0, MOE_CALL_BWD_DX = 1, MOE_CALL_BWD_DW = 2 } moe_call;

/* Host-side description of one MoE layer call. */
typedef struct {
  int64_t T;       /* tokens in this call (a batch partition passes its own T) */
  int32_t d_model; /* multiple of 8; the bf16 expert GEMMs need a multiple of 64 */
  int32_t d_ff;    /* multiple of 8; the bf16 expert GEMMs need a multiple of 64 */
  int32_t E;       /* 1..64 */
  int32_t k;       /* 1..min(E, 8) */
  int32_t C;       /* rows per expert in every [E][C][*] buffer, >= 1 */
  int32_t G;       /* destination slices, E % G == 0 */
  int32_t dtype;   /* moe_dtype */
  int32_t act;     /* moe_act */
  int32_t renorm;  /* 1: top-k weights renormalised over the selected experts; 0: w = softmax(l)[e] */
} moe_cfg;

/* Expert capacity C = ceil(k*T*cf_num / (E*cf_den)) in exact integer
 * arithmetic (Background, "Expert-parallelism": each expert accepts at most C
 * tokens per device).  Host only.  Returns -1 on invalid arguments
 * (E, k, cf_num, cf_den < 1, T < 0) or if C exceeds INT32_MAX. */
int32_t moe_capacity(int64_t T, int32_t E, int32_t k, int32_t cf_num, int32_t cf_den);

/* Bytes of caller-provided device workspace `call` needs for cfg (host only,
 * 0 if none; 0 and a message on invalid cfg). */
size_t moe_workspace_bytes(const moe_cfg* cfg, int32_t call);

/* Message of the last failed call on this thread ("" if none).  Owned by the
 * library, valid until the next call on this thread. */
const char* moe_last_error(void);

/* Top-k gate (Background, "Routing algorithms"; Switch top-1, Sec. 2.3).
 *   x [T][d] dtype, Wg [E][d] dtype, bias [E] float or NULL (a constant
 *   per-expert offset; it receives no gradient).
 *   Out: logits [T][E] float = <x_t, Wg_e> + b_e accumulated in double and
 *   rounded once to float; idx [T][k] int32 = the k experts ordered by
 *   (logit descending, expert index ascending); w [T][k] float = softmax
 *   weight of each choice (renorm: divided by the selected experts' sum). */
moe_status moe_gate_topk(const moe_cfg* cfg, const void* x, const void* Wg, const float* bias,
                         float* logits, int32_t* idx, float* w, moe_stream_t stream);

/* Capacity-bounded dispatch into the all-to-all send layout (Sec. 2.3
 * "Challenge 1"; Implementation, irregular all-to-all with fixed G x C
 * buffers and runtime counts).
 *   In: x [T][d] dtype, idx [T][k] int32, carry [E] int32 rows already used in
 *   each expert by earlier batch partitions (NULL = zeros; 0 <= carry_e <= C).
 *   Assignments are taken token by token, each token's choices in rank order;
 *   an assignment to expert e gets the next free row of e if one is left
 *   below C, else it is dropped.
 *   Out: slot [T][k] int32 (row in the expert's block, -1 = dropped);
 *   fill [E] int32 = carry + rows taken by this call (the next partition's
 *   carry; the per-destination sizes of the first all-to-all are sums of
 *   fill over each slice's E/G experts); send_buf [G][E/G][C][d] dtype
 *   (== [E][C][d]) rows carry_e..fill_e-1 = the kept tokens' rows, bitwise.
 *   ws: moe_workspace_bytes(cfg, MOE_CALL_DISPATCH) bytes of device memory.
 *   carry and fill may not alias. */
moe_status moe_dispatch(const moe_cfg* cfg, const void* x, const int32_t* idx, const int32_t* carry,
                        int32_t* fill, int32_t* slot, void* send_buf, void* ws, size_t ws_bytes,
                        moe_stream_t stream);

/* Expert FFNs forward (Background, "Mixture of Experts"): for every expert e
 * and buffer row i in [row_begin_e, row_end_e):
 *   H[e][i] = W1_e x_i, A[e][i] = act(H[e][i]), expert_out[e][i] = W2_e A[e][i].
 *   send_buf [E][C][d], H and A [E][C][f], expert_out [E][C][d], all dtype;
 *   row_begin/row_end [E] int32 device arrays (row_begin NULL = zeros), the
 *   carry-in and fill of the dispatch that wrote these rows.  H and A are
 *   saved for the backward.  bf16 inputs use MFMA with float accumulation. */
moe_status moe_expert_ffn_fwd(const moe_cfg* cfg, const void* send_buf, const int32_t* row_begin,
                              const int32_t* row_end, const void* W1, const void* W2, void* H, void* A,
                              void* expert_out, moe_stream_t stream);

/* Weighted gather back to token order (Fig. "moe_and_sharding", Gather):
 *   y[t] = sum over r with slot[t][r] >= 0 of w[t][r] * expert_out[idx[t][r]][slot[t][r]],
 *   summed in rank order in float; a token with every choice dropped gets 0.
 *   y [T][d] dtype. */
moe_status moe_combine(const moe_cfg* cfg, const void* expert_out, const int32_t* idx,
                       const int32_t* slot, const float* w, void* y, moe_stream_t stream);

/* Activation-gradient (dX) chain of the layer backward for L = sum <dy, y>
 * (Sec. 2.2 "Opportunity 1", Fig. "example_dw"):
 *   combine backward: dO[e][s] = w[t][r] dy[t], g[t][r] = <dy[t], expert_out[e][s]>;
 *   gate backward (gradient through the weights only, not the selection):
 *     renorm:  dlogits[t][e_r] = w_r (g_r - sum_s w_s g_s), 0 for unselected;
 *     plain:   dlogits[t][j] = sum_r g_r w_r (delta(j, e_r) - p_j), p = softmax(logits[t]);
 *   experts: dH = (dO W2_e) * act'(H), dXe = dH W1_e on rows [row_begin_e, row_end_e);
 *   dispatch backward: dx[t] = sum over kept r of dXe[e_r][s_r] + sum_j dlogits[t][j] Wg_j.
 *   dO, dXe [E][C][d] and dH [E][C][f] dtype (dO and dH are kept for
 *   moe_bwd_dw), dlogits [T][E] float, dx [T][d] dtype.
 *   ws: moe_workspace_bytes(cfg, MOE_CALL_BWD_DX) bytes. */
moe_status moe_bwd_dx(const moe_cfg* cfg, const void* Wg, const float* logits, const int32_t* idx,
                      const float* w, const int32_t* slot, const int32_t* row_begin,
                      const int32_t* row_end, const void* H, const void* expert_out, const void* W1,
                      const void* W2, const void* dy, void* dO, void* dH, void* dXe, float* dlogits,
                      void* dx, void* ws, size_t ws_bytes, moe_stream_t stream);

/* Weight-gradient (dW) products, schedulable on any stream after moe_bwd_dx
 * has been issued (Sec. 4: dW computations may overlap any all-to-all they
 * have no dependency path to):
 *   dW2_e = dO_e^T A_e  [d][f],  dW1_e = dH_e^T X_e  [f][d]  over rows
 *   [row_begin_e, row_end_e) of the expert (X_e = send_buf rows); an expert
 *   with no rows gets exact zeros;  dWg = dlogits^T x  [E][d] float.
 *   dW1, dW2 dtype (float accumulation).  x [T][d] dtype.
 *   ws: moe_workspace_bytes(cfg, MOE_CALL_BWD_DW) bytes. */
moe_status moe_bwd_dw(const moe_cfg* cfg, const void* x, const float* dlogits,
                      const int32_t* row_begin, const int32_t* row_end, const void* send_buf,
                      const void* A, const void* dO, const void* dH, void* dW1, void* dW2, float* dWg,
                      void* ws, size_t ws_bytes, moe_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* LANCET_MOE_H */
