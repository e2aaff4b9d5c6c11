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
 *   - Expert buffers [E][C][X] hold E*Cp*X elements, with Cp = C rounded up
 *     to 16 for MOE_BF16 and Cp = C for MOE_F32.  The buffers an expert
 *     product reads (send_buf, H, A, dO, dH) and the packed weights are, for
 *     MOE_BF16, stored in 16-row x 32-column blocks of 1 KiB: element
 *     (e, r, c) is at e*Cp*X + ((r/16)*(X/32) + c/32)*512 + (r%16)*32 + c%32.
 *     (Each block is one MFMA operand fragment; the GEMMs load it as one
 *     contiguous 1 KiB run.)  The product outputs that only the gathers read
 *     (expert_out, dXe) are row-major: (e, r, c) at (e*Cp + r)*X + c, so a
 *     row is one contiguous run.  For MOE_F32 every buffer is row-major.
 *   - A device other than gfx950 gives MOE_EDEVICE; a failed launch
 *     MOE_ELAUNCH.
 *
 * Layouts (nn.Linear [out][in]): Wg [E][d], W1 [E][f][d], W2 [E][d][f]
 * (row-major; the expert GEMMs take copies made by moe_pack_weights).
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
typedef enum {
  MOE_CALL_DISPATCH = 0,
  MOE_CALL_BWD_DX = 1,
  MOE_CALL_BWD_DW = 2,
  MOE_CALL_FFN_FWD = 3,
  MOE_CALL_DISPATCH_BPR = 4
} moe_call;

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
  int32_t wpacked; /* 1: moe_bwd_dw writes dW1, dW2 in the packed layout of moe_pack_weights (a
                      training loop that keeps the packed copies as its parameters updates them
                      in place and never re-packs); 0: row-major [out][in] */
  int32_t ksplit;  /* bf16 expert products that store a plain product (expert_out in
                      moe_expert_ffn_fwd, dXe in moe_bwd_dx):
                      1: when the call's tile count leaves a short last round, the K sums of
                         those last tiles are split over several blocks and their float
                         partials added in a fixed order (deterministic for a given call, but
                         the summation order, hence the last bits, depends on how many rows
                         the call covers);
                      0: every output element is one K sum taken in order, so results are
                         bitwise independent of how an expert's rows are split into calls
                         (batch partitions) */
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

/* moe_dispatch for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same arguments, kernels and results, without the workspace argument.  The
 * workspace is a fixed 1 MiB array inside the library, one per GPU, held until
 * the process ends; its device address is looked up on the first call on each
 * device.  The call allocates nothing.
 *   Limit: 4 * (2 * ceil(T / 256) * E + T * k) <= 1 MiB (for example T = 65536
 *   tokens at k = 2 and E = 64); larger calls return MOE_ESHAPE and must use
 *   moe_dispatch.
 *   All calls on one GPU share the array: calls that overlap in time on that
 *   GPU (on different streams, or from different threads) race and must not
 *   be issued.  Nothing in the array needs to start at zero. */
moe_status moe_dispatch_noalloc(const moe_cfg* cfg, const void* x, const int32_t* idx, const int32_t* carry,
                                int32_t* fill, int32_t* slot, void* send_buf, moe_stream_t stream);

/* Capacity-bounded dispatch with Batch-prioritized Routing (Sec. 2.3,
 * "Opportunities and Challenges": the tokens of the batch are sorted by
 * importance, the sum of their top-k gating scores, before they are assigned
 * to experts, so the least important tokens are dropped first).
 *   importance[t] = sum over r of softmax(logits[t])[idx[t][r]] (softmax over
 *   all E experts, not renormalised), evaluated in double and rounded once to
 *   float.  The tokens are visited by importance descending, equal importance
 *   in token order, each token's choices in rank order; an assignment takes
 *   the next free row of its expert below C, else it is dropped.  An expert's
 *   rows therefore hold its kept tokens by descending importance.
 *   In: x [T][d] dtype, logits [T][E] float (moe_gate_topk), idx [T][k] int32.
 *   Out: fill [E] int32 = rows taken (min(C, demand_e)); slot [T][k] int32
 *   (token order; -1 = dropped); send_buf as in moe_dispatch, rows 0..fill_e-1;
 *   order [T] int32 (nullable): the visiting order, order[j] = the token
 *   visited j-th.
 *   The whole batch decides the order, so there is no carry-in: partitions of
 *   the batch may only start after this call (the paper's pipelining after the
 *   gate).  ws: moe_workspace_bytes(cfg, MOE_CALL_DISPATCH_BPR) bytes of device
 *   memory.  The sort: 4096-token tiles sorted in LDS, then merged by binary
 *   search (deterministic, no atomics on device memory). */
moe_status moe_dispatch_bpr(const moe_cfg* cfg, const void* x, const float* logits, const int32_t* idx,
                            int32_t* fill, int32_t* slot, void* send_buf, int32_t* order, void* ws, size_t ws_bytes,
                            moe_stream_t stream);

/* Expert weights in the layout the expert GEMMs read, written once per
 * weight update and used by moe_expert_ffn_fwd and moe_bwd_dx:
 *   W1 [E][f][d], W2 [E][d][f] row-major dtype -> W1p [E][f][d], W2p [E][d][f]
 *   in the expert-buffer layout above (bf16: blocks; float: a plain copy). */
moe_status moe_pack_weights(const moe_cfg* cfg, const void* W1, const void* W2, void* W1p, void* W2p,
                            moe_stream_t stream);

/* Expert FFNs forward (Background, "Mixture of Experts"): for every expert e
 * and buffer row i in [row_begin_e, row_end_e):
 *   H[e][i] = W1_e x_i, A[e][i] = act(H[e][i]), expert_out[e][i] = W2_e A[e][i].
 *   send_buf [E][C][d], H and A [E][C][f], expert_out [E][C][d], all dtype;
 *   W1p, W2p from moe_pack_weights; row_begin/row_end [E] int32 device arrays
 *   (row_begin NULL = zeros), the carry-in and fill of the dispatch that
 *   wrote these rows.  H and A are saved for the backward.  bf16 inputs use
 *   MFMA with float accumulation.
 *   ws: moe_workspace_bytes(cfg, MOE_CALL_FFN_FWD) bytes (bf16: partial tiles
 *   and counters of the products' K-split schedule, cleared by the call
 *   itself; float: none, ws may be NULL).  Calls that overlap in time need
 *   separate workspaces. */
moe_status moe_expert_ffn_fwd(const moe_cfg* cfg, const void* send_buf, const int32_t* row_begin,
                              const int32_t* row_end, const void* W1p, const void* W2p, void* H, void* A,
                              void* expert_out, void* ws, size_t ws_bytes, moe_stream_t stream);

/* Weighted gather back to token order (Fig. "moe_and_sharding", Gather):
 *   y[t] = sum over r with slot[t][r] >= 0 of w[t][r] * expert_out[idx[t][r]][slot[t][r]],
 *   summed in rank order in float; a token with every choice dropped gets 0.
 *   y [T][d] dtype. */
moe_status moe_combine(const moe_cfg* cfg, const void* expert_out, const int32_t* idx,
                       const int32_t* slot, const float* w, void* y, moe_stream_t stream);

/* Activation-gradient (dX) chain of the layer backward for L = sum <dy, y>
 * (Sec. 2.3 "Opportunity 1"; Fig. "example_dw" in Sec. 2.2):
 *   combine backward: dO[e][s] = w[t][r] dy[t], g[t][r] = <dy[t], expert_out[e][s]>;
 *   gate backward (gradient through the weights only, not the selection):
 *     renorm:  dlogits[t][e_r] = w_r (g_r - sum_s w_s g_s), 0 for unselected;
 *     plain:   dlogits[t][j] = sum_r g_r w_r (delta(j, e_r) - p_j), p = softmax(logits[t]);
 *   experts: dH = (dO W2_e) * act'(H), dXe = dH W1_e on rows [row_begin_e, row_end_e);
 *   dispatch backward: dx[t] = sum over kept r of dXe[e_r][s_r] + sum_j dlogits[t][j] Wg_j.
 *   dO, dXe [E][C][d] and dH [E][C][f] dtype (dO and dH are kept for
 *   moe_bwd_dw), dlogits [T][E] float, dx [T][d] dtype; W1p, W2p from
 *   moe_pack_weights.
 *   ws: moe_workspace_bytes(cfg, MOE_CALL_BWD_DX) bytes (bf16: the expert
 *   products' K-split workspace, as for moe_expert_ffn_fwd; float: none). */
moe_status moe_bwd_dx(const moe_cfg* cfg, const void* Wg, const float* logits, const int32_t* idx,
                      const float* w, const int32_t* slot, const int32_t* row_begin,
                      const int32_t* row_end, const void* H, const void* expert_out, const void* W1p,
                      const void* W2p, const void* dy, void* dO, void* dH, void* dXe, float* dlogits,
                      void* dx, void* ws, size_t ws_bytes, moe_stream_t stream);

/* Weight-gradient (dW) products, schedulable on any stream after moe_bwd_dx
 * has been issued (Sec. 4: dW computations may overlap any all-to-all they
 * have no dependency path to):
 *   dW2_e = dO_e^T A_e  [d][f],  dW1_e = dH_e^T X_e  [f][d]  over rows
 *   [row_begin_e, row_end_e) of the expert (X_e = send_buf rows); an expert
 *   with no rows gets exact zeros;  dWg = dlogits^T x  [E][d] float.
 *   dW1, dW2 dtype (float accumulation), row-major, or for cfg->wpacked = 1
 *   and MOE_BF16 in the blocked layout of W1p, W2p.  x [T][d] dtype.
 *   ws: moe_workspace_bytes(cfg, MOE_CALL_BWD_DW) bytes. */
moe_status moe_bwd_dw(const moe_cfg* cfg, const void* x, const float* dlogits,
                      const int32_t* row_begin, const int32_t* row_end, const void* send_buf,
                      const void* A, const void* dO, const void* dH, void* dW1, void* dW2, float* dWg,
                      void* ws, size_t ws_bytes, moe_stream_t stream);

/* Per-product timing of the expert GEMMs, a measurement aid: the paper's
 * planners work from measured per-operation times (Sec. 3 "Overview", its
 * profiler and cost model), and a product's own duration is what its
 * roofline needs.  moe_product_timing(1) makes every later expert-product
 * launch of the calling thread, on the device current at this call, record
 * a pair of HIP events around the product on that call's stream (a K-split
 * fix-up launch falls inside its product's pair); moe_product_timing(0)
 * stops.  Either clears the record.  Do not leave it on while a stream is
 * being captured into a graph.  moe_product_times (host; waits for the
 * events) writes, per product in the order FWD1 (H = X W1^T with act(H)),
 * FWD2 (O = A W2^T), dA (with dH = dA act'(H)), dXe (dH W1), dW2, dW1, the
 * summed milliseconds ms[6] and the launch counts counts[6] since the last
 * clear, then clears.  The library owns the events (reused, kept until the
 * process ends).  Errors: MOE_EDEVICE (no device), MOE_EINVAL (NULL
 * arguments), MOE_ELAUNCH (an event could not be made or recorded, or a
 * timed launch came on another device). */
moe_status moe_product_timing(int32_t on);
moe_status moe_product_times(double* ms, int32_t* counts);

/* ------------------------------------------------------------------ block */

/* The pre-LN transformer block whose FFN is the MoE layer, with its
 * non-MoE computation partitioned along the batch and pipelined against the
 * MoE layer's data movement (Sec. 2.3 "Opportunity 2" and "Challenge 1",
 * Fig. "part_all"; Sec. 5.3 "Pipeline Scheduling"):
 *   a = LN1(x), [q k v] = a Wqkv^T, o = causal multi-head attention(q, k, v),
 *   h = x + o Wo^T, m = LN2(h), out = h + MoE(m).
 * LayerNorm: eps 1e-5, gain and bias.  Attention: head dim 128, scores
 * scaled by 1/sqrt(128), softmax in float; head j uses columns
 * 128 j .. 128 j + 127 of each of the q, k, v blocks of Wqkv [3d][d].  No
 * projection biases.  bf16 only (moe.dtype = MOE_BF16). */
/* The block backward's operations, as moe_block_chunked issues them:
 * streams[0] runs the activation-gradient chain 0..7 in this order; the
 * weight-gradient groups 8..13 go to streams[2], each after the chain
 * operation whose output it reads (8 after 1, 9 after 0, 10 and 11 after 3,
 * 12 after 5, 13 after 7). */
typedef enum {
  MOE_BOP_COMBINE_BWD = 0,  /* combine and gate backward: dO, dlogits */
  MOE_BOP_EXPERT_DX = 1,    /* dH = (dO W2) * act'(H), dXe = dH W1 */
  MOE_BOP_DISPATCH_BWD = 2, /* dm = gathered dXe + dlogits Wg */
  MOE_BOP_LN2_BWD = 3,      /* dh = dy + LN2'(dm) (and the gain/bias partials) */
  MOE_BOP_DATTN = 4,        /* d(attention output) = dh Wo */
  MOE_BOP_ATTN_BWD = 5,     /* dqkv */
  MOE_BOP_DA = 6,           /* da = dqkv Wqkv */
  MOE_BOP_LN1_BWD = 7,      /* dx = dh + LN1'(da) (and partials) */
  MOE_BOP_DW_EXPERT = 8,    /* dW1, dW2 */
  MOE_BOP_DWG = 9,          /* dWg */
  MOE_BOP_DLN2 = 10,        /* LN2 gain and bias gradients */
  MOE_BOP_DWO = 11,         /* dWo = dh^T o */
  MOE_BOP_DWQKV = 12,       /* dWqkv = dqkv^T a */
  MOE_BOP_DLN1 = 13,        /* LN1 gain and bias gradients */
  MOE_BOP_COUNT = 14
} moe_block_op;

typedef struct {
  int32_t B;     /* sequences */
  int32_t S;     /* tokens per sequence (any S >= 1) */
  int32_t heads; /* d_model = 128 * heads, d_model <= 4096 */
  moe_cfg moe;   /* the MoE layer: moe.T = B*S, moe.d_model = d_model, moe.C = the
                    capacity of all B*S tokens (batch partitions share it) */
  int32_t dw_order[6]; /* the order in which streams[2] launches the weight-gradient
                          groups: a permutation of MOE_BOP_DW_EXPERT .. MOE_BOP_DLN1
                          (moe_block_dw_schedule computes one); dw_order[0] < 0: the
                          default order 8, 9, 10, 11, 12, 13.  Any order gives the same
                          gradients bit for bit; it changes only when each group runs. */
} moe_block_cfg;

typedef struct {           /* all bf16, caller-owned, read only */
  const void* ln1_g;       /* [d] */
  const void* ln1_b;       /* [d] */
  const void* Wqkv;        /* [3d][d] */
  const void* Wo;          /* [d][d] */
  const void* ln2_g;       /* [d] */
  const void* ln2_b;       /* [d] */
  const void* Wg;          /* [E][d] */
  const void* W1;          /* [E][f][d]; with moe.wpacked = 1 the packed copy (moe_pack_weights) */
  const void* W2;          /* [E][d][f]; likewise */
} moe_block_weights;

typedef struct {           /* written by the backward (overwritten, not accumulated) */
  float* dln1_g;           /* [d] float */
  float* dln1_b;           /* [d] float */
  void* dWqkv;             /* [3d][d] bf16 */
  void* dWo;               /* [d][d] bf16 */
  float* dln2_g;           /* [d] float */
  float* dln2_b;           /* [d] float */
  float* dWg;              /* [E][d] float */
  void* dW1;               /* [E][f][d] bf16 (moe.wpacked = 1: in the packed layout) */
  void* dW2;               /* [E][d][f] bf16 (likewise) */
} moe_block_grads;

/* Caller-owned activations: the forward writes the first group, the backward
 * reads it and writes the second.  bf16 unless marked float/int32.
 * T = B*S, Sp = S rounded up to a multiple of 64. */
typedef struct {
  void* a;                 /* [T][d] LN1(x) */
  float* ln1_mean;         /* [T] float */
  float* ln1_rstd;         /* [T] float, 1/sqrt(var + eps) */
  void* qkv;               /* [T][3d] */
  void* attn;              /* [T][d] attention output o, heads concatenated */
  float* lse;              /* [B][heads][Sp] float, per-query log-sum-exp (base 2) */
  void* h;                 /* [T][d] residual stream after attention */
  float* ln2_mean;         /* [T] float */
  float* ln2_rstd;         /* [T] float */
  void* m;                 /* [T][d] LN2(h), the MoE layer's input */
  float* logits;           /* [T][E] float */
  int32_t* idx;            /* [T][k] int32 */
  float* w;                /* [T][k] float */
  int32_t* slot;           /* [T][k] int32 */
  int32_t* fill;           /* [n_chunks][E] int32: fill after chunk i's dispatch; chunk i
                              owns expert rows [fill[i-1], fill[i]) (fill[-1] = 0) */
  void* send_buf;          /* [E][C][d] (expert buffers in the blocked layout, E*Cp*X elements) */
  void* H;                 /* [E][C][f] */
  void* A;                 /* [E][C][f] */
  void* expert_out;        /* [E][C][d] */
  void* W1p;               /* [E][f][d] packed copy of W1 (moe_pack_weights), written by the forward;
                              unused (may be NULL) with moe.wpacked = 1, whose weights come packed */
  void* W2p;               /* [E][d][f] packed copy of W2 (likewise) */
  /* backward */
  void* dO;                /* [E][C][d] */
  void* dH;                /* [E][C][f] */
  void* dXe;               /* [E][C][d] */
  float* dlogits;          /* [T][E] float */
  void* dm;                /* [T][d] gradient at m */
  void* dh;                /* [T][d] gradient at h */
  void* dattn;             /* [T][d] gradient at o */
  float* delta;            /* [B][heads][Sp] float, rowsum(dO * O) per query and head */
  void* dqkv;              /* [T][3d] */
  void* da;                /* [T][d] gradient at a */
} moe_block_acts;

/* MOE_BLOCK_TIMED (with MOE_BLOCK_BWD): the backward also records timing
 * events around each operation on its stream (no host synchronisation);
 * moe_block_op_times reads them afterwards. */
typedef enum { MOE_BLOCK_FWD = 1, MOE_BLOCK_BWD = 2, MOE_BLOCK_TIMED = 4 } moe_block_pass;

/* Workspace bytes moe_block_chunked needs (host only; 0 and a message on an
 * invalid cfg or n_chunks). */
size_t moe_block_workspace_bytes(const moe_block_cfg* cfg, int32_t n_chunks);

/* One forward and/or backward pass of the block (passes = MOE_BLOCK_FWD,
 * MOE_BLOCK_BWD or both, optionally | MOE_BLOCK_TIMED).
 *   Forward: the B sequences are split into n_chunks partitions of
 *   B/n_chunks whole sequences.  streams[0] (compute) runs LN1, the QKV
 *   projection, attention, the output projection with the residual, LN2 and
 *   the gate of partition 0, 1, ...; then the experts of partition 0, 1, ...
 *   streams[1] (data movement) runs partition i's dispatch as soon as its gate
 *   is done -- starting from the capacity partition i-1 left, so routing,
 *   slots and drops equal the unpartitioned layer -- and its combine (plus the
 *   residual h) as soon as its experts are done.  Partition i's dispatch thus
 *   overlaps partition i+1's attention, and its combine the next partition's
 *   experts.  The block's expert products never split a K sum (moe.ksplit
 *   is ignored and taken as 0), so every output is bitwise independent of
 *   n_chunks.
 *   Backward (unpartitioned; L = sum <dy, out>): the dX chain runs on
 *   streams[0]; every weight gradient (MoE dW1, dW2, dWg, dWo, dWqkv and the
 *   LayerNorm gains and biases) is deferred to streams[2], in cfg->dw_order,
 *   each as soon as its inputs exist (Sec. 2.3 "Opportunity 1"; Sec. 4).
 *   x [T][d], out [T][d], dy [T][d], dx [T][d], bf16.  The backward reads the
 *   forward's acts (a forward with the same n_chunks must precede it).
 *   streams: three hipStream_t (entries may repeat).  When the call returns,
 *   all its work is ordered before any later work on streams[0].
 *   ws: moe_block_workspace_bytes(cfg, n_chunks) bytes.
 *   Errors: n_chunks must divide B (1 <= n_chunks <= 64); d_model = 128 heads
 *   <= 4096; d_ff a multiple of 64; moe.T = B*S. */
moe_status moe_block_chunked(const moe_block_cfg* cfg, const moe_block_weights* wts,
                             const moe_block_grads* grads, const void* x, void* out, const void* dy,
                             void* dx, const moe_block_acts* acts, int32_t passes, int32_t n_chunks,
                             const moe_stream_t* streams, void* ws, size_t ws_bytes);

/* Durations (ms) of the MOE_BOP_COUNT backward operations of this thread's
 * last moe_block_chunked call with MOE_BLOCK_TIMED, from its timing events
 * (host: waits for them, so call it off the hot path).  With all three
 * streams the same, each is that operation's own time.  MOE_EINVAL if no
 * timed backward was issued on this thread and device. */
moe_status moe_block_op_times(double* ms);

/* The weight-gradient schedule pass (Sec. 4; Alg. 1; moe_dw_schedule below)
 * applied to the block backward.  Host only.
 *   The instance: the block backward as the paper's expert-parallel step
 *   would run it, in the order reverse-mode differentiation emits it (each
 *   weight gradient where its layer's backward produces it), 16 instructions:
 *     0 combine bwd, 1 all-to-all (dO to the experts' GPUs), 2 expert dX,
 *     3 expert dW, 4 all-to-all (dXe back), 5 dispatch bwd, 6 dWg (the gate's
 *     backward), 7 LN2 bwd, 8 LN2 gain/bias, 9 dWo, 10 d(attn out),
 *     11 attention bwd, 12 dWqkv, 13 da, 14 LN1 bwd, 15 LN1 gain/bias,
 *   with the edges 0-1, 1-2, 1-3, 2-3, 2-4, 4-5, 0-5, 0-6, 5-7, 7-8, 7-9,
 *   7-10, 10-11, 11-12, 11-13, 13-14, 14-15 (dst reads src's output).
 *   Without a schedule (no all-to-all time) the weight gradients keep this
 *   order, which is the default dw_order.
 *   op_ms [MOE_BOP_COUNT] gives the operations' times (for example from
 *   moe_block_op_times), a2a_ms each all-to-all's (one GPU runs none; the
 *   caller models it, e.g. bytes over link bandwidth).
 *   Out: dw_order [6] = the weight-gradient groups (MOE_BOP_DW_EXPERT ..
 *   MOE_BOP_DLN1) in the order of the reordered sequence, ready for
 *   moe_block_cfg.dw_order; assign [16] (nullable) = the all-to-all
 *   (instruction 1 or 4) each instruction overlaps, -1 if none; *overlap =
 *   the overlapped time.
 *   Errors (MOE_EINVAL): NULL op_ms, dw_order or overlap; a negative or
 *   non-finite time. */
moe_status moe_block_dw_schedule(const double* op_ms, double a2a_ms, int32_t* dw_order, int32_t* assign,
                                 double* overlap);

/* ------------------------------------------------------------ host planner */

/* Weight-gradient computation schedule pass (Sec. 4; Alg. 1).  Host only:
 * every pointer is a host pointer and no GPU is touched.
 *   The instance: n instructions in a valid execution order, kind[i] = 0
 *   (other), 1 (all-to-all) or 2 (weight-gradient computation), time[i] >= 0
 *   (one unit for all), and n_edges dependencies src[e] -> dst[e] (dst
 *   consumes an output of src; src < dst).
 *   Labelling (Sec. 4.1): the candidates of an all-to-all a are the
 *   weight-gradient instructions with no directed path to or from a.
 *   Assignment (Sec. 4.2): all-to-alls in sequence order; for each, while its
 *   unoverlapped time t_u > 0 and an unused candidate is left, the candidate
 *   whose time is closest to t_u (ties: the lower index) is assigned to it and
 *   t_u decreases by its time.
 *   Reordering: each assigned instruction moves right after its all-to-all
 *   (after its last predecessor, if that comes later; an instruction that
 *   consumes an assigned one not yet placed pulls it in first), so the result
 *   is always a valid execution order.
 *   Out: assign[n] = the all-to-all that instruction i overlaps, -1 if none
 *   (always -1 for other kinds); order[n] = the new sequence (a permutation
 *   of 0..n-1); *overlap = sum over all-to-alls of min(t_a, assigned time),
 *   the integer program's objective.  n <= 16384.
 *   Errors (MOE_EINVAL): unknown kind, negative or non-finite time, an edge
 *   with src >= dst or outside 0..n-1, a NULL required pointer. */
moe_status moe_dw_schedule(int32_t n, const int32_t* kind, const double* time, int32_t n_edges, const int32_t* src,
                           const int32_t* dst, int32_t* assign, int32_t* order, double* overlap);

/* Operator-partition pass: pipeline cost and partition-range choice (Sec. 5.1
 * dynamic program; Sec. 5.3 pipeline scheduler).  Host only.
 *   The instance: N forward instructions in execution order, kind[j] = 0
 *   (computation) or 1 (communication); times[j * K + (k - 1)] = the time of
 *   one of k parts of instruction j when its range is split k ways (k = 1:
 *   unsplit; +inf: it cannot be split k ways; the k = 1 time must be finite);
 *   join[k - 1] = the cost of splitting a range's inputs and joining its
 *   outputs for k parts (join[0] is not used).
 *   Range cost P(i, n, k) of instructions i..n (1-based): k = 1, the sum of
 *   the times; otherwise the range's stages (maximal runs of one kind) are
 *   laid out for k partitions, each partition's stage after its previous
 *   stage and after the previous instruction of the same kind in the order
 *   stage by stage, partition by partition; P = the end of the last one plus
 *   join[k - 1].
 *   Plan: T(0) = 0, T(n) = min over ranges i..n of at most G instructions
 *   (G <= 0: no limit) and k = 1..K of T(i - 1) + P(i, n, k); ties take the
 *   smaller i, then the smaller k.
 *   Out: *n_seg ranges seg_begin..seg_end (1-based, in order) with their
 *   seg_k (arrays of N entries); *total = T(N).  N <= 16384, K <= 64.
 *   Cost: O(N * G * K) range evaluations of O(G * K) each; group instructions
 *   (as the paper does) or bound G for long sequences.
 *   Errors (MOE_EINVAL): bad kinds, NaN or negative times, infinite unsplit
 *   times, bad join values, NULL required pointers. */
moe_status moe_pipeline_plan(int32_t N, int32_t K, const int32_t* kind, const double* times, const double* join,
                             int32_t G, int32_t* seg_begin, int32_t* seg_end, int32_t* seg_k, int32_t* n_seg,
                             double* total);

/* P(i, n, k) of moe_pipeline_plan alone (same instance arguments): the
 * predicted time of instructions i..n split k ways. */
moe_status moe_pipeline_range_cost(int32_t N, int32_t K, const int32_t* kind, const double* times,
                                   const double* join, int32_t i, int32_t n, int32_t k, double* cost);

#ifdef __cplusplus
}
#endif

#endif /* LANCET_MOE_H */
