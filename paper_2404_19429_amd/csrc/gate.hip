// Top-k gate: logits = x Wg^T (+ bias), top-k selection and combine weights.
//
// The logits are a skinny product (tokens x E, E <= 64) computed on the fp64
// matrix cores: a block owns 16 * MT tokens and every expert, as MT x NT tiles
// of 16 x 16 doubles (v_mfma_f64_16x16x4).  Its NWV waves split d into
// interleaved chunks and meet in LDS, summing in wave order.  Because bf16 x bf16 (and
// f32 x f32) products are exact in double and the double sum is far more
// precise than float, the emitted float logit is the correctly rounded dot
// product except when the exact value lies within ~1e-15 relative of a float
// rounding boundary.  The top-k decision is taken on these float logits, so it
// matches any other evaluation that rounds the same values the same way.
//
// Operand mapping of one 16-byte load per lane: lane (i = lane & 15,
// q = lane >> 4) loads V consecutive elements of row i (a token of x, or an
// expert of Wg) at column 4V*c + V*q of the piece; MFMA j of chunk c then
// takes element j.  The product's k-index q therefore stands for the same
// column in both operands, which is all a dot product needs.
#include "internal.h"

namespace lmoe {

typedef double f64x4 __attribute__((ext_vector_type(4)));

// Order-preserving map of a float to uint32 (-0 treated as +0).
__device__ __forceinline__ uint32_t float_order_key(float f) {
  uint32_t u = __float_as_uint(f);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float float_from_order_key(uint32_t o) {
  uint32_t u = (o & 0x80000000u) ? (o & 0x7fffffffu) : ~o;
  return __uint_as_float(u);
}

// Element j of a 16-byte vector as a double.
template <typename T> __device__ __forceinline__ double elem_f64(const u32x4& v, int j);
template <> __device__ __forceinline__ double elem_f64<uint16_t>(const u32x4& v, int j) {
  const uint32_t w = v[j >> 1];
  return (double)__uint_as_float((j & 1) ? (w & 0xffff0000u) : (w << 16));
}
template <> __device__ __forceinline__ double elem_f64<float>(const u32x4& v, int j) {
  return (double)__uint_as_float(v[j]);
}

constexpr int kGateGroup = 4;   // chunks whose loads are in flight together

template <typename T, int MT, int NT, int NWV>
__global__ __launch_bounds__(64 * NWV) void gate_topk_kernel(const T* __restrict__ x, const T* __restrict__ Wg,
                                                            const float* __restrict__ bias,
                                                            float* __restrict__ logits, int32_t* __restrict__ idx,
                                                            float* __restrict__ wout, int64_t T_tokens, int d,
                                                            int E, int k, int renorm) {
  constexpr int V = Vec<T>::N;          // elements per 16-byte load
  constexpr int CW = 4 * V;             // columns per chunk (four lane groups)
  constexpr int TM = 16 * MT;           // tokens per block
  __shared__ double red[NWV - 1][MT][NT][4][kWave];
  __shared__ float lg[TM][kMaxE + 1];

  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int i16 = lane & 15, q = lane >> 4;
  const int64_t t0 = (int64_t)blockIdx.x * TM;

  const T* xr[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    int64_t t = t0 + mt * 16 + i16;
    if (t >= T_tokens) t = T_tokens - 1;  // rows past the end are computed and discarded
    xr[mt] = x + t * d;
  }
  const T* wr[NT];
  bool wok[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int e = nt * 16 + i16;
    wok[nt] = e < E;
    wr[nt] = Wg + (int64_t)(wok[nt] ? e : 0) * d;
  }

  f64x4 acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f64x4{0.0, 0.0, 0.0, 0.0};

  // Wave wid takes chunks wid, wid + NWV, ...; kGateGroup of them per round,
  // loads first (unconditional, from a clamped column; masked after), then
  // the products, so the waits can retire one chunk at a time.
  const int nchunks = (d + CW - 1) / CW;
  for (int c0 = wid; c0 < nchunks; c0 += NWV * kGateGroup) {
    u32x4 xv[kGateGroup][MT], wv[kGateGroup][NT];
    bool ok[kGateGroup];
#pragma unroll
    for (int g = 0; g < kGateGroup; ++g) {
      const int col = (c0 + g * NWV) * CW + q * V;
      ok[g] = col < d;   // d is a multiple of V: a load is wholly inside or outside
      const int colc = ok[g] ? col : 0;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) xv[g][mt] = *reinterpret_cast<const u32x4*>(xr[mt] + colc);
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) wv[g][nt] = *reinterpret_cast<const u32x4*>(wr[nt] + colc);
    }
    __builtin_amdgcn_sched_barrier(0);   // keep every load of the round ahead of the products
#pragma unroll
    for (int g = 0; g < kGateGroup; ++g) {
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        if (!ok[g] || !wok[nt]) wv[g][nt] = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int j = 0; j < V; ++j) {
        double a[MT], b[NT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) a[mt] = elem_f64<T>(xv[g][mt], j);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) b[nt] = elem_f64<T>(wv[g][nt], j);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt)
            acc[mt][nt] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[mt], b[nt], acc[mt][nt], 0, 0, 0);
      }
    }
  }

  // Wave sums meet in wave order.  Accumulator element r of a lane holds
  // row q + 4r, column i16 of its 16 x 16 tile: token mt*16 + q + 4r, expert
  // nt*16 + i16.
  if (wid > 0) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[wid - 1][mt][nt][r][lane] = acc[mt][nt][r];
  }
  __syncthreads();
  if (wid == 0) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        const int e = nt * 16 + i16;
        if (e >= E) continue;
        const double b = bias ? (double)bias[e] : 0.0;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          double s = acc[mt][nt][r];
#pragma unroll
          for (int w = 0; w < NWV - 1; ++w) s += red[w][mt][nt][r][lane];
          lg[mt * 16 + q + 4 * r][e] = (float)(s + b);
        }
      }
  }
  __syncthreads();

  // Logits out: the block's rows are one contiguous run of [T][E].
  const int64_t ntok = (T_tokens - t0) < TM ? (T_tokens - t0) : TM;
  for (int i = threadIdx.x; i < ntok * E; i += blockDim.x) logits[t0 * E + i] = lg[i / E][i % E];

  // Top-k by (logit desc, expert asc), one thread per token.
  if (threadIdx.x < ntok) {
    const int tl = threadIdx.x;
    uint64_t best[kMaxK];
#pragma unroll
    for (int r = 0; r < kMaxK; ++r) best[r] = 0ull;
    for (int e = 0; e < E; ++e) {
      uint64_t key = ((uint64_t)float_order_key(lg[tl][e]) << 32) | (uint64_t)(0xffffffffu - (uint32_t)e);
#pragma unroll
      for (int r = 0; r < kMaxK; ++r) {
        if (r < k && key > best[r]) {
          const uint64_t tmp = best[r];
          best[r] = key;
          key = tmp;
        }
      }
    }
    const float m = float_from_order_key((uint32_t)(best[0] >> 32));
    float denom = 0.f;
    if (renorm) {
#pragma unroll
      for (int r = 0; r < kMaxK; ++r)
        if (r < k) denom += expf(float_from_order_key((uint32_t)(best[r] >> 32)) - m);
    } else {
      for (int e = 0; e < E; ++e) denom += expf(lg[tl][e] - m);
    }
    const int64_t t = t0 + tl;
#pragma unroll
    for (int r = 0; r < kMaxK; ++r) {
      if (r < k) {
        const int be = (int)(0xffffffffu - (uint32_t)(best[r] & 0xffffffffu));
        const float bl = float_from_order_key((uint32_t)(best[r] >> 32));
        idx[t * k + r] = be;
        wout[t * k + r] = expf(bl - m) / denom;
      }
    }
  }
}

template <typename T, int MT, int NT, int NWV>
static void launch_gate_e(const moe_cfg& c, const void* x, const void* Wg, const float* bias, float* logits,
                          int32_t* idx, float* w, hipStream_t s) {
  const int64_t blocks = (c.T + 16 * MT - 1) / (16 * MT);
  hipLaunchKernelGGL((gate_topk_kernel<T, MT, NT, NWV>), dim3((unsigned)blocks), dim3(64 * NWV), 0, s,
                     (const T*)x, (const T*)Wg, bias, logits, idx, w, c.T, c.d_model, c.E, c.k, c.renorm);
}

// 32 tokens per block; d is split over 8 waves (4 when four expert tiles
// already give each wave independent accumulators and more registers).
template <typename T>
static void launch_gate_t(const moe_cfg& c, const void* x, const void* Wg, const float* bias, float* logits,
                          int32_t* idx, float* w, hipStream_t s) {
  if (c.E <= 16) launch_gate_e<T, 2, 1, 8>(c, x, Wg, bias, logits, idx, w, s);
  else if (c.E <= 32) launch_gate_e<T, 2, 2, 8>(c, x, Wg, bias, logits, idx, w, s);
  else if (c.E <= 48) launch_gate_e<T, 2, 3, 4>(c, x, Wg, bias, logits, idx, w, s);
  else launch_gate_e<T, 2, 4, 4>(c, x, Wg, bias, logits, idx, w, s);
}

void launch_gate(const moe_cfg& c, const void* x, const void* Wg, const float* bias, float* logits,
                 int32_t* idx, float* w, hipStream_t s) {
  if (c.T == 0) return;
  if (c.dtype == MOE_BF16) launch_gate_t<uint16_t>(c, x, Wg, bias, logits, idx, w, s);
  else launch_gate_t<float>(c, x, Wg, bias, logits, idx, w, s);
}

}  // namespace lmoe
