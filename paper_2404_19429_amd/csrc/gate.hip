// Top-k gate: logits = x Wg^T (+ bias), top-k selection and combine weights.
//
// One wavefront scores TPW tokens.  Lanes own 16-byte column chunks of the
// token row and accumulate every expert's partial dot product in double;
// a recursive-halving reduce-scatter across lanes then leaves each expert's
// full sum in one lane.  Because bf16 x bf16 (and f32 x f32) products are
// exact in double and the double sum is far more precise than float, the
// emitted float logit is the correctly rounded dot product except when the
// exact value lies within ~1e-16 relative of a float rounding boundary; the
// top-k decision is taken on these float logits, so it matches any other
// correctly rounded evaluation bit for bit.
#include "internal.h"

namespace lmoe {

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

template <int EMAX>
struct Log2 { static constexpr int v = (EMAX <= 1) ? 0 : 1 + Log2<(EMAX >> 1)>::v; };
template <> struct Log2<1> { static constexpr int v = 0; };

template <typename T, int EMAX, int TPW>
__global__ __launch_bounds__(256) void gate_topk_kernel(const T* __restrict__ x, const T* __restrict__ Wg,
                                                       const float* __restrict__ bias,
                                                       float* __restrict__ logits, int32_t* __restrict__ idx,
                                                       float* __restrict__ wout, int64_t T_tokens, int d,
                                                       int E, int k, int renorm) {
  constexpr int V = Vec<T>::N;
  constexpr int LE = Log2<EMAX>::v;
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  const int64_t t0 = wave * TPW;
  if (t0 >= T_tokens) return;

  double acc[TPW][EMAX];
#pragma unroll
  for (int tt = 0; tt < TPW; ++tt)
#pragma unroll
    for (int e = 0; e < EMAX; ++e) acc[tt][e] = 0.0;

  const int nchunk = d / V;
  for (int c = lane; c < nchunk; c += kWave) {
    float xv[TPW][V];
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
      if (t0 + tt < T_tokens) {
        Vec<T>::load(x + (t0 + tt) * (int64_t)d + (int64_t)c * V, xv[tt]);
      } else {
#pragma unroll
        for (int i = 0; i < V; ++i) xv[tt][i] = 0.f;
      }
    }
#pragma unroll
    for (int e = 0; e < EMAX; ++e) {
      if (e < E) {
        float wv[V];
        Vec<T>::load(Wg + (int64_t)e * d + (int64_t)c * V, wv);
#pragma unroll
        for (int tt = 0; tt < TPW; ++tt)
#pragma unroll
          for (int i = 0; i < V; ++i) acc[tt][e] = fma((double)xv[tt][i], (double)wv[i], acc[tt][e]);
      }
    }
  }

  // Reduce-scatter: after round j the lane keeps half of its list (upper half
  // if lane bit j is set) and adds the partner's copy of that half.
#pragma unroll
  for (int j = 0; j < LE; ++j) {
    const int L = EMAX >> j;
    const int h = L >> 1;
    const bool up = (lane >> j) & 1;
#pragma unroll
    for (int i = 0; i < EMAX / 2; ++i) {
      if (i < h) {
#pragma unroll
        for (int tt = 0; tt < TPW; ++tt) {
          double send = up ? acc[tt][i] : acc[tt][i + h];
          double keep = up ? acc[tt][i + h] : acc[tt][i];
          double recv = __shfl_xor(send, 1 << j, kWave);
          acc[tt][i] = keep + recv;
        }
      }
    }
  }
#pragma unroll
  for (int j = LE; j < 6; ++j)
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) acc[tt][0] += __shfl_xor(acc[tt][0], 1 << j, kWave);

  // Expert owned by this lane: bit-reversal of the low LE lane bits.
  int e_own = 0;
#pragma unroll
  for (int j = 0; j < LE; ++j) e_own |= ((lane >> j) & 1) << (LE - 1 - j);
  const bool valid = (lane < EMAX) && (e_own < E);
  const double b = (valid && bias) ? (double)bias[e_own] : 0.0;

#pragma unroll
  for (int tt = 0; tt < TPW; ++tt) {
    const int64_t t = t0 + tt;
    if (t >= T_tokens) break;
    const float l = valid ? (float)(acc[tt][0] + b) : 0.f;
    if (valid) logits[t * E + e_own] = l;
    uint64_t key = valid ? (((uint64_t)float_order_key(l) << 32) | (uint64_t)(0xffffffffu - (uint32_t)e_own)) : 0ull;
    // k rounds of a wave-wide max over (logit, -expert) keys; lane r keeps choice r.
    int my_e = 0;
    float my_l = 0.f, m = 0.f, sel_sum = 0.f;
#pragma unroll
    for (int r = 0; r < kMaxK; ++r) {
      if (r < k) {
        const uint64_t best = wave_max_u64(key);
        const int be = (int)(0xffffffffu - (uint32_t)(best & 0xffffffffu));
        const float bl = float_from_order_key((uint32_t)(best >> 32));
        if (r == 0) m = bl;
        sel_sum += expf(bl - m);
        if (lane == r) { my_e = be; my_l = bl; }
        if (valid && e_own == be) key = 0ull;
      }
    }
    const float denom = renorm ? sel_sum : wave_sum(valid ? expf(l - m) : 0.f);
    if (lane < k) {
      idx[t * k + lane] = my_e;
      wout[t * k + lane] = expf(my_l - m) / denom;
    }
  }
}

template <typename T, int EMAX>
static void launch_gate_e(const moe_cfg& c, const void* x, const void* Wg, const float* bias, float* logits,
                          int32_t* idx, float* w, hipStream_t s) {
  constexpr int TPW = EMAX >= 64 ? 1 : (EMAX >= 32 ? 2 : 4);
  const int64_t waves = (c.T + TPW - 1) / TPW;
  const int64_t blocks = (waves + 3) / 4;
  hipLaunchKernelGGL((gate_topk_kernel<T, EMAX, TPW>), dim3((unsigned)blocks), dim3(256), 0, s,
                     (const T*)x, (const T*)Wg, bias, logits, idx, w, c.T, c.d_model, c.E, c.k, c.renorm);
}

template <typename T>
static void launch_gate_t(const moe_cfg& c, const void* x, const void* Wg, const float* bias, float* logits,
                          int32_t* idx, float* w, hipStream_t s) {
  if (c.E <= 4) launch_gate_e<T, 4>(c, x, Wg, bias, logits, idx, w, s);
  else if (c.E <= 8) launch_gate_e<T, 8>(c, x, Wg, bias, logits, idx, w, s);
  else if (c.E <= 16) launch_gate_e<T, 16>(c, x, Wg, bias, logits, idx, w, s);
  else if (c.E <= 32) launch_gate_e<T, 32>(c, x, Wg, bias, logits, idx, w, s);
  else launch_gate_e<T, 64>(c, x, Wg, bias, logits, idx, w, s);
}

void launch_gate(const moe_cfg& c, const void* x, const void* Wg, const float* bias, float* logits,
                 int32_t* idx, float* w, hipStream_t s) {
  if (c.T == 0) return;
  if (c.dtype == MOE_BF16) launch_gate_t<uint16_t>(c, x, Wg, bias, logits, idx, w, s);
  else launch_gate_t<float>(c, x, Wg, bias, logits, idx, w, s);
}

}  // namespace lmoe
