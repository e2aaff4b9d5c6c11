// Capacity-bounded slot assignment, dispatch (scatter), combine (weighted
// gather) and their backward counterparts, plus the gate's weight gradient.
//
// Slot assignment walks assignments token by token, rank by rank; the row an
// assignment receives is carry_e plus the number of earlier assignments to
// the same expert.  It is computed without order-defining atomics in three
// launches: per-chunk expert histograms, a per-expert exclusive scan over
// chunks (starting at carry, which makes batch partitions exact), and
// in-chunk ranks from wavefront ballots.  Rows are then copied with 16-byte
// vector accesses, one thread per (token, 16-byte column chunk).
#include "internal.h"

namespace lmoe {

// Element offset of (expert e, row s, column col) in an [E][C][d] buffer:
// blocked for bf16 (rows padded to 16), row-major for float.
template <typename T>
__device__ __forceinline__ int64_t eoff(int e, int s, int col, int d, int C) {
  const int64_t rows = sizeof(T) == 2 ? pad16(C) : C;
  return (int64_t)e * rows * d + ebuf_off<T>(s, col, d);
}

// ------------------------------------------------------------ slot assignment
// counts[chunk][E]: assignments of each expert inside one chunk of tokens.
__global__ __launch_bounds__(kRouteChunk) void route_count_kernel(const int32_t* __restrict__ idx,
                                                                  int32_t* __restrict__ counts,
                                                                  int64_t T_tokens, int E, int k) {
  __shared__ int32_t hist[kMaxE];
  for (int e = threadIdx.x; e < E; e += blockDim.x) hist[e] = 0;
  __syncthreads();
  const int64_t t = (int64_t)blockIdx.x * kRouteChunk + threadIdx.x;
  if (t < T_tokens)
    for (int r = 0; r < k; ++r) {
      const int e = idx[t * k + r];
      if (e >= 0 && e < E) atomicAdd(&hist[e], 1);  // counts only: order-free
    }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += blockDim.x) counts[(int64_t)blockIdx.x * E + e] = hist[e];
}

// base[chunk][e] = carry_e + assignments to e in earlier chunks; fill_e = min(C, carry_e + all).
__global__ __launch_bounds__(256) void route_scan_kernel(const int32_t* __restrict__ counts,
                                                         int32_t* __restrict__ base,
                                                         const int32_t* __restrict__ carry,
                                                         int32_t* __restrict__ fill, int nchunks, int E,
                                                         int C) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  for (int e = wave; e < E; e += (blockDim.x >> 6)) {
    int running = carry ? carry[e] : 0;
    for (int c0 = 0; c0 < nchunks; c0 += kWave) {
      const int c = c0 + lane;
      const int v = c < nchunks ? counts[(int64_t)c * E + e] : 0;
      int incl = v;
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const int u = __shfl_up(incl, o, kWave);
        if (lane >= o) incl += u;
      }
      if (c < nchunks) base[(int64_t)c * E + e] = running + incl - v;
      running += __shfl(incl, kWave - 1, kWave);
    }
    if (lane == 0) fill[e] = running < C ? running : C;
  }
}

// slot[t][r] = base[chunk][e] + rank among earlier same-expert assignments in the chunk, or -1.
__global__ __launch_bounds__(kRouteChunk) void route_slots_kernel(const int32_t* __restrict__ idx,
                                                                  const int32_t* __restrict__ base,
                                                                  int32_t* __restrict__ slot,
                                                                  int64_t T_tokens, int E, int k, int C) {
  constexpr int NW = kRouteChunk / kWave;
  __shared__ int32_t wcnt[NW][kMaxE];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < NW * kMaxE; i += blockDim.x) (&wcnt[0][0])[i] = 0;
  __syncthreads();

  const int64_t t = (int64_t)blockIdx.x * kRouteChunk + threadIdx.x;
  const bool active = t < T_tokens;
  int my[kMaxK];
  int rank[kMaxK];
#pragma unroll
  for (int r = 0; r < kMaxK; ++r) {
    const int e = (active && r < k) ? idx[t * k + r] : -1;
    my[r] = (e >= 0 && e < E) ? e : -1;  // an out-of-range expert is treated as dropped
    rank[r] = 0;
  }
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
  for (int rp = 0; rp < kMaxK; ++rp) {
    if (rp >= k) break;
    const int v = my[rp];
    uint64_t rem = __ballot(v >= 0);
    while (rem) {
      const int leader = __ffsll((unsigned long long)rem) - 1;
      const int ev = __shfl(v, leader, kWave);
      const uint64_t m = __ballot(v == ev);
      rem &= ~m;
      const int before = __popcll(m & lt);
#pragma unroll
      for (int r = 0; r < kMaxK; ++r)
        if (my[r] == ev) rank[r] += before;
      if (lane == 0) wcnt[wave][ev] += __popcll(m);
    }
  }
  __syncthreads();
  if (!active) return;
#pragma unroll
  for (int r = 0; r < kMaxK; ++r) {
    if (r < k) {
      const int e = my[r];
      int s = -1;
      if (e >= 0) {
        s = base[(int64_t)blockIdx.x * E + e] + rank[r];
        for (int w = 0; w < wave; ++w) s += wcnt[w][e];
      }
      slot[t * k + r] = (s >= 0 && s < C) ? s : -1;
    }
  }
}

// send_buf[e][slot][:] = x[t][:] for every kept (t, r).
template <typename T>
__global__ __launch_bounds__(256) void dispatch_copy_kernel(const T* __restrict__ x, const int32_t* __restrict__ idx,
                                                            const int32_t* __restrict__ slot, T* __restrict__ send,
                                                            int64_t T_tokens, int d, int E, int k, int C) {
  constexpr int V = Vec<T>::N;
  const int nc = d / V;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t t = gid / nc;
  const int c = (int)(gid - t * nc);
  if (t >= T_tokens) return;
  const u32x4 v = *reinterpret_cast<const u32x4*>(x + t * d + (int64_t)c * V);
  for (int r = 0; r < k; ++r) {
    const int s = slot[t * k + r];
    const int e = idx[t * k + r];
    if (s >= 0 && s < C && e >= 0 && e < E) {
      *reinterpret_cast<u32x4*>(send + eoff<T>(e, s, c * V, d, C)) = v;
    }
  }
}

size_t dispatch_ws_bytes(const moe_cfg& c) {
  const int64_t nch = (c.T + kRouteChunk - 1) / kRouteChunk;
  return (size_t)(2 * nch * c.E) * sizeof(int32_t);
}

void launch_dispatch(const moe_cfg& c, const void* x, const int32_t* idx, const int32_t* carry, int32_t* fill,
                     int32_t* slot, void* send_buf, void* ws, hipStream_t s) {
  const int64_t nch = (c.T + kRouteChunk - 1) / kRouteChunk;
  int32_t* counts = (int32_t*)ws;
  int32_t* base = counts + nch * c.E;
  if (nch > 0)
    hipLaunchKernelGGL(route_count_kernel, dim3((unsigned)nch), dim3(kRouteChunk), 0, s, idx, counts, c.T, c.E, c.k);
  hipLaunchKernelGGL(route_scan_kernel, dim3(1), dim3(256), 0, s, counts, base, carry, fill, (int)nch, c.E, c.C);
  if (nch == 0) return;
  hipLaunchKernelGGL(route_slots_kernel, dim3((unsigned)nch), dim3(kRouteChunk), 0, s, idx, base, slot, c.T, c.E,
                     c.k, c.C);
  if (c.dtype == MOE_BF16) {
    const int64_t n = c.T * (c.d_model / 8);
    hipLaunchKernelGGL(dispatch_copy_kernel<uint16_t>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       (const uint16_t*)x, idx, slot, (uint16_t*)send_buf, c.T, c.d_model, c.E, c.k, c.C);
  } else {
    const int64_t n = c.T * (c.d_model / 4);
    hipLaunchKernelGGL(dispatch_copy_kernel<float>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       (const float*)x, idx, slot, (float*)send_buf, c.T, c.d_model, c.E, c.k, c.C);
  }
}

// -------------------------------------------------------------------- combine
// y[t][:] = resid[t][:] + sum_r kept w[t][r] * O[e][s][:], in rank order, float
// accumulation (resid NULL = 0; the block passes its residual stream).
template <typename T>
__global__ __launch_bounds__(256) void combine_kernel(const T* __restrict__ O, const int32_t* __restrict__ idx,
                                                      const int32_t* __restrict__ slot, const float* __restrict__ w,
                                                      const T* __restrict__ resid, T* __restrict__ y, int64_t T_tokens,
                                                      int d, int E, int k, int C) {
  constexpr int V = Vec<T>::N;
  const int nc = d / V;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t t = gid / nc;
  const int c = (int)(gid - t * nc);
  if (t >= T_tokens) return;
  float acc[V];
  if (resid) {
    Vec<T>::load(resid + t * d + (int64_t)c * V, acc);
  } else {
#pragma unroll
    for (int i = 0; i < V; ++i) acc[i] = 0.f;
  }
  for (int r = 0; r < k; ++r) {
    const int s = slot[t * k + r];
    const int e = idx[t * k + r];
    if (s >= 0 && s < C && e >= 0 && e < E) {
      const float wr = w[t * k + r];
      float v[V];
      Vec<T>::load(O + eoff<T>(e, s, c * V, d, C), v);
#pragma unroll
      for (int i = 0; i < V; ++i) acc[i] = fmaf(wr, v[i], acc[i]);
    }
  }
  Vec<T>::store(y + t * d + (int64_t)c * V, acc);
}

void launch_combine(const moe_cfg& c, const void* O, const int32_t* idx, const int32_t* slot, const float* w,
                    void* y, hipStream_t s, const void* resid) {
  if (c.T == 0) return;
  if (c.dtype == MOE_BF16) {
    const int64_t n = c.T * (c.d_model / 8);
    hipLaunchKernelGGL(combine_kernel<uint16_t>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       (const uint16_t*)O, idx, slot, w, (const uint16_t*)resid, (uint16_t*)y, c.T, c.d_model, c.E,
                       c.k, c.C);
  } else {
    const int64_t n = c.T * (c.d_model / 4);
    hipLaunchKernelGGL(combine_kernel<float>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       (const float*)O, idx, slot, w, (const float*)resid, (float*)y, c.T, c.d_model, c.E, c.k, c.C);
  }
}

// ------------------------------------------------------ combine + gate backward
// One wavefront per token: dO[e][s] = w dy, g_r = <dy, O[e][s]>, then dlogits.
template <typename T>
__global__ __launch_bounds__(256) void combine_bwd_kernel(const float* __restrict__ logits,
                                                          const int32_t* __restrict__ idx,
                                                          const float* __restrict__ w,
                                                          const int32_t* __restrict__ slot,
                                                          const T* __restrict__ O, const T* __restrict__ dy,
                                                          T* __restrict__ dO, float* __restrict__ dlogits,
                                                          int64_t T_tokens, int d, int E, int k, int C, int renorm) {
  constexpr int V = Vec<T>::N;
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (t >= T_tokens) return;
  int er[kMaxK], sr[kMaxK];
  float wr[kMaxK], gp[kMaxK];
#pragma unroll
  for (int r = 0; r < kMaxK; ++r) {
    er[r] = r < k ? idx[t * k + r] : 0;
    sr[r] = r < k ? slot[t * k + r] : -1;
    if (er[r] < 0 || er[r] >= E || sr[r] >= C) { er[r] = 0; sr[r] = -1; }
    wr[r] = r < k ? w[t * k + r] : 0.f;
    gp[r] = 0.f;
  }
  const int nc = d / V;
  for (int c = lane; c < nc; c += kWave) {
    float g[V];
    Vec<T>::load(dy + t * d + (int64_t)c * V, g);
#pragma unroll
    for (int r = 0; r < kMaxK; ++r) {
      if (sr[r] >= 0) {
        const int64_t off = eoff<T>(er[r], sr[r], c * V, d, C);
        float o[V], out[V];
        Vec<T>::load(O + off, o);
#pragma unroll
        for (int i = 0; i < V; ++i) {
          gp[r] = fmaf(g[i], o[i], gp[r]);
          out[i] = wr[r] * g[i];
        }
        Vec<T>::store(dO + off, out);
      }
    }
  }
  float gsum = 0.f;  // sum_r w_r g_r
#pragma unroll
  for (int r = 0; r < kMaxK; ++r) {
    gp[r] = wave_sum(gp[r]);
    gsum = fmaf(wr[r], gp[r], gsum);
  }
  // dlogits: lane j handles expert j (E <= 64).
  const int j = lane;
  float dl = 0.f;
  if (renorm) {
#pragma unroll
    for (int r = 0; r < kMaxK; ++r)
      if (r < k && er[r] == j) dl = wr[r] * (gp[r] - gsum);
  } else {
    const float lj = j < E ? logits[t * E + j] : -INFINITY;
    float m = lj;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, kWave));
    const float ex = j < E ? expf(lj - m) : 0.f;
    const float pj = ex / wave_sum(ex);
    dl = -pj * gsum;
#pragma unroll
    for (int r = 0; r < kMaxK; ++r)
      if (r < k && er[r] == j) dl += gp[r] * wr[r];
  }
  if (j < E) dlogits[t * E + j] = dl;
}

size_t bwd_dx_ws_bytes(const moe_cfg&) { return 0; }

void launch_combine_bwd(const moe_cfg& c, const float* logits, const int32_t* idx, const float* w,
                        const int32_t* slot, const void* O, const void* dy, void* dO, float* dlogits,
                        hipStream_t s) {
  if (c.T == 0) return;
  const unsigned blocks = (unsigned)((c.T + 3) / 4);
  if (c.dtype == MOE_BF16)
    hipLaunchKernelGGL(combine_bwd_kernel<uint16_t>, dim3(blocks), dim3(256), 0, s, logits, idx, w, slot,
                       (const uint16_t*)O, (const uint16_t*)dy, (uint16_t*)dO, dlogits, c.T, c.d_model, c.E, c.k,
                       c.C, c.renorm);
  else
    hipLaunchKernelGGL(combine_bwd_kernel<float>, dim3(blocks), dim3(256), 0, s, logits, idx, w, slot,
                       (const float*)O, (const float*)dy, (float*)dO, dlogits, c.T, c.d_model, c.E, c.k, c.C,
                       c.renorm);
}

// ----------------------------------------------------------- dispatch backward
// dx[t] = sum_r kept dXe[e][s] + sum_j dlogits[t][j] Wg[j]  (renorm: only the k selected j are nonzero).
template <typename T>
__global__ __launch_bounds__(256) void dispatch_bwd_kernel(const T* __restrict__ Wg, const float* __restrict__ dl,
                                                           const int32_t* __restrict__ idx,
                                                           const int32_t* __restrict__ slot,
                                                           const T* __restrict__ dXe, T* __restrict__ dx,
                                                           int64_t T_tokens, int d, int E, int k, int C, int renorm) {
  constexpr int V = Vec<T>::N;
  const int nc = d / V;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t t = gid / nc;
  const int c = (int)(gid - t * nc);
  if (t >= T_tokens) return;
  float acc[V];
#pragma unroll
  for (int i = 0; i < V; ++i) acc[i] = 0.f;
  for (int r = 0; r < k; ++r) {
    const int s = slot[t * k + r];
    const int e = idx[t * k + r];
    if (s >= 0 && s < C && e >= 0 && e < E) {
      float v[V];
      Vec<T>::load(dXe + eoff<T>(e, s, c * V, d, C), v);
#pragma unroll
      for (int i = 0; i < V; ++i) acc[i] += v[i];
    }
  }
  const int nj = renorm ? k : E;
  for (int q = 0; q < nj; ++q) {
    const int j = renorm ? idx[t * k + q] : q;
    if (j < 0 || j >= E) continue;
    const float a = dl[t * E + j];
    float g[V];
    Vec<T>::load(Wg + (int64_t)j * d + (int64_t)c * V, g);
#pragma unroll
    for (int i = 0; i < V; ++i) acc[i] = fmaf(a, g[i], acc[i]);
  }
  Vec<T>::store(dx + t * d + (int64_t)c * V, acc);
}

void launch_dispatch_bwd(const moe_cfg& c, const void* Wg, const float* dlogits, const int32_t* idx,
                         const int32_t* slot, const void* dXe, void* dx, hipStream_t s) {
  if (c.T == 0) return;
  if (c.dtype == MOE_BF16) {
    const int64_t n = c.T * (c.d_model / 8);
    hipLaunchKernelGGL(dispatch_bwd_kernel<uint16_t>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       (const uint16_t*)Wg, dlogits, idx, slot, (const uint16_t*)dXe, (uint16_t*)dx, c.T,
                       c.d_model, c.E, c.k, c.C, c.renorm);
  } else {
    const int64_t n = c.T * (c.d_model / 4);
    hipLaunchKernelGGL(dispatch_bwd_kernel<float>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       (const float*)Wg, dlogits, idx, slot, (const float*)dXe, (float*)dx, c.T, c.d_model, c.E,
                       c.k, c.C, c.renorm);
  }
}

// -------------------------------------------------------------------- dWg
// dWg[e][:] = sum_t dlogits[t][e] x[t][:].  Stage 1: per token chunk partial
// sums (one thread per column, float accumulators per expert); stage 2: sum
// of the partials in chunk order.  Deterministic.
constexpr int kDwgCols = 256;

static int64_t dwg_chunk_tokens(int64_t T) {
  int64_t tch = (T + 127) / 128;
  return tch < 64 ? 64 : tch;
}

template <typename T, int EMAX>
__global__ __launch_bounds__(kDwgCols) void dwg_partial_kernel(const T* __restrict__ x, const float* __restrict__ dl,
                                                               float* __restrict__ part, int64_t T_tokens, int d,
                                                               int E, int64_t tch) {
  __shared__ float sdl[64][EMAX];
  const int64_t ch = blockIdx.y;
  const int col = blockIdx.x * kDwgCols + threadIdx.x;
  float acc[EMAX];
#pragma unroll
  for (int e = 0; e < EMAX; ++e) acc[e] = 0.f;
  const int64_t t_begin = ch * tch;
  const int64_t t_end = (t_begin + tch < T_tokens) ? t_begin + tch : T_tokens;
  for (int64_t tb = t_begin; tb < t_end; tb += 64) {
    __syncthreads();
    for (int i = threadIdx.x; i < 64 * EMAX; i += kDwgCols) {
      const int tt = i / EMAX, e = i % EMAX;
      sdl[tt][e] = (tb + tt < t_end && e < E) ? dl[(tb + tt) * E + e] : 0.f;
    }
    __syncthreads();
    if (col < d) {
      const int64_t n = (t_end - tb) < 64 ? (t_end - tb) : 64;
      for (int tt = 0; tt < n; ++tt) {
        float xv;
        if constexpr (sizeof(T) == 2) xv = bf16_bits_to_f32(x[(tb + tt) * d + col]);
        else xv = x[(tb + tt) * d + col];
#pragma unroll
        for (int e = 0; e < EMAX; ++e) acc[e] = fmaf(sdl[tt][e], xv, acc[e]);
      }
    }
  }
  if (col < d) {
#pragma unroll
    for (int e = 0; e < EMAX; ++e)
      if (e < E) part[(ch * E + e) * d + col] = acc[e];
  }
}

__global__ __launch_bounds__(256) void dwg_reduce_kernel(const float* __restrict__ part, float* __restrict__ dWg,
                                                         int nch, int E, int d) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)E * d) return;
  float s = 0.f;
  for (int c = 0; c < nch; ++c) s += part[(int64_t)c * E * d + i];
  dWg[i] = s;
}

size_t bwd_dw_ws_bytes(const moe_cfg& c) {
  const int64_t tch = dwg_chunk_tokens(c.T);
  const int64_t nch = (c.T + tch - 1) / tch;
  return (size_t)(nch * c.E * (int64_t)c.d_model) * sizeof(float);
}

template <typename T, int EMAX>
static void launch_dwg_e(const moe_cfg& c, const void* x, const float* dl, float* part, int64_t tch, int64_t nch,
                         hipStream_t s) {
  dim3 grid((unsigned)((c.d_model + kDwgCols - 1) / kDwgCols), (unsigned)nch);
  hipLaunchKernelGGL((dwg_partial_kernel<T, EMAX>), grid, dim3(kDwgCols), 0, s, (const T*)x, dl, part, c.T,
                     c.d_model, c.E, tch);
}

template <typename T>
static void launch_dwg_t(const moe_cfg& c, const void* x, const float* dl, float* part, int64_t tch, int64_t nch,
                         hipStream_t s) {
  if (c.E <= 4) launch_dwg_e<T, 4>(c, x, dl, part, tch, nch, s);
  else if (c.E <= 8) launch_dwg_e<T, 8>(c, x, dl, part, tch, nch, s);
  else if (c.E <= 16) launch_dwg_e<T, 16>(c, x, dl, part, tch, nch, s);
  else if (c.E <= 32) launch_dwg_e<T, 32>(c, x, dl, part, tch, nch, s);
  else launch_dwg_e<T, 64>(c, x, dl, part, tch, nch, s);
}

void launch_dwg(const moe_cfg& c, const void* x, const float* dlogits, float* dWg, void* ws, hipStream_t s) {
  const int64_t ed = (int64_t)c.E * c.d_model;
  const int64_t tch = dwg_chunk_tokens(c.T);
  const int64_t nch = (c.T + tch - 1) / tch;   // 0 when T == 0: the reduce then writes zeros
  float* part = (float*)ws;
  if (nch > 0) {
    if (c.dtype == MOE_BF16) launch_dwg_t<uint16_t>(c, x, dlogits, part, tch, nch, s);
    else launch_dwg_t<float>(c, x, dlogits, part, tch, nch, s);
  }
  hipLaunchKernelGGL(dwg_reduce_kernel, dim3((unsigned)((ed + 255) / 256)), dim3(256), 0, s, part, dWg, (int)nch,
                     c.E, c.d_model);
}

}  // namespace lmoe

namespace lmoe {

// ------------------------------------------------------------- weight packing
// Row-major [R][X] matrices -> blocked layout (bf16), one thread per 16-byte
// chunk: reads are coalesced along rows, writes land as 64-byte block rows.
__global__ __launch_bounds__(256) void pack_blocked_kernel(const uint16_t* __restrict__ src, uint16_t* __restrict__ dst,
                                                           int64_t nmat, int R, int X) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int cpr = X / 8;
  const int64_t per = (int64_t)R * cpr;
  if (gid >= nmat * per) return;
  const int64_t m = gid / per;
  const int64_t rem = gid - m * per;
  const int r = (int)(rem / cpr), c = (int)(rem % cpr) * 8;
  const int64_t base = m * (int64_t)R * X;
  *reinterpret_cast<u32x4*>(dst + base + blk_off(r, c, X)) =
      *reinterpret_cast<const u32x4*>(src + base + (int64_t)r * X + c);
}

void launch_pack_weights(const moe_cfg& c, const void* W1, const void* W2, void* W1p, void* W2p, hipStream_t s) {
  const int64_t E = c.E, d = c.d_model, f = c.d_ff;
  if (c.dtype == MOE_BF16) {
    const int64_t n = E * f * d / 8;
    hipLaunchKernelGGL(pack_blocked_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       (const uint16_t*)W1, (uint16_t*)W1p, E, (int)f, (int)d);
    hipLaunchKernelGGL(pack_blocked_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s,
                       (const uint16_t*)W2, (uint16_t*)W2p, E, (int)d, (int)f);
  } else {
    const size_t bytes = (size_t)E * f * d * sizeof(float);
    (void)hipMemcpyAsync(W1p, W1, bytes, hipMemcpyDeviceToDevice, s);
    (void)hipMemcpyAsync(W2p, W2, bytes, hipMemcpyDeviceToDevice, s);
  }
}

}  // namespace lmoe
