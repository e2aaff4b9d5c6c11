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

size_t bwd_dx_ws_bytes(const moe_cfg& c) { return expert_sk_ws_bytes(c); }

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
// dWg[e][:] = sum_t dlogits[t][e] x[t][:].  Stage 1: a block owns a slab of
// 512 columns (each lane 8 consecutive columns, one 16-byte load per token),
// a chunk of tokens and a group of up to 16 experts; its four waves take
// every fourth token of the chunk, and their sums meet in LDS in wave order.
// Stage 2 adds the chunk partials in chunk order.  Deterministic.
constexpr int kDwgSlab = 512;     // columns per block
constexpr int kDwgEG = 16;        // experts per block

struct DwgPlan {
  int64_t tch, nch;
  int slabs, egroups;
};
static DwgPlan dwg_plan(const moe_cfg& c) {
  DwgPlan q;
  q.slabs = (c.d_model + kDwgSlab - 1) / kDwgSlab;
  q.egroups = (c.E + kDwgEG - 1) / kDwgEG;
  // about 256 blocks over the chunks, at least 64 tokens per chunk
  int64_t want = 256 / (q.slabs * q.egroups);
  if (want < 1) want = 1;
  int64_t tch = (c.T + want - 1) / want;
  if (tch < 64) tch = 64;
  q.tch = tch;
  q.nch = (c.T + tch - 1) / tch;
  return q;
}

template <typename T> __device__ __forceinline__ void load8(const T* p, float (&v)[8]);
template <> __device__ __forceinline__ void load8<uint16_t>(const uint16_t* p, float (&v)[8]) { Vec<uint16_t>::load(p, v); }
template <> __device__ __forceinline__ void load8<float>(const float* p, float (&v)[8]) {
  float a[4], b[4];
  Vec<float>::load(p, a);
  Vec<float>::load(p + 4, b);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[i] = a[i];
    v[4 + i] = b[i];
  }
}

template <typename T, int EG>
__global__ __launch_bounds__(256) void dwg_partial_kernel(const T* __restrict__ x, const float* __restrict__ dl,
                                                          float* __restrict__ part, int64_t T_tokens, int d, int E,
                                                          int64_t tch) {
  __shared__ float red[3][EG][kDwgSlab];
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = blockIdx.x * kDwgSlab + 8 * lane;
  const int e0 = blockIdx.z * kDwgEG;
  const int64_t ch = blockIdx.y;
  const int64_t t_begin = ch * tch;
  const int64_t t_end = min(t_begin + tch, T_tokens);
  float acc[EG][8];
#pragma unroll
  for (int e = 0; e < EG; ++e)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[e][j] = 0.f;
  const bool colok = col < d;
  constexpr int U = 4;   // tokens in flight per wave
  for (int64_t t0 = t_begin + wid; t0 < t_end; t0 += 4 * U) {
    float xv[U][8];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t t = t0 + 4 * u;
      if (colok && t < t_end) load8<T>(x + t * d + col, xv[u]);
      else
#pragma unroll
        for (int j = 0; j < 8; ++j) xv[u][j] = 0.f;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t t = t0 + 4 * u;
      const bool tok = t < t_end;
      const float* dr = dl + (tok ? t : t_begin) * E + e0;
#pragma unroll
      for (int e = 0; e < EG; ++e) {
        const float g = (tok && e0 + e < E) ? dr[e] : 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[e][j] = fmaf(g, xv[u][j], acc[e][j]);
      }
    }
  }
  // Block sum in wave order: waves 1..3 hand their sums to wave 0 through LDS.
  if (wid > 0) {
#pragma unroll
    for (int e = 0; e < EG; ++e)
#pragma unroll
      for (int j = 0; j < 8; ++j) red[wid - 1][e][8 * lane + j] = acc[e][j];
  }
  __syncthreads();
  if (wid == 0 && colok) {
    float* out = part + (ch * E + e0) * (int64_t)d + col;
#pragma unroll
    for (int e = 0; e < EG; ++e) {
      if (e0 + e >= E) continue;
      float v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = ((acc[e][j] + red[0][e][8 * lane + j]) + red[1][e][8 * lane + j]) + red[2][e][8 * lane + j];
      Vec<float>::store(out + (int64_t)e * d, v);
      Vec<float>::store(out + (int64_t)e * d + 4, v + 4);
    }
  }
}

// dWg[i] = sum over chunks of part[c][i], in chunk order; 4 consecutive outputs per thread.
__global__ __launch_bounds__(256) void dwg_reduce_kernel(const float* __restrict__ part, float* __restrict__ dWg,
                                                         int nch, int64_t ed) {
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= ed) return;
  float s[4] = {0.f, 0.f, 0.f, 0.f};
  int c = 0;
  for (; c + 4 <= nch; c += 4) {
    float v[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u) Vec<float>::load(part + (int64_t)(c + u) * ed + i, v[u]);
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int j = 0; j < 4; ++j) s[j] += v[u][j];
  }
  for (; c < nch; ++c) {
    float v[4];
    Vec<float>::load(part + (int64_t)c * ed + i, v);
#pragma unroll
    for (int j = 0; j < 4; ++j) s[j] += v[j];
  }
  Vec<float>::store(dWg + i, s);
}

size_t bwd_dw_ws_bytes(const moe_cfg& c) {
  const DwgPlan q = dwg_plan(c);
  return (size_t)(q.nch * c.E * (int64_t)c.d_model) * sizeof(float);
}

template <typename T>
static void launch_dwg_t(const moe_cfg& c, const void* x, const float* dl, float* part, const DwgPlan& q,
                         hipStream_t s) {
  dim3 grid((unsigned)q.slabs, (unsigned)q.nch, (unsigned)q.egroups);
  if (c.E <= 4)
    hipLaunchKernelGGL((dwg_partial_kernel<T, 4>), grid, dim3(256), 0, s, (const T*)x, dl, part, c.T, c.d_model, c.E, q.tch);
  else if (c.E <= 8)
    hipLaunchKernelGGL((dwg_partial_kernel<T, 8>), grid, dim3(256), 0, s, (const T*)x, dl, part, c.T, c.d_model, c.E, q.tch);
  else
    hipLaunchKernelGGL((dwg_partial_kernel<T, 16>), grid, dim3(256), 0, s, (const T*)x, dl, part, c.T, c.d_model, c.E, q.tch);
}

void launch_dwg(const moe_cfg& c, const void* x, const float* dlogits, float* dWg, void* ws, hipStream_t s) {
  const int64_t ed = (int64_t)c.E * c.d_model;   // a multiple of 8
  const DwgPlan q = dwg_plan(c);                 // nch = 0 when T == 0: the reduce then writes zeros
  float* part = (float*)ws;
  if (q.nch > 0) {
    if (c.dtype == MOE_BF16) launch_dwg_t<uint16_t>(c, x, dlogits, part, q, s);
    else launch_dwg_t<float>(c, x, dlogits, part, q, s);
  }
  hipLaunchKernelGGL(dwg_reduce_kernel, dim3((unsigned)((ed / 4 + 255) / 256)), dim3(256), 0, s, part, dWg,
                     (int)q.nch, ed);
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
