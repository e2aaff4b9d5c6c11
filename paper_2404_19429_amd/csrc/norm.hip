// LayerNorm of the pre-LN block (eps 1e-5, affine gain and bias), bf16 in and out.
//
// Forward: one wavefront per row, statistics and the affine map in double,
// one rounding of the double result to bf16 -- the stored output is the
// correctly rounded LayerNorm of the stored input.  Mean and 1/std are kept
// as float for the backward.
// Backward (float): dx = dres + rstd * (g dy - mean(g dy) - xhat * mean(g dy xhat)),
// fusing the residual branch's gradient dres; the gain and bias gradients are
// written as per-block partial column sums and reduced in a fixed order by a
// second kernel (deterministic).
//
// Rows are split into 16-byte chunks; lane l handles chunks l, l + 64, ...
// (consecutive lanes read consecutive 16 bytes).  Either kernel may also write
// its output in the 16 x 32 blocked layout that the dense products read
// (y_blk / dx_blk non-null; d a multiple of 32): each 16-byte chunk lies
// within one block row, so it is one more 16-byte store.
#include "internal.h"

namespace lmoe {

constexpr int kLnMaxChunks = 8;   // chunks per lane: d <= 64 * 8 * 8 = 4096
// Kernels are instantiated for NC = 1, 2, 4, 8 chunks per lane (the smallest that covers d).
constexpr int kLnBwdRows = 32;    // rows per backward block (4 waves x 8)

// Nearest-even bf16 of a double, rounded once: round the significand to 8
// bits in double, after which the value converts to float exactly.
__device__ __forceinline__ uint32_t f64_to_bf16_bits(double v) {
  uint64_t u = (uint64_t)__double_as_longlong(v);
  u += ((uint64_t)1 << 44) - 1 + ((u >> 45) & 1);
  u &= ~(((uint64_t)1 << 45) - 1);
  return __float_as_uint((float)__longlong_as_double((long long)u)) >> 16;
}

__device__ __forceinline__ void unpack8(const u32x4& r, float* v) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(r[i] << 16);
    v[2 * i + 1] = __uint_as_float(r[i] & 0xffff0000u);
  }
}

template <int NC>
__global__ __launch_bounds__(256) void ln_fwd_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ g,
                                                     const uint16_t* __restrict__ b, uint16_t* __restrict__ y,
                                                     uint16_t* __restrict__ y_blk, float* __restrict__ mean_out,
                                                     float* __restrict__ rstd_out, int64_t T, int d, double eps) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= T) return;
  const int nch = d / 8;
  const uint16_t* xr = x + row * d;
  float v[NC][8];
  double s = 0.0;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int ch = c * 64 + lane;
    if (ch < nch) {
      Vec<uint16_t>::load(xr + 8 * ch, v[c]);
#pragma unroll
      for (int i = 0; i < 8; ++i) s += (double)v[c][i];
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
  const double mu = s / d;
  double q = 0.0;
#pragma unroll
  for (int c = 0; c < NC; ++c)
    if (c * 64 + lane < nch)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const double t = (double)v[c][i] - mu;
        q += t * t;
      }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) q += __shfl_xor(q, o, 64);
  const double rstd = 1.0 / sqrt(q / d + eps);
  uint16_t* yr = y + row * d;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int ch = c * 64 + lane;
    if (ch < nch) {
      float gg[8], bb[8];
      Vec<uint16_t>::load(g + 8 * ch, gg);
      Vec<uint16_t>::load(b + 8 * ch, bb);
      u32x4 r;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const double y0 = ((double)v[c][2 * i] - mu) * rstd * (double)gg[2 * i] + (double)bb[2 * i];
        const double y1 = ((double)v[c][2 * i + 1] - mu) * rstd * (double)gg[2 * i + 1] + (double)bb[2 * i + 1];
        r[i] = f64_to_bf16_bits(y0) | (f64_to_bf16_bits(y1) << 16);
      }
      *reinterpret_cast<u32x4*>(yr + 8 * ch) = r;
      if (y_blk) *reinterpret_cast<u32x4*>(y_blk + blk_off(row, 8 * ch, d)) = r;
    }
  }
  if (lane == 0) {
    mean_out[row] = (float)mu;
    rstd_out[row] = (float)rstd;
  }
}

// part: [gridDim.x][2][d] float partial sums of dy * xhat (gain) and dy (bias).
template <int NC>
__global__ __launch_bounds__(256) void ln_bwd_kernel(const uint16_t* __restrict__ dyl, const uint16_t* __restrict__ x,
                                                     const float* __restrict__ mean, const float* __restrict__ rstd,
                                                     const uint16_t* __restrict__ g, const uint16_t* __restrict__ dres,
                                                     uint16_t* __restrict__ dx, uint16_t* __restrict__ dx_blk,
                                                     float* __restrict__ part, int64_t T, int d) {
  __shared__ __attribute__((aligned(16))) float red[4][64][16];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int nch = d / 8;
  const float inv_d = 1.f / (float)d;
  float pg[NC][8], pb[NC][8];
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int i = 0; i < 8; ++i) pg[c][i] = pb[c][i] = 0.f;
  float gv[NC][8];
#pragma unroll
  for (int c = 0; c < NC; ++c)
    if (c * 64 + lane < nch) Vec<uint16_t>::load(g + 8 * (c * 64 + lane), gv[c]);

  for (int rr = 0; rr < kLnBwdRows / 4; ++rr) {
    const int64_t row = (int64_t)blockIdx.x * kLnBwdRows + wid * (kLnBwdRows / 4) + rr;
    if (row >= T) break;
    const float mu = mean[row], rs = rstd[row];
    // The row's bf16 values, kept packed between the two passes; dres is
    // loaded with x and dy so that its latency hides under the reduction.
    u32x4 xr[NC], dr[NC], rv[NC];
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int ch = c * 64 + lane;
      if (ch < nch) {
        xr[c] = *reinterpret_cast<const u32x4*>(x + row * d + 8 * ch);
        dr[c] = *reinterpret_cast<const u32x4*>(dyl + row * d + 8 * ch);
        rv[c] = *reinterpret_cast<const u32x4*>(dres + row * d + 8 * ch);
        float xv[8], dv[8];
        unpack8(xr[c], xv);
        unpack8(dr[c], dv);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float xh = (xv[i] - mu) * rs;
          const float gy = dv[i] * gv[c][i];
          s1 += gy;
          s2 += gy * xh;
          pg[c][i] = fmaf(dv[i], xh, pg[c][i]);
          pb[c][i] += dv[i];
        }
      }
    }
    s1 = wave_sum(s1) * inv_d;
    s2 = wave_sum(s2) * inv_d;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int ch = c * 64 + lane;
      if (ch < nch) {
        float xv[8], dv[8], r[8], o[8];
        unpack8(xr[c], xv);
        unpack8(dr[c], dv);
        unpack8(rv[c], r);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const float xh = (xv[i] - mu) * rs;
          o[i] = r[i] + rs * (dv[i] * gv[c][i] - s1 - xh * s2);
        }
        Vec<uint16_t>::store(dx + row * d + 8 * ch, o);
        if (dx_blk) Vec<uint16_t>::store(dx_blk + blk_off(row, 8 * ch, d), o);
      }
    }
  }
  // Block partials: the four waves' sums meet in LDS and are added in wave order.
  float* out = part + (int64_t)blockIdx.x * 2 * d;
  const int t = threadIdx.x, tl = t & 63, tp = t >> 6;  // tp: which 4 of a lane's 16 values
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    if (c * 64 >= nch) break;  // uniform
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      red[wid][lane][i] = pg[c][i];
      red[wid][lane][8 + i] = pb[c][i];
    }
    __syncthreads();
    const int ch = c * 64 + tl;
    if (ch < nch) {
      f32x4 acc = *reinterpret_cast<const f32x4*>(&red[0][tl][4 * tp]);
#pragma unroll
      for (int w = 1; w < 4; ++w) acc += *reinterpret_cast<const f32x4*>(&red[w][tl][4 * tp]);
      float* dst = out + (tp >> 1) * d + 8 * ch + 4 * (tp & 1);
      *reinterpret_cast<f32x4*>(dst) = acc;
    }
    __syncthreads();
  }
}

// dg[j] = sum over blocks of part[blk][0][j], db likewise, in a fixed order:
// runs of kGainRun consecutive block partials are summed first (in block
// order, the sum left in the run's first partial row), then the run sums in
// run order.  Two launches spread the reads of the partials over the GPU.
constexpr int kGainRun = 32;
__global__ __launch_bounds__(256) void ln_gain_run_kernel(float* __restrict__ part, int nblk, int d) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= 2 * d) return;
  const int b0 = blockIdx.y * kGainRun, b1 = min(nblk, b0 + kGainRun);
  float acc = 0.f;
#pragma unroll 8
  for (int b = b0; b < b1; ++b) acc += part[(int64_t)b * 2 * d + j];
  part[(int64_t)b0 * 2 * d + j] = acc;
}

__global__ __launch_bounds__(256) void ln_gain_reduce_kernel(const float* __restrict__ part, int nblk, int d,
                                                             float* __restrict__ dg, float* __restrict__ db) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= 2 * d) return;
  const int which = j / d, col = j % d;
  float acc = 0.f;
  for (int b = 0; b < nblk; b += kGainRun) acc += part[(int64_t)b * 2 * d + j];
  (which == 0 ? dg : db)[col] = acc;
}

static int ln_chunks(int d) {
  const int per = (d / 8 + 63) / 64;
  return per <= 1 ? 1 : per <= 2 ? 2 : per <= 4 ? 4 : 8;
}

int ln_bwd_blocks(int64_t T) { return (int)((T + kLnBwdRows - 1) / kLnBwdRows); }

void launch_ln_fwd(const void* x, const void* g, const void* b, void* y, float* mean, float* rstd, int64_t T, int d,
                   hipStream_t s, void* y_blk) {
  if (T <= 0) return;
  const dim3 grid((unsigned)((T + 3) / 4));
  const int nc = ln_chunks(d);
#define LMOE_LN_FWD(NC)                                                                                     \
  hipLaunchKernelGGL(ln_fwd_kernel<NC>, grid, dim3(256), 0, s, (const uint16_t*)x, (const uint16_t*)g,      \
                     (const uint16_t*)b, (uint16_t*)y, (uint16_t*)y_blk, mean, rstd, T, d, 1e-5)
  if (nc == 1) LMOE_LN_FWD(1); else if (nc == 2) LMOE_LN_FWD(2); else if (nc == 4) LMOE_LN_FWD(4); else LMOE_LN_FWD(8);
#undef LMOE_LN_FWD
}

void launch_ln_bwd(const void* dyl, const void* x, const float* mean, const float* rstd, const void* g,
                   const void* dres, void* dx, float* part, int64_t T, int d, hipStream_t s, void* dx_blk) {
  if (T <= 0) return;
  const dim3 grid((unsigned)ln_bwd_blocks(T));
  const int nc = ln_chunks(d);
#define LMOE_LN_BWD(NC)                                                                                     \
  hipLaunchKernelGGL(ln_bwd_kernel<NC>, grid, dim3(256), 0, s, (const uint16_t*)dyl, (const uint16_t*)x,    \
                     mean, rstd, (const uint16_t*)g, (const uint16_t*)dres, (uint16_t*)dx, (uint16_t*)dx_blk, part, T, d)
  if (nc == 1) LMOE_LN_BWD(1); else if (nc == 2) LMOE_LN_BWD(2); else if (nc == 4) LMOE_LN_BWD(4); else LMOE_LN_BWD(8);
#undef LMOE_LN_BWD
}

void launch_ln_gain_reduce(float* part, int64_t T, int d, float* dg, float* db, hipStream_t s) {
  const int nblk = T > 0 ? ln_bwd_blocks(T) : 0;
  const unsigned cols = (unsigned)((2 * d + 255) / 256);
  if (nblk > 0)
    hipLaunchKernelGGL(ln_gain_run_kernel, dim3(cols, (unsigned)((nblk + kGainRun - 1) / kGainRun)), dim3(256), 0, s,
                       part, nblk, d);
  hipLaunchKernelGGL(ln_gain_reduce_kernel, dim3(cols), dim3(256), 0, s, (const float*)part, nblk, d, dg, db);
}

}  // namespace lmoe
