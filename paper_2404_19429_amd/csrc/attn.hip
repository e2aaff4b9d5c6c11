// Causal multi-head self-attention of the pre-LN block, forward and backward,
// on bf16 MFMA (v_mfma_f32_16x16x32_bf16) with float softmax.
//
// Layout: q, k, v are column blocks of qkv [T][3d] (row stride 3d); head h
// uses columns h*128 .. h*128+127 of each block; token t = b*S + s.  The
// output o [T][d] holds head h at columns h*128.  lse [B][H][Sp] (Sp = S
// rounded up to 64; entries past S unspecified) keeps, per query, the
// log-sum-exp of its scores in base-2 units (m + log2 l with scores scaled by
// log2(e)/sqrt(128)); the backward recomputes probabilities from it.  delta
// has the same layout.
//
// Transposed-score trick.  With the MFMA output layout (lane l holds column
// l%16 and rows 4*(l/16) .. +3 of a 16x16 tile), computing S^T = K Q^T puts
// one query per lane column, so per-query softmax statistics are lane-local
// up to a reduction over the four 16-lane groups, and the probabilities a
// lane holds -- 4 consecutive keys in each 16-key fragment -- are exactly an
// MFMA B operand for O^T = V^T P^T once its K index is read as
// (fragment pair, lane group, register) -> key.  The matching A operand V^T
// comes from row-major V in LDS through ds_read_b64_tr_b16.  Nothing is
// transposed through LDS and P never leaves registers.
//
// K, V, Q and dO tiles are 64 rows x 128 columns, row-major in LDS with the
// 16-byte chunk c of row r stored at chunk c ^ 2*(r & 7), loaded with
// global_load_lds_dwordx4 into a two-stage ring.  Rows past the sequence are
// loaded from a zero page and masked.
//
// The backward is deterministic: a delta pre-pass (D = rowsum(dO * O)), a
// query-owned kernel for dQ and a key-owned kernel for dK and dV, each
// recomputing the probabilities it needs (no atomics).
#include "internal.h"
#include "lds_ops.h"

namespace lmoe {

constexpr int kHD = 128;  // head dimension
constexpr int kTR = 64;   // rows per K/V/Q/dO tile
constexpr int kTileElems = kTR * kHD;
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ int rsw(int r) { return 2 * (r & 7); }

// Element offset of (row r, column n) in a swizzled 64 x 128 tile.
__device__ __forceinline__ int toff(int r, int n) { return r * kHD + (((n >> 3) ^ rsw(r)) << 3) + (n & 7); }

// One 64 x 128 tile: 1024 chunks of 16 bytes = 16 wave instructions, split over NW waves.
template <int NW>
__device__ __forceinline__ void load_tile(const uint16_t* base, int64_t ld, int row0, int rowlim, uint16_t* stage,
                                          int wid, int lane) {
#pragma unroll
  for (int i = 0; i < 16 / NW; ++i) {
    const int q = i * NW + wid;            // LDS bytes [1024 q, 1024 q + 1024): rows 4q .. 4q+3
    const int L = q * 64 + lane;
    const int r = L >> 4, c = (L & 15) ^ rsw(r);
    const int row = row0 + r;
    const void* src = row < rowlim ? (const void*)(base + (int64_t)row * ld + 8 * c) : (const void*)g_zero16;
    dma16(src, stage + q * 512);
  }
}

// Fragment reads, split into issue and wait: the *_issue calls start 8 reads
// and return; the registers are pending until the matching wait (an
// s_waitcnt lgkmcnt(0) that names them), so MFMAs on other registers overlap
// the reads.  At most 8 reads are in flight (the counter holds 15).
// rows_issue: A operand with K = the 128 columns, fragments (rf = u % 4,
// kk = kk0 + u / 4): rows 16 rf + l%16, columns 32 kk + 8 (l/16) .. +7.
// cols_issue / cols_finish: A operand with K = rows (transposed reads),
// fragments (cf, ks) for cf in {cf0, cf0 + 1}, ks in {0, 1}: columns
// 16 cf + l%16; K index 8 (l/16) + j reads row 16 (2 ks) + 4 (l/16) + j for
// j < 4 and row 16 (2 ks + 1) + 4 (l/16) + j - 4 for j >= 4; stored
// f[2 (cf - cf0) + ks].
__device__ __forceinline__ void rows_issue(u32x4 (&f)[8], const uint16_t* st, int kk0, int lane) {
  uint32_t a[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) a[u] = lds_addr(st + toff(16 * (u % 4) + (lane & 15), 32 * (kk0 + u / 4) + 8 * (lane >> 4)));
  Rd128Issue<8>::run(f, a);
}
__device__ __forceinline__ void cols_issue(u32x2 (&o)[8], const uint16_t* st, int cf0, int lane) {
  const int g = lane >> 4, j = lane & 15;
  uint32_t a[8];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int cf = cf0 + (u >> 1), ks = u & 1;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = 16 * (2 * ks + h) + 4 * g + (j >> 2);
      a[2 * u + h] = lds_addr(st + toff(r, 16 * cf + 4 * (j & 3)));
    }
  }
  RdTrIssue8::run(o, a);
}
// Wait states before LDS reads land in registers that MFMAs issued just
// before still read as sources.
__device__ __forceinline__ void mfma_src_gap() { asm volatile("s_nop 7" ::: "memory"); }

__device__ __forceinline__ void cols_finish(u32x4 (&f)[4], u32x2 (&o)[8]) {
  lds_wait(o);
#pragma unroll
  for (int u = 0; u < 4; ++u) f[u] = u32x4{o[2 * u][0], o[2 * u][1], o[2 * u + 1][0], o[2 * u + 1][1]};
}

// 2^x with the hardware instruction (v_exp_f32, about 1 ulp; results below
// the float normal range flush to 0, which only a probability too small to
// change a bf16-rounded product can be).  The library exp2f adds a range
// fix-up around it (five more instructions per value).
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ f32x4 mfma(const u32x4& a, const u32x4& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// B operand from two 16-row accumulator fragments (rows 4*(l/16)+v of each):
// K index j < 4 -> x0[j], j >= 4 -> x1[j-4].
__device__ __forceinline__ u32x4 pack_b(const f32x4& x0, const f32x4& x1) {
  return u32x4{pack_bf16x2(x0[0], x0[1]), pack_bf16x2(x0[2], x0[3]), pack_bf16x2(x1[0], x1[1]),
               pack_bf16x2(x1[2], x1[3])};
}

// 16 bytes of row `row` (columns c0 .. c0+7) or zeros past the limit.
__device__ __forceinline__ u32x4 load_row16(const uint16_t* base, int64_t ld, int row, int rowlim, int c0) {
  if (row >= rowlim) return u32x4{0u, 0u, 0u, 0u};
  return *reinterpret_cast<const u32x4*>(base + (int64_t)row * ld + c0);
}


// Max / sum over the four 16-lane groups (lanes l, l^16, l^32, l^48) with
// gfx950's lane-swap instructions: swapping v with itself, permlane16_swap
// returns (v, partner at l^16) in one order or the other, and permlane32_swap
// likewise for l^32, so combining the two results needs no lane select and no
// trip through the LDS crossbar.
__device__ __forceinline__ float group_max(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float group_sum(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Store 4 consecutive columns (c0 .. c0+3) of one row as bf16.
__device__ __forceinline__ void store4(uint16_t* p, float a, float b, float c, float d) {
  *reinterpret_cast<u32x2*>(p) = u32x2{pack_bf16x2(a, b), pack_bf16x2(c, d)};
}

// ------------------------------------------------------------------- forward
// Block: 4 waves x 32 queries = 128 queries of one (sequence, head); key tiles
// of 64 up to the block's last query.  Grid: q tiles, heaviest (last) first,
// times sequences x heads (so all q tiles of one head share an XCD's L2).
constexpr int kFwdQ = 128;

__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(2, 2))) void
attn_fwd_kernel(const uint16_t* __restrict__ qkv, uint16_t* __restrict__ o, uint16_t* __restrict__ o_blk,
                float* __restrict__ lse, int S, int Sp, int H, int nbh, float c2) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2][2][kTileElems];  // [stage][K, V]
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int g = lane >> 4, jq = lane & 15;
  const int nqt = (S + kFwdQ - 1) / kFwdQ;
  const int qt = nqt - 1 - (int)(blockIdx.x / nbh);
  const int bh = (int)(blockIdx.x % nbh);
  const int b = bh / H, h = bh % H;
  const int d = H * kHD;
  const int64_t ld = 3 * (int64_t)d;
  const uint16_t* Qb = qkv + (int64_t)b * S * ld + h * kHD;
  const uint16_t* Kb = Qb + d;
  const uint16_t* Vb = Qb + 2 * d;
  const int q0 = qt * kFwdQ;
  const int qw = q0 + 32 * wid;              // this wave's first query
  const int kend = min(S, q0 + kFwdQ);
  const int nkt = (kend + kTR - 1) / kTR;

  auto issue = [&](int kt) {
    load_tile<4>(Kb, ld, kt * kTR, S, lds[kt & 1][0], wid, lane);
    load_tile<4>(Vb, ld, kt * kTR, S, lds[kt & 1][1], wid, lane);
  };
  // Q as the B operand of S^T = K Q^T: query qw + 16 qf + l%16, columns 32 kk + 8 g.
  u32x4 qf[2][4];
#pragma unroll
  for (int f = 0; f < 2; ++f)
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) qf[f][kk] = load_row16(Qb, ld, qw + 16 * f + jq, S, 32 * kk + 8 * g);
  issue(0);

  f32x4 acc_o[8][2];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc_o[i][0] = acc_o[i][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  float mrow[2] = {-INFINITY, -INFINITY}, lsum[2] = {0.f, 0.f};

  for (int kt = 0; kt < nkt; ++kt) {
    wait_vm<0>();
    lds_barrier();  // tile kt is in LDS; every wave is done with tile kt-1's stage
    if (kt + 1 < nkt) issue(kt + 1);
    const int k0 = kt * kTR;
    if (k0 > qw + 31) continue;  // every key of this tile is after every query of this wave
    const uint16_t* Ks = lds[kt & 1][0];
    const uint16_t* Vs = lds[kt & 1][1];
    f32x4 s[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i) s[i][0] = s[i][1] = f32x4{0.f, 0.f, 0.f, 0.f};
    // Reads one batch ahead of the MFMAs: K columns 0..63 (wait), then K
    // columns 64..127 in flight under the first half's MFMAs, then the first V
    // batch in flight under the second half's MFMAs and the softmax.
    u32x4 kf0[8], kf1[8];
    u32x2 vp[8];
    rows_issue(kf0, Ks, 0, lane);
    lds_wait(kf0);
    rows_issue(kf1, Ks, 2, lane);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int f = 0; f < 2; ++f) s[u % 4][f] = mfma(kf0[u], qf[f][u / 4], s[u % 4][f]);
    __builtin_amdgcn_sched_barrier(0);
    lds_wait(kf1);
    cols_issue(vp, Vs, 0, lane);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int f = 0; f < 2; ++f) s[u % 4][f] = mfma(kf1[u], qf[f][2 + u / 4], s[u % 4][f]);
    __builtin_amdgcn_sched_barrier(0);
    // Online softmax per query (lane column); keys 16 i + 4 g + v.  The
    // running max is kept in the base-2 units of s c2 (c2 > 0, and rounding is
    // monotonic, so the max of the products is the product of the max), and
    // p = 2^(s c2 - m) is one fused multiply-add ahead of the exponential.
    // Only a tile reaching past the wave's first query has keys to mask.
    u32x4 pb[2][2];
    const bool diag = k0 + kTR - 1 > qw;
#pragma unroll
    for (int f = 0; f < 2; ++f) {
      const int q = qw + 16 * f + jq;
      if (diag) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            if (k0 + 16 * i + 4 * g + v > q) s[i][f][v] = -INFINITY;
      }
      float tmax = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) tmax = fmaxf(tmax, s[i][f][v]);
      tmax = group_max(tmax);
      const float mnew = fmaxf(mrow[f], tmax * c2);
      const float alpha = exp2_hw(mrow[f] - mnew);
      mrow[f] = mnew;
      float ps = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float p = exp2_hw(fmaf(s[i][f][v], c2, -mnew));
          s[i][f][v] = p;
          ps += p;
        }
      lsum[f] = lsum[f] * alpha + ps;
#pragma unroll
      for (int i = 0; i < 8; ++i) acc_o[i][f] *= alpha;
      pb[f][0] = pack_b(s[0][f], s[1][f]);
      pb[f][1] = pack_b(s[2][f], s[3][f]);
    }
    // O^T += V^T P^T, two head-dim fragments per transposed read batch, the
    // next batch in flight under the current batch's MFMAs.
    u32x4 vf[4];
    cols_finish(vf, vp);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if (c + 1 < 4) cols_issue(vp, Vs, 2 * (c + 1), lane);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int f = 0; f < 2; ++f)
          acc_o[2 * c + (u >> 1)][f] = mfma(vf[u], pb[f][u & 1], acc_o[2 * c + (u >> 1)][f]);
      __builtin_amdgcn_sched_barrier(0);
      if (c + 1 < 4) cols_finish(vf, vp);
    }
  }

  // Normalise and store: lane holds query qw + 16 f + l%16, head columns 16 i + 4 g .. +3.
  uint16_t* Ob = o + (int64_t)b * S * d + h * kHD;
#pragma unroll
  for (int f = 0; f < 2; ++f) {
    const float l = group_sum(lsum[f]);
    const int q = qw + 16 * f + jq;
    if (q < S) {
      const float inv = 1.f / l;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float o0 = acc_o[i][f][0] * inv, o1 = acc_o[i][f][1] * inv, o2 = acc_o[i][f][2] * inv,
                    o3 = acc_o[i][f][3] * inv;
        store4(Ob + (int64_t)q * d + 16 * i + 4 * g, o0, o1, o2, o3);
        if (o_blk) store4(o_blk + blk_off((int64_t)b * S + q, h * kHD + 16 * i + 4 * g, d), o0, o1, o2, o3);
      }
      if (g == 0) lse[(int64_t)bh * Sp + q] = mrow[f] + log2f(l);
    }
  }
}

// ------------------------------------------------------------- delta pre-pass
// delta[b][h][s] = sum over the head's 128 columns of dO * O (float).
__global__ __launch_bounds__(256) void attn_delta_kernel(const uint16_t* __restrict__ dout,
                                                         const uint16_t* __restrict__ o, float* __restrict__ delta,
                                                         int64_t T, int S, int Sp, int H) {
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t row = gid >> 4;  // (token, head)
  const int part = (int)(gid & 15);
  if (row >= T * H) return;
  const int64_t t = row / H;
  const int h = (int)(row % H);
  const int64_t off = t * (int64_t)H * kHD + h * kHD + 8 * part;
  float a[8], c[8];
  Vec<uint16_t>::load(dout + off, a);
  Vec<uint16_t>::load(o + off, c);
  float acc = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) acc = fmaf(a[i], c[i], acc);
#pragma unroll
  for (int m = 1; m < 16; m <<= 1) acc += __shfl_xor(acc, m, 64);
  if (part == 0) {
    const int64_t b = t / S, s = t % S;
    delta[(b * H + h) * Sp + s] = acc;
  }
}

// ------------------------------------------------------------------------ dQ
// Block: 4 waves x 16 queries = 64 queries.  Per key tile:
//   S^T = K Q^T, P^T = 2^(S^T c2 - lse), dP^T = V dO^T, dS^T = P^T (dP^T - delta),
//   dQ^T += K^T dS^T (scaled by 1/sqrt(128) at the end).
constexpr int kDqQ = 64;

__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(2, 2))) void
attn_dq_kernel(const uint16_t* __restrict__ qkv, const uint16_t* __restrict__ dout, const float* __restrict__ lse,
               const float* __restrict__ delta, uint16_t* __restrict__ dqkv, uint16_t* __restrict__ dqkv_blk, int S,
               int Sp, int H, int nbh, float c2, float scale) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2][2][kTileElems];  // [stage][K, V]
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int g = lane >> 4, jq = lane & 15;
  const int nqt = (S + kDqQ - 1) / kDqQ;
  const int qt = nqt - 1 - (int)(blockIdx.x / nbh);
  const int bh = (int)(blockIdx.x % nbh);
  const int b = bh / H, h = bh % H;
  const int d = H * kHD;
  const int64_t ld = 3 * (int64_t)d;
  const uint16_t* Qb = qkv + (int64_t)b * S * ld + h * kHD;
  const uint16_t* Kb = Qb + d;
  const uint16_t* Vb = Qb + 2 * d;
  const uint16_t* dOb = dout + (int64_t)b * S * d + h * kHD;
  const int q0 = qt * kDqQ;
  const int qw = q0 + 16 * wid;
  const int kend = min(S, q0 + kDqQ);
  const int nkt = (kend + kTR - 1) / kTR;

  auto issue = [&](int kt) {
    load_tile<4>(Kb, ld, kt * kTR, S, lds[kt & 1][0], wid, lane);
    load_tile<4>(Vb, ld, kt * kTR, S, lds[kt & 1][1], wid, lane);
  };
  const int q = qw + jq;  // this lane's query
  u32x4 qf[4], dof[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    qf[kk] = load_row16(Qb, ld, q, S, 32 * kk + 8 * g);
    dof[kk] = load_row16(dOb, d, q, S, 32 * kk + 8 * g);
  }
  const float lq = q < S ? lse[(int64_t)bh * Sp + q] : 0.f;
  const float dq_delta = q < S ? delta[(int64_t)bh * Sp + q] : 0.f;
  issue(0);

  f32x4 acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int kt = 0; kt < nkt; ++kt) {
    wait_vm<0>();
    lds_barrier();
    if (kt + 1 < nkt) issue(kt + 1);
    const int k0 = kt * kTR;
    if (k0 > qw + 15) continue;
    const uint16_t* Ks = lds[kt & 1][0];
    const uint16_t* Vs = lds[kt & 1][1];
    f32x4 s[4], dp[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) s[i] = dp[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    // Each batch of fragment reads is in flight under the previous batch's MFMAs.
    u32x4 fr0[8], fr1[8];
    u32x2 cp[8];
    rows_issue(fr0, Ks, 0, lane);
    lds_wait(fr0);
    rows_issue(fr1, Ks, 2, lane);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < 8; ++u) s[u % 4] = mfma(fr0[u], qf[u / 4], s[u % 4]);
    __builtin_amdgcn_sched_barrier(0);
    lds_wait(fr1);
    mfma_src_gap();
    rows_issue(fr0, Vs, 0, lane);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < 8; ++u) s[u % 4] = mfma(fr1[u], qf[2 + u / 4], s[u % 4]);
    __builtin_amdgcn_sched_barrier(0);
    lds_wait(fr0);
    mfma_src_gap();
    rows_issue(fr1, Vs, 2, lane);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < 8; ++u) dp[u % 4] = mfma(fr0[u], dof[u / 4], dp[u % 4]);
    __builtin_amdgcn_sched_barrier(0);
    lds_wait(fr1);
    cols_issue(cp, Ks, 0, lane);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < 8; ++u) dp[u % 4] = mfma(fr1[u], dof[2 + u / 4], dp[u % 4]);
    __builtin_amdgcn_sched_barrier(0);
    u32x4 kt_f[4];
    // dS = P (dP - delta), P = 2^(s c2 - lse); masked entries (a key after
    // the query, or a query past S) only in a tile reaching past the wave's
    // first query or holding the end of the sequence.
    if (k0 + kTR - 1 > qw || qw + 15 >= S) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int key = k0 + 16 * i + 4 * g + v;
          s[i][v] = (key > q || q >= S) ? 0.f : exp2_hw(fmaf(s[i][v], c2, -lq)) * (dp[i][v] - dq_delta);
        }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) s[i][v] = exp2_hw(fmaf(s[i][v], c2, -lq)) * (dp[i][v] - dq_delta);
    }
    const u32x4 ds0 = pack_b(s[0], s[1]), ds1 = pack_b(s[2], s[3]);
    cols_finish(kt_f, cp);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      if (c + 1 < 4) cols_issue(cp, Ks, 2 * (c + 1), lane);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < 4; ++u) acc[2 * c + (u >> 1)] = mfma(kt_f[u], (u & 1) ? ds1 : ds0, acc[2 * c + (u >> 1)]);
      __builtin_amdgcn_sched_barrier(0);
      if (c + 1 < 4) cols_finish(kt_f, cp);
    }
  }
  if (q < S) {
    uint16_t* dQ = dqkv + ((int64_t)b * S + q) * ld + h * kHD;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float v0 = acc[i][0] * scale, v1 = acc[i][1] * scale, v2 = acc[i][2] * scale, v3 = acc[i][3] * scale;
      store4(dQ + 16 * i + 4 * g, v0, v1, v2, v3);
      if (dqkv_blk) store4(dqkv_blk + blk_off((int64_t)b * S + q, h * kHD + 16 * i + 4 * g, ld), v0, v1, v2, v3);
    }
  }
}

// -------------------------------------------------------------------- dK, dV
// Block: 4 waves x 16 keys = 64 keys; query tiles of 64 from the diagonal on.
// Per query tile (rows = queries, lane column = key):
//   S = Q K^T, P = 2^(S c2 - lse), dP = dO V^T, dS = P (dP - delta),
//   dV^T += dO^T P, dK^T += Q^T dS (scaled by 1/sqrt(128) at the end).
// Grid: key blocks in order (the first has the most query tiles).
constexpr int kKvK = 64;

__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(2, 2))) void
attn_dkdv_kernel(const uint16_t* __restrict__ qkv, const uint16_t* __restrict__ dout, const float* __restrict__ lse,
                 const float* __restrict__ delta, uint16_t* __restrict__ dqkv, uint16_t* __restrict__ dqkv_blk, int S,
                 int Sp, int H, int nbh, float c2,
                 float scale) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2][2][kTileElems];  // [stage][Q, dO]
  // [stage][lse (64), delta (64), zeros (128)]: one wave instruction fills a stage
  __shared__ __attribute__((aligned(16))) float stat[2][4 * kTR];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int g = lane >> 4, jk = lane & 15;
  const int kb = (int)(blockIdx.x / nbh);
  const int bh = (int)(blockIdx.x % nbh);
  const int b = bh / H, h = bh % H;
  const int d = H * kHD;
  const int64_t ld = 3 * (int64_t)d;
  const uint16_t* Qb = qkv + (int64_t)b * S * ld + h * kHD;
  const uint16_t* Kb = Qb + d;
  const uint16_t* Vb = Qb + 2 * d;
  const uint16_t* dOb = dout + (int64_t)b * S * d + h * kHD;
  const float* lse_b = lse + (int64_t)bh * Sp;
  const float* del_b = delta + (int64_t)bh * Sp;
  const int k0 = kb * kKvK;
  const int key = k0 + 16 * wid + jk;  // this lane's key
  const int nqt = (S + kTR - 1) / kTR;
  const int qt0 = k0 / kTR;

  // Tiles and statistics of query tile qt; the statistic rows are padded to
  // Sp, so a 16-byte chunk never passes the end of the row.
  auto issue = [&](int qt) {
    load_tile<4>(Qb, ld, qt * kTR, S, lds[qt & 1][0], wid, lane);
    load_tile<4>(dOb, d, qt * kTR, S, lds[qt & 1][1], wid, lane);
    if (wid == 0) {
      const int c = lane & 15;
      const void* src = lane < 16 ? (const void*)(lse_b + qt * kTR + 4 * c)
                                  : lane < 32 ? (const void*)(del_b + qt * kTR + 4 * c) : (const void*)g_zero16;
      dma16(src, reinterpret_cast<uint16_t*>(stat[qt & 1]));
    }
  };
  // K and V as B operands: key column l%16, head columns 32 kk + 8 g.
  u32x4 kf[4], vf[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    kf[kk] = load_row16(Kb, ld, key, S, 32 * kk + 8 * g);
    vf[kk] = load_row16(Vb, ld, key, S, 32 * kk + 8 * g);
  }
  issue(qt0);

  f32x4 dv[8], dk[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) dv[i] = dk[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int qt = qt0; qt < nqt; ++qt) {
    wait_vm<0>();
    lds_barrier();  // tile qt and its statistics are in LDS; tile qt-1's stage is free
    if (qt + 1 < nqt) issue(qt + 1);
    const uint16_t* Qs = lds[qt & 1][0];
    const uint16_t* dOs = lds[qt & 1][1];
    const float* Ls = stat[qt & 1];
    const float* Ds = stat[qt & 1] + kTR;
    const int qbase = qt * kTR;
    f32x4 s[4], dp[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) s[i] = dp[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    // Each batch of fragment reads is in flight under the previous batch's MFMAs.
    u32x4 fr0[8], fr1[8];
    u32x2 cp[8];
    rows_issue(fr0, Qs, 0, lane);
    lds_wait(fr0);
    rows_issue(fr1, Qs, 2, lane);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < 8; ++u) s[u % 4] = mfma(fr0[u], kf[u / 4], s[u % 4]);
    __builtin_amdgcn_sched_barrier(0);
    lds_wait(fr1);
    mfma_src_gap();
    rows_issue(fr0, dOs, 0, lane);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < 8; ++u) s[u % 4] = mfma(fr1[u], kf[2 + u / 4], s[u % 4]);
    __builtin_amdgcn_sched_barrier(0);
    lds_wait(fr0);
    mfma_src_gap();
    rows_issue(fr1, dOs, 2, lane);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < 8; ++u) dp[u % 4] = mfma(fr0[u], vf[u / 4], dp[u % 4]);
    __builtin_amdgcn_sched_barrier(0);
    lds_wait(fr1);
    cols_issue(cp, dOs, 0, lane);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < 8; ++u) dp[u % 4] = mfma(fr1[u], vf[2 + u / 4], dp[u % 4]);
    __builtin_amdgcn_sched_barrier(0);
    // Statistics of queries qbase + 16 i + 4 g .. +3 (asm reads: see lds_ops.h).
    u32x4 st8[8];
    {
      uint32_t a[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = lds_addr(reinterpret_cast<const uint16_t*>(Ls + 16 * i + 4 * g));
        a[4 + i] = lds_addr(reinterpret_cast<const uint16_t*>(Ds + 16 * i + 4 * g));
      }
      Rd128<8>::run(st8, a);
    }
    // Masked entries (a query before the key, or past S, whose statistics
    // are unspecified) only in a tile starting before the wave's last key or
    // holding the end of the sequence.
    if (k0 + 16 * wid + 15 > qbase || qbase + kTR > S) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const f32x4 L4 = __builtin_bit_cast(f32x4, st8[i]);
        const f32x4 D4 = __builtin_bit_cast(f32x4, st8[4 + i]);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int q = qbase + 16 * i + 4 * g + v;
          const bool live = key <= q && q < S;
          const float p = live ? exp2_hw(fmaf(s[i][v], c2, -L4[v])) : 0.f;
          s[i][v] = p;
          dp[i][v] = live ? p * (dp[i][v] - D4[v]) : 0.f;
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const f32x4 L4 = __builtin_bit_cast(f32x4, st8[i]);
        const f32x4 D4 = __builtin_bit_cast(f32x4, st8[4 + i]);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float p = exp2_hw(fmaf(s[i][v], c2, -L4[v]));
          s[i][v] = p;
          dp[i][v] = p * (dp[i][v] - D4[v]);
        }
      }
    }
    const u32x4 p0 = pack_b(s[0], s[1]), p1 = pack_b(s[2], s[3]);
    const u32x4 ds0 = pack_b(dp[0], dp[1]), ds1 = pack_b(dp[2], dp[3]);
    u32x4 tf[4];
    cols_finish(tf, cp);   // dO columns 0..31
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      cols_issue(cp, Qs, 2 * c, lane);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < 4; ++u) dv[2 * c + (u >> 1)] = mfma(tf[u], (u & 1) ? p1 : p0, dv[2 * c + (u >> 1)]);
      __builtin_amdgcn_sched_barrier(0);
      cols_finish(tf, cp);
      if (c + 1 < 4) cols_issue(cp, dOs, 2 * (c + 1), lane);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int u = 0; u < 4; ++u) dk[2 * c + (u >> 1)] = mfma(tf[u], (u & 1) ? ds1 : ds0, dk[2 * c + (u >> 1)]);
      __builtin_amdgcn_sched_barrier(0);
      if (c + 1 < 4) cols_finish(tf, cp);
    }
  }
  if (key < S) {
    uint16_t* row = dqkv + ((int64_t)b * S + key) * ld + h * kHD;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float k0v = dk[i][0] * scale, k1v = dk[i][1] * scale, k2v = dk[i][2] * scale, k3v = dk[i][3] * scale;
      store4(row + d + 16 * i + 4 * g, k0v, k1v, k2v, k3v);
      store4(row + 2 * d + 16 * i + 4 * g, dv[i][0], dv[i][1], dv[i][2], dv[i][3]);
      if (dqkv_blk) {
        const int64_t t = (int64_t)b * S + key;
        const int c = h * kHD + 16 * i + 4 * g;
        store4(dqkv_blk + blk_off(t, d + c, ld), k0v, k1v, k2v, k3v);
        store4(dqkv_blk + blk_off(t, 2 * d + c, ld), dv[i][0], dv[i][1], dv[i][2], dv[i][3]);
      }
    }
  }
}

// ---------------------------------------------------------------- launchers
// qkv/o/dout/dqkv point at the first token of `nseq` whole sequences.
void launch_attn_fwd(const void* qkv, void* o, float* lse, int nseq, int S, int H, hipStream_t s, void* o_blk) {
  if (nseq <= 0 || S <= 0) return;
  const int nbh = nseq * H;
  const int nqt = (S + kFwdQ - 1) / kFwdQ;
  const float c2 = kLog2e / sqrtf((float)kHD);
  hipLaunchKernelGGL(attn_fwd_kernel, dim3((unsigned)(nqt * nbh)), dim3(256), 0, s, (const uint16_t*)qkv,
                     (uint16_t*)o, (uint16_t*)o_blk, lse, S, attn_stat_stride(S), H, nbh, c2);
}

void launch_attn_bwd(const void* qkv, const void* o, const void* dout, const float* lse, float* delta, void* dqkv,
                     int nseq, int S, int H, hipStream_t s, void* dqkv_blk) {
  if (nseq <= 0 || S <= 0) return;
  const int nbh = nseq * H;
  const int64_t T = (int64_t)nseq * S;
  const int64_t nthr = T * H * 16;
  const int Sp = attn_stat_stride(S);
  hipLaunchKernelGGL(attn_delta_kernel, dim3((unsigned)((nthr + 255) / 256)), dim3(256), 0, s,
                     (const uint16_t*)dout, (const uint16_t*)o, delta, T, S, Sp, H);
  const float scale = 1.f / sqrtf((float)kHD);
  const float c2 = kLog2e * scale;
  const int nq = (S + kDqQ - 1) / kDqQ;
  hipLaunchKernelGGL(attn_dq_kernel, dim3((unsigned)(nq * nbh)), dim3(256), 0, s, (const uint16_t*)qkv,
                     (const uint16_t*)dout, lse, delta, (uint16_t*)dqkv, (uint16_t*)dqkv_blk, S, Sp, H, nbh, c2, scale);
  const int nk = (S + kKvK - 1) / kKvK;
  hipLaunchKernelGGL(attn_dkdv_kernel, dim3((unsigned)(nk * nbh)), dim3(256), 0, s, (const uint16_t*)qkv,
                     (const uint16_t*)dout, lse, delta, (uint16_t*)dqkv, (uint16_t*)dqkv_blk, S, Sp, H, nbh, c2, scale);
}

}  // namespace lmoe
