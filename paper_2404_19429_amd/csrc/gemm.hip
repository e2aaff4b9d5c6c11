// Grouped expert GEMMs over the [E][C][*] dispatch layout.
//
// One launch covers every expert (grid z = expert).  Two raggedness modes:
//   ragged-M (forward and dX products): expert e owns buffer rows
//     [rb_e, re_e); C(m, n) = sum_k A(rb_e + m, k) B(k, n) with A row-major
//     (K contiguous).  Tiles past the expert's row count exit at once, so no
//     host read-back of the counts is needed.
//   ragged-K (dW products): C_e = A_e^T B_e reduced over the expert's rows
//     [rb_e, re_e); both operands are row-major in the token dimension, i.e.
//     MN contiguous.  An expert with no rows stores exact zeros.
//
// bf16 path: v_mfma_f32_16x16x32_bf16 with float accumulation.  Tiles are
// staged global -> VGPR -> LDS with one barrier per K step (double buffer);
// operands that are MN-contiguous in memory are transposed in registers
// (8x8 or 4x8 blocks of 16-bit values) while being written to LDS, so every
// LDS tile is K-contiguous and each lane reads its 8-element K run with one
// 16-byte LDS read.  Epilogues: plain store, (H, act(H)) store, and
// dA * act'(H) for the backward.
// f32 path: a plain LDS-tiled FMA GEMM with the same addressing.
#include "internal.h"

namespace lmoe {

enum { EPI_STORE = 0, EPI_FWD1 = 1, EPI_DACT = 2 };

struct GemmParams {
  const void* A;
  int64_t lda, sA;
  const void* B;
  int64_t ldb, sB;
  void* C;
  int64_t ldc, sC;
  void* C2;         // EPI_FWD1: act(acc), same layout as C
  const void* Aux;  // EPI_DACT: pre-activation H, same layout as C
  const int32_t* rb;
  const int32_t* re;
  int M, N, K;      // ragged-M: N, K used;  ragged-K: M, N used
  int act;
  int cap;          // rows per expert block (C): row ranges are clamped to [0, cap]
};

// Row range of group g, clamped to the buffer so bad ranges cannot reach outside it.
__device__ __forceinline__ void group_rows(const GemmParams& p, int g, int& lo, int& span) {
  int a = p.rb ? p.rb[g] : 0;
  int b = p.re[g];
  a = a < 0 ? 0 : (a > p.cap ? p.cap : a);
  b = b < a ? a : (b > p.cap ? p.cap : b);
  lo = a;
  span = b - a;
}

template <typename OutT> __device__ __forceinline__ void store_out(OutT* p, float v);
template <> __device__ __forceinline__ void store_out<uint16_t>(uint16_t* p, float v) { *p = (uint16_t)f32_to_bf16_bits(v); }
template <> __device__ __forceinline__ void store_out<float>(float* p, float v) { *p = v; }
template <typename OutT> __device__ __forceinline__ float load_out(const OutT* p);
template <> __device__ __forceinline__ float load_out<uint16_t>(const uint16_t* p) { return bf16_bits_to_f32(*p); }
template <> __device__ __forceinline__ float load_out<float>(const float* p) { return *p; }

template <int EPI, typename OutT>
__device__ __forceinline__ void epilogue_store(const GemmParams& p, int64_t off, float v) {
  OutT* C = (OutT*)p.C;
  if constexpr (EPI == EPI_FWD1) {
    store_out<OutT>(C + off, v);
    store_out<OutT>((OutT*)p.C2 + off, act_fwd(v, p.act));
  } else if constexpr (EPI == EPI_DACT) {
    const float h = load_out<OutT>((const OutT*)p.Aux + off);
    store_out<OutT>(C + off, v * act_bwd(h, p.act));
  } else {
    store_out<OutT>(C + off, v);
  }
}

// ----------------------------------------------------------------- bf16 MFMA
// Tile loader for an operand whose K dimension is contiguous in memory:
// ROWS (M or N) x BK tile, 16-byte vectors along K.
template <int ROWS, int BK, int NT>
struct LoadKContig {
  static constexpr int KV = BK / 8;
  static constexpr int NV = ROWS * KV / NT;
  static_assert(NV >= 1 && ROWS * KV % NT == 0, "tile/threads mismatch");
  u32x4 v[NV];
  __device__ void load(const uint16_t* base, int64_t ld, int row0, int rowlim, int k0, int klim, int tid) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int q = tid + i * NT;
      const int r = q / KV, kc = q % KV;
      const int row = row0 + r, k = k0 + kc * 8;
      if (row < rowlim && k < klim) v[i] = *reinterpret_cast<const u32x4*>(base + (int64_t)row * ld + k);
      else v[i] = u32x4{0u, 0u, 0u, 0u};
    }
  }
  __device__ void store(uint16_t* lds, int ldk, int tid) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int q = tid + i * NT;
      const int r = q / KV, kc = q % KV;
      *reinterpret_cast<u32x4*>(lds + r * ldk + kc * 8) = v[i];
    }
  }
};

// Tile loader for an operand that is contiguous along M/N: memory row = k.
// Each thread loads R consecutive k rows of 8 MN values and writes the
// transposed 8 x R block as K runs.
template <int COLS, int BK, int NT>
struct LoadMNContig {
  static constexpr int CB = COLS / 8;
  static constexpr int R = ((BK / 8) * CB >= NT) ? 8 : 4;
  static constexpr int NS = (BK / R) * CB / NT;
  static_assert(NS >= 1 && (BK / R) * CB % NT == 0, "tile/threads mismatch");
  u32x4 v[NS][R];
  __device__ void load(const uint16_t* base, int64_t ld, int col0, int collim, int k0, int klim, int tid) {
#pragma unroll
    for (int i = 0; i < NS; ++i) {
      const int q = tid + i * NT;
      const int cb = q % CB, kb = q / CB;
      const int col = col0 + cb * 8;
#pragma unroll
      for (int j = 0; j < R; ++j) {
        const int k = k0 + kb * R + j;
        if (col < collim && k < klim) v[i][j] = *reinterpret_cast<const u32x4*>(base + (int64_t)k * ld + col);
        else v[i][j] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  }
  __device__ void store(uint16_t* lds, int ldk, int tid) const {
#pragma unroll
    for (int i = 0; i < NS; ++i) {
      const int q = tid + i * NT;
      const int cb = q % CB, kb = q / CB;
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        uint32_t o[R / 2];
#pragma unroll
        for (int qq = 0; qq < R / 2; ++qq) {
          const uint32_t lo = v[i][2 * qq][c >> 1], hi = v[i][2 * qq + 1][c >> 1];
          o[qq] = (c & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
        }
        uint16_t* dst = lds + (cb * 8 + c) * ldk + kb * R;
        if constexpr (R == 8) *reinterpret_cast<u32x4*>(dst) = u32x4{o[0], o[1], o[2], o[3]};
        else *reinterpret_cast<u32x2*>(dst) = u32x2{o[0], o[1]};
      }
    }
  }
};

template <int BM, int BN, int BK, int WGM, int WGN, bool B_K, bool RAGGED_K, int EPI, typename OutT>
__global__ __launch_bounds__(WGM* WGN * 64) void gemm_bf16_kernel(GemmParams p) {
  constexpr int NT = WGM * WGN * 64;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  constexpr int LDK = BK + 8;
  static_assert(BK % 32 == 0, "BK must be a multiple of the MFMA K (32)");
  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * LDK];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = tid >> 6;
  const int wm = wid / WGN, wn = wid % WGN;
  const int g = blockIdx.z;
  const int m0 = blockIdx.y * BM;
  const int n0 = blockIdx.x * BN;

  int lo, span;
  group_rows(p, g, lo, span);
  int Mlim, Klim;
  if constexpr (RAGGED_K) {
    Mlim = p.M;
    Klim = span;
  } else {
    Mlim = span;
    Klim = p.K;
    if (m0 >= Mlim) return;
  }

  const uint16_t* Ab;
  const uint16_t* Bb;
  if constexpr (RAGGED_K) {
    Ab = (const uint16_t*)p.A + g * p.sA + (int64_t)lo * p.lda;
    Bb = (const uint16_t*)p.B + g * p.sB + (int64_t)lo * p.ldb;
  } else {
    Ab = (const uint16_t*)p.A + g * p.sA + (int64_t)lo * p.lda;
    Bb = (const uint16_t*)p.B + g * p.sB;
  }

  using ALoader = typename std::conditional<RAGGED_K, LoadMNContig<BM, BK, NT>, LoadKContig<BM, BK, NT>>::type;
  using BLoader = typename std::conditional<B_K && !RAGGED_K, LoadKContig<BN, BK, NT>, LoadMNContig<BN, BK, NT>>::type;
  ALoader la;
  BLoader lb;

  f32x4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = (Klim + BK - 1) / BK;
  if (nk > 0) {
    la.load(Ab, p.lda, m0, Mlim, 0, Klim, tid);
    lb.load(Bb, p.ldb, n0, p.N, 0, Klim, tid);
    la.store(As[0], LDK, tid);
    lb.store(Bs[0], LDK, tid);
    __syncthreads();
  }
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      la.load(Ab, p.lda, m0, Mlim, (kt + 1) * BK, Klim, tid);
      lb.load(Bb, p.ldb, n0, p.N, (kt + 1) * BK, Klim, tid);
    }
    const uint16_t* as = As[cur] + (wm * WTM + (lane & 15)) * LDK + (lane >> 4) * 8;
    const uint16_t* bs = Bs[cur] + (wn * WTN + (lane & 15)) * LDK + (lane >> 4) * 8;
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      bf16x8 af[FM], bfr[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) af[i] = *reinterpret_cast<const bf16x8*>(as + i * 16 * LDK + ks * 32);
#pragma unroll
      for (int j = 0; j < FN; ++j) bfr[j] = *reinterpret_cast<const bf16x8*>(bs + j * 16 * LDK + ks * 32);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      la.store(As[cur ^ 1], LDK, tid);
      lb.store(Bs[cur ^ 1], LDK, tid);
    }
    __syncthreads();
  }

  // Lane holds C[4*(lane/16) + v][lane % 16] of each 16x16 block.
  const int64_t cbase = (int64_t)g * p.sC + (RAGGED_K ? 0 : (int64_t)lo * p.ldc);
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = m0 + wm * WTM + i * 16 + 4 * (lane >> 4) + v;
      if (row >= Mlim) continue;
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int col = n0 + wn * WTN + j * 16 + (lane & 15);
        if (col < p.N) epilogue_store<EPI, OutT>(p, cbase + (int64_t)row * p.ldc + col, acc[i][j][v]);
      }
    }
  }
}

// ------------------------------------------------------------------ f32 path
template <bool B_K, bool RAGGED_K, int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmParams p) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ float As[BK][BM + 4];
  __shared__ float Bs[BK][BN + 4];
  const int tid = threadIdx.x;
  const int tx = tid % 16, ty = tid / 16;
  const int g = blockIdx.z;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  int lo, span;
  group_rows(p, g, lo, span);
  int Mlim, Klim;
  if constexpr (RAGGED_K) {
    Mlim = p.M;
    Klim = span;
  } else {
    Mlim = span;
    Klim = p.K;
    if (m0 >= Mlim) return;
  }
  const float* Ab = (const float*)p.A + g * p.sA + (int64_t)lo * p.lda;
  const float* Bb = (const float*)p.B + g * p.sB + (RAGGED_K ? (int64_t)lo * p.ldb : 0);
  float acc[4][4] = {};
  for (int k0 = 0; k0 < Klim; k0 += BK) {
    for (int i = tid; i < BM * BK; i += 256) {
      int m, k;
      float a = 0.f;
      if constexpr (RAGGED_K) {
        k = i / BM; m = i % BM;
        if (m0 + m < Mlim && k0 + k < Klim) a = Ab[(int64_t)(k0 + k) * p.lda + m0 + m];
      } else {
        m = i / BK; k = i % BK;
        if (m0 + m < Mlim && k0 + k < Klim) a = Ab[(int64_t)(m0 + m) * p.lda + k0 + k];
      }
      As[k][m] = a;
    }
    for (int i = tid; i < BN * BK; i += 256) {
      int n, k;
      float b = 0.f;
      if constexpr (B_K && !RAGGED_K) {
        n = i / BK; k = i % BK;
        if (n0 + n < p.N && k0 + k < Klim) b = Bb[(int64_t)(n0 + n) * p.ldb + k0 + k];
      } else {
        k = i / BN; n = i % BN;
        if (n0 + n < p.N && k0 + k < Klim) b = Bb[(int64_t)(k0 + k) * p.ldb + n0 + n];
      }
      Bs[k][n] = b;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < BK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
  const int64_t cbase = (int64_t)g * p.sC + (RAGGED_K ? 0 : (int64_t)lo * p.ldc);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = m0 + ty * 4 + i;
    if (row >= Mlim) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = n0 + tx * 4 + j;
      if (col < p.N) epilogue_store<EPI, float>(p, cbase + (int64_t)row * p.ldc + col, acc[i][j]);
    }
  }
}

// --------------------------------------------------------------- launchers
constexpr int kBM = 128, kBN = 128, kBK = 64, kWGM = 2, kWGN = 2;

template <bool B_K, bool RAGGED_K, int EPI>
static void run_gemm(const moe_cfg& c, const GemmParams& p, int tilesM, int tilesN, hipStream_t s) {
  if (tilesM <= 0 || tilesN <= 0 || c.E <= 0) return;
  if (c.dtype == MOE_BF16) {
    dim3 grid((unsigned)tilesN, (unsigned)tilesM, (unsigned)c.E);
    hipLaunchKernelGGL((gemm_bf16_kernel<kBM, kBN, kBK, kWGM, kWGN, B_K, RAGGED_K, EPI, uint16_t>), grid,
                       dim3(kWGM * kWGN * 64), 0, s, p);
  } else {
    dim3 grid((unsigned)tilesN, (unsigned)tilesM, (unsigned)c.E);
    hipLaunchKernelGGL((gemm_f32_kernel<B_K, RAGGED_K, EPI>), grid, dim3(256), 0, s, p);
  }
}

static int tile_m(const moe_cfg& c) { return c.dtype == MOE_BF16 ? kBM : 64; }
static int tile_n(const moe_cfg& c) { return c.dtype == MOE_BF16 ? kBN : 64; }
static int cdiv(int64_t a, int b) { return (int)((a + b - 1) / b); }

void launch_expert_fwd(const moe_cfg& c, const void* X, const int32_t* rb, const int32_t* re, const void* W1,
                       const void* W2, void* H, void* A, void* O, hipStream_t s) {
  const int64_t d = c.d_model, f = c.d_ff, C = c.C;
  GemmParams p1{X, d, C * d, W1, d, f * d, H, f, C * f, A, nullptr, rb, re, 0, (int)f, (int)d, c.act, (int)C};
  run_gemm<true, false, EPI_FWD1>(c, p1, cdiv(C, tile_m(c)), cdiv(f, tile_n(c)), s);
  GemmParams p2{A, f, C * f, W2, f, d * f, O, d, C * d, nullptr, nullptr, rb, re, 0, (int)d, (int)f, c.act, (int)C};
  run_gemm<true, false, EPI_STORE>(c, p2, cdiv(C, tile_m(c)), cdiv(d, tile_n(c)), s);
}

void launch_expert_bwd_dx(const moe_cfg& c, const void* dO, const int32_t* rb, const int32_t* re, const void* H,
                          const void* W1, const void* W2, void* dH, void* dXe, hipStream_t s) {
  const int64_t d = c.d_model, f = c.d_ff, C = c.C;
  // dA = dO W2_e  (B(k=i, n=j) = W2[e][i][j], N contiguous), epilogue dH = dA * act'(H)
  GemmParams p1{dO, d, C * d, W2, f, d * f, dH, f, C * f, nullptr, H, rb, re, 0, (int)f, (int)d, c.act, (int)C};
  run_gemm<false, false, EPI_DACT>(c, p1, cdiv(C, tile_m(c)), cdiv(f, tile_n(c)), s);
  // dXe = dH W1_e  (B(k=i, n=j) = W1[e][i][j])
  GemmParams p2{dH, f, C * f, W1, d, f * d, dXe, d, C * d, nullptr, nullptr, rb, re, 0, (int)d, (int)f, c.act, (int)C};
  run_gemm<false, false, EPI_STORE>(c, p2, cdiv(C, tile_m(c)), cdiv(d, tile_n(c)), s);
}

void launch_expert_bwd_dw(const moe_cfg& c, const void* X, const void* A, const void* dO, const void* dH,
                          const int32_t* rb, const int32_t* re, void* dW1, void* dW2, hipStream_t s) {
  const int64_t d = c.d_model, f = c.d_ff, C = c.C;
  // dW2_e [d][f] = dO_e^T A_e : A-operand(m, k) = dO[e][k][m], B(k, n) = A[e][k][n]
  GemmParams p2{dO, d, C * d, A, f, C * f, dW2, f, d * f, nullptr, nullptr, rb, re, (int)d, (int)f, 0, c.act, (int)C};
  run_gemm<false, true, EPI_STORE>(c, p2, cdiv(d, tile_m(c)), cdiv(f, tile_n(c)), s);
  // dW1_e [f][d] = dH_e^T X_e
  GemmParams p1{dH, f, C * f, X, d, C * d, dW1, d, f * d, nullptr, nullptr, rb, re, (int)f, (int)d, 0, c.act, (int)C};
  run_gemm<false, true, EPI_STORE>(c, p1, cdiv(f, tile_m(c)), cdiv(d, tile_n(c)), s);
}

}  // namespace lmoe
