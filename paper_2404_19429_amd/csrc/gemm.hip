// Grouped expert GEMMs over the [E][C][*] dispatch layout.
//
// One launch covers every expert.  Two raggedness modes:
//   ragged-M (forward and dX products): expert e owns buffer rows
//     [rb_e, re_e); C(m, n) = sum_k A(rb_e + m, k) B(k, n) with A row-major
//     (K contiguous).  Tiles past the expert's row count exit at once, so no
//     host read-back of the counts is needed.
//   ragged-K (dW products): C_e = A_e^T B_e reduced over the expert's rows
//     [rb_e, re_e); both operands are row-major in the token dimension, i.e.
//     MN contiguous.  An expert with no rows stores exact zeros.
//
// bf16 path: a persistent kernel with v_mfma_f32_16x16x32_bf16 and float
// accumulation; operand tiles stream global -> LDS asynchronously through a
// multi-stage ring (details below).  Epilogues: plain store, (H, act(H))
// store, dA * act'(H) for the backward, and a residual add.
// The same kernel serves dense products (one group, no row ranges): the
// block's projections and their weight gradients.
// f32 path: a plain LDS-tiled FMA GEMM with the same addressing.
#include "internal.h"
#include "lds_ops.h"

namespace lmoe {

enum { EPI_STORE = 0, EPI_FWD1 = 1, EPI_DACT = 2, EPI_RES = 3 };

struct GemmParams {
  const void* A;
  int64_t lda, sA;
  const void* B;
  int64_t ldb, sB;
  void* C;
  int64_t ldc, sC;
  void* C2;         // EPI_FWD1: act(acc), same layout as C
  const void* Aux;  // EPI_DACT: pre-activation H; EPI_RES: residual added to the product; same layout as C
  const int32_t* rb;
  const int32_t* re;
  int M, N, K;      // ragged-M: N, K used;  ragged-K: M, N used
  int act;
  int cap;          // rows per expert block (C): row ranges are clamped to [0, cap]; re == NULL means [0, cap)
};

// Row range of group g, clamped to the buffer so bad ranges cannot reach outside it.
__device__ __forceinline__ void group_rows(const GemmParams& p, int g, int& lo, int& span) {
  int a = p.rb ? p.rb[g] : 0;
  int b = p.re ? p.re[g] : p.cap;
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
// Operand tiles (BK = 32, one MFMA K step) move global -> LDS with
// global_load_lds_dwordx4 (each lane's 16 bytes land at LDS base + 16 * lane)
// into a STAGES-deep ring.  A lane whose element lies outside the operand
// reads a 16-byte zero page instead, so every wave issues the same number of
// loads per tile and the vmcnt arithmetic below is exact.  Barriers inside the
// K loop are plain s_barrier (with a compiler memory clobber) preceded by an
// explicit s_waitcnt: a full __syncthreads() fence would also drain the loads
// that are meant to stay in flight.
//
// Schedule of iteration kt: wait until tile kt+1 has landed, barrier, refill
// the stage of tile kt (its fragments are already in registers) with tile
// kt+STAGES, read the fragments of tile kt+1, and multiply tile kt.  Loads get
// STAGES-1 iterations to land and fragment reads overlap the MFMAs.
//
// LDS layouts:
//  * K-contiguous operand, ROWS x 32: fragment-linear.  The 16 x 32 MFMA
//    fragment of rows 16f..16f+15 is 1 KB at offset 1 KB * f, lane L's 16
//    bytes (row 16f + L%16, k = 8*(L/16) .. +7) at 16 * L: one DMA instruction
//    fills one fragment and one ds_read_b128 reads it, both linear.
//  * MN-contiguous operand, 32 x COLS (row = k, as in memory): 16-byte chunk c
//    of row k stored at chunk c ^ hsw(k), hsw(k) = 2 * ((k & 3) | ((k >> 3) & 1) << 2).
//    Fragments are read with ds_read_b64_tr_b16: within each 16-lane group,
//    lane j addresses row k0 + j/4, columns n0 + 4*(j%4) .. +3, and receives
//    column n0 + j of rows k0 .. k0+3 -- two such reads give the 8-element K
//    run of the MFMA operand.
constexpr int kBKb = 32;
__device__ __forceinline__ int hsw(int k) { return 2 * ((k & 3) | (((k >> 3) & 1) << 2)); }

// K-contiguous operand: ROWS x 32 tile, one wave instruction fills one fragment.
template <int ROWS, int NW>
struct TileK {
  static constexpr int NI = ROWS / 16 / NW;     // loads per wave per tile
  static_assert(NI >= 1 && ROWS % (16 * NW) == 0, "tile/waves mismatch");
  __device__ static void issue(const uint16_t* base, int64_t ld, int row0, int rowlim, int k0, int klim,
                               uint16_t* stage, int wid, int lane) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int q = i * NW + wid;
      const int row = row0 + 16 * q + (lane & 15), k = k0 + 8 * (lane >> 4);
      const void* src = (row < rowlim && k < klim) ? (const void*)(base + (int64_t)row * ld + k) : (const void*)g_zero16;
      dma16(src, stage + q * 512);
    }
  }
  // Reads FN fragments (rows r0 + 16 j) of one stage, kReadChunk per asm block.
  template <int NF>
  __device__ static void read(u32x4 (&f)[NF], const uint16_t* stage, int r0, int lane) {
    static_assert(NF % 4 == 0, "fragment count");
#pragma unroll
    for (int c = 0; c < NF; c += (NF >= 8 ? 8 : 4)) {
      constexpr int N = NF >= 8 ? 8 : 4;
      uint32_t a[N];
#pragma unroll
      for (int u = 0; u < N; ++u) a[u] = lds_addr(stage + ((r0 >> 4) + c + u) * 512 + lane * 8);
      Rd128<N>::run(&f[c], a);
    }
  }
};

// MN-contiguous operand: 32 x COLS tile (row = k), one wave instruction fills 64 chunks.
template <int COLS, int NW>
struct TileMN {
  static constexpr int CPR = COLS / 8;          // 16-byte chunks per row
  static constexpr int NI = kBKb * CPR / 64 / NW;
  static_assert(NI >= 1 && (kBKb * CPR) % (64 * NW) == 0 && CPR >= 16, "tile/waves mismatch");
  __device__ static void issue(const uint16_t* base, int64_t ld, int col0, int collim, int k0, int klim,
                               uint16_t* stage, int wid, int lane) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int q = i * NW + wid;
      const int L = q * 64 + lane;
      const int k = L / CPR;
      const int lc = (L % CPR) ^ hsw(k);
      const int col = col0 + 8 * lc, kk = k0 + k;
      const void* src = (col < collim && kk < klim) ? (const void*)(base + (int64_t)kk * ld + col) : (const void*)g_zero16;
      dma16(src, stage + q * 512);
    }
  }
  // Reads NF 16 (m or n) x 32 k fragments at columns c0 + 16 j: lane gets column
  // c0 + 16 j + lane%16, k = 8*(lane/16) .. +7 (two transposed reads: k .. k+3, k+4 .. k+7).
  template <int NF>
  __device__ static void read(u32x4 (&f)[NF], const uint16_t* stage, int c0, int lane) {
    static_assert(NF % 4 == 0, "fragment count");
    const int j = lane & 15;
    const int k = 8 * (lane >> 4) + (j >> 2);
    const int h = hsw(k);                                 // hsw(k + 4) == hsw(k)
#pragma unroll
    for (int c = 0; c < NF; c += 4) {
      uint32_t a[8];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int col = c0 + 16 * (c + u) + 4 * (j & 3);
        const int off = k * COLS + (((col >> 3) ^ h) << 3) + (col & 7);
        a[2 * u] = lds_addr(stage + off);
        a[2 * u + 1] = lds_addr(stage + off + 4 * COLS);
      }
      u32x2 o[8];
      RdTr<8>::run(o, a);
#pragma unroll
      for (int u = 0; u < 4; ++u) f[c + u] = u32x4{o[2 * u][0], o[2 * u][1], o[2 * u + 1][0], o[2 * u + 1][1]};
    }
  }
};

// Persistent grouped GEMM: one block per CU walks the list of real tiles of
// all groups.  Tiles are numbered group by group, m-tile by m-tile, n fastest;
// the list is cut into 8 contiguous ranges, one per XCD (workgroups are
// dealt to XCDs round-robin by block index), so the blocks sharing an XCD's
// L2 work on neighbouring tiles that share A rows and B columns.
template <int BM, int BN, int WGM, int WGN, int STAGES, int OCC, bool B_K, bool RAGGED_K, int EPI, int ACT>
__global__ __attribute__((amdgpu_flat_work_group_size(WGM * WGN * 64, WGM * WGN * 64),
                          amdgpu_waves_per_eu(OCC, OCC))) void
gemm_bf16_kernel(GemmParams p, int tilesM, int tilesN, int groups) {
  constexpr int NW = WGM * WGN;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  constexpr int BK = kBKb;
  constexpr int STAGE = (BM + BN) * BK;          // elements per pipeline stage
  constexpr int EPI_LD = WTN + 4;                // fp32 staging row stride
  constexpr int EPI_ROWS = (NW * 32 * EPI_LD * 4 <= STAGES * STAGE * 2) ? 32 : 16;  // rows staged at once
  constexpr bool A_K = !RAGGED_K;
  constexpr bool BK_C = B_K && !RAGGED_K;
  using TA = typename std::conditional<A_K, TileK<BM, NW>, TileMN<BM, NW>>::type;
  using TB = typename std::conditional<BK_C, TileK<BN, NW>, TileMN<BN, NW>>::type;
  constexpr int LPS = TA::NI + TB::NI;           // loads per wave per stage
  static_assert(STAGES >= 2 && LPS * (STAGES - 1) < 64, "vmcnt range");
  static_assert(WTM % EPI_ROWS == 0, "wave tile rows must be a multiple of the staged slice");
  static_assert(NW * EPI_ROWS * EPI_LD * 4 <= STAGES * STAGE * 2, "epilogue staging does not fit");
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  __shared__ int s_prefix[kMaxE + 1];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wid = tid >> 6;
  const int wm = wid / WGN, wn = wid % WGN;

  // Tile counts per group -> exclusive prefix (one wave, groups <= 64).
  if (wid == 0) {
    int cnt = 0;
    if (lane < groups) {
      if constexpr (RAGGED_K) {
        cnt = tilesM * tilesN;
      } else {
        int lo, span;
        group_rows(p, lane, lo, span);
        cnt = ((span + BM - 1) / BM) * tilesN;
      }
    }
    int incl = cnt;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int u = __shfl_up(incl, o, 64);
      if (lane >= o) incl += u;
    }
    if (lane < groups) s_prefix[lane + 1] = incl;
    if (lane == 0) s_prefix[0] = 0;
  }
  __syncthreads();
  const int total = s_prefix[groups];
  const int nslot = gridDim.x / 8;
  const int xcd = blockIdx.x % 8, slot = blockIdx.x / 8;
  const int per = (total + 7) / 8;
  const int t_begin = xcd * per + slot;
  const int t_end = min(total, (xcd + 1) * per);

  for (int t = t_begin; t < t_end; t += nslot) {
    int g = 0;
    while (g + 1 < groups && s_prefix[g + 1] <= t) ++g;
    const int local = t - s_prefix[g];
    const int m0 = (local / tilesN) * BM;
    const int n0 = (local % tilesN) * BN;
    int lo, span;
    group_rows(p, g, lo, span);
    const int Mlim = RAGGED_K ? p.M : span;
    const int Klim = RAGGED_K ? span : p.K;
    const uint16_t* Ab = (const uint16_t*)p.A + g * p.sA + (int64_t)lo * p.lda;
    const uint16_t* Bb = (const uint16_t*)p.B + g * p.sB + (RAGGED_K ? (int64_t)lo * p.ldb : 0);

    f32x4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nk = (Klim + BK - 1) / BK;
    auto issue = [&](int kt) {
      uint16_t* st = lds + (kt % STAGES) * STAGE;
      TA::issue(Ab, p.lda, m0, Mlim, kt * BK, Klim, st, wid, lane);
      TB::issue(Bb, p.ldb, n0, p.N, kt * BK, Klim, st + BM * BK, wid, lane);
    };
    // Fragment reads of one tile: the A fragments, then the B fragments, each in
    // asm blocks of at most kReadChunk reads that complete before they return.
    auto read_a = [&](int kt, u32x4 (&fa)[FM]) {
      TA::template read<FM>(fa, lds + (kt % STAGES) * STAGE, wm * WTM, lane);
    };
    auto read_b = [&](int kt, u32x4 (&fb)[FN]) {
      TB::template read<FN>(fb, lds + (kt % STAGES) * STAGE + BM * BK, wn * WTN, lane);
    };
    auto mfma_rows = [&](int i0, int i1, u32x4 (&ca)[FM], u32x4 (&cb)[FN]) {
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        if (i < i0 || i >= i1) continue;
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ca[i]),
                                                              __builtin_bit_cast(bf16x8, cb[j]), acc[i][j], 0, 0, 0);
      }
    };
    // One K step: multiply tile kt (fragments in ca/cb) in two halves; the
    // fragments of tile kt+1 are read into na/nb before each half, so the read
    // latency overlaps the MFMAs already in the pipe.  Called with the two
    // register sets in alternating roles (static indexing).
    auto step = [&](int kt, u32x4 (&ca)[FM], u32x4 (&cb)[FN], u32x4 (&na)[FM], u32x4 (&nb)[FN]) {
      const bool more = kt + 1 < nk;
      if (more) {
        // tile kt+1 has landed once only tiles kt+2 .. min(kt+STAGES-1, nk-1) are pending
        wait_vm_tiles<LPS, STAGES - 2>(min(STAGES - 2, nk - 2 - kt));
        lds_barrier();  // tile kt+1 is in LDS for every wave; no wave reads tile kt's stage any more
        if (kt + STAGES < nk) issue(kt + STAGES);
        read_a(kt + 1, na);
      }
      __builtin_amdgcn_sched_barrier(0);
      mfma_rows(0, FM / 2, ca, cb);
      __builtin_amdgcn_sched_barrier(0);
      if (more) read_b(kt + 1, nb);
      __builtin_amdgcn_sched_barrier(0);
      mfma_rows(FM / 2, FM, ca, cb);
      __builtin_amdgcn_sched_barrier(0);
    };

    u32x4 fa0[FM], fb0[FN], fa1[FM], fb1[FN];
    if (nk > 0) {
#pragma unroll
      for (int s = 0; s < STAGES; ++s)
        if (s < nk) issue(s);
      wait_vm_tiles<LPS, STAGES - 1>(min(STAGES - 1, nk - 1));  // tile 0 has landed
      lds_barrier();
      read_a(0, fa0);
      read_b(0, fb0);
    }
    for (int kt = 0; kt < nk; kt += 2) {
      step(kt, fa0, fb0, fa1, fb1);
      if (kt + 1 < nk) step(kt + 1, fa1, fb1, fa0, fb0);
    }
    wait_vm<0>();
    lds_barrier();  // all waves are done reading the operand stages

    // Epilogue: stage 32-row slices of the wave tile through LDS as float,
    // then write 16-byte vectors (8 bf16) with the epilogue applied.
    float* st = reinterpret_cast<float*>(lds) + wid * (EPI_ROWS * EPI_LD);
    uint16_t* C = (uint16_t*)p.C + (int64_t)g * p.sC + (RAGGED_K ? 0 : (int64_t)lo * p.ldc);
    uint16_t* C2 = EPI == EPI_FWD1 ? (uint16_t*)p.C2 + (int64_t)g * p.sC + (int64_t)lo * p.ldc : nullptr;
    const uint16_t* Aux = (EPI == EPI_DACT || EPI == EPI_RES)
                              ? (const uint16_t*)p.Aux + (int64_t)g * p.sC + (int64_t)lo * p.ldc : nullptr;
    const int g4 = lane >> 4;
#pragma unroll
    for (int pass = 0; pass < WTM / EPI_ROWS; ++pass) {
#pragma unroll
      for (int ii = 0; ii < EPI_ROWS / 16; ++ii) {
        const int i = pass * (EPI_ROWS / 16) + ii;
#pragma unroll
        for (int j = 0; j < FN; ++j)
#pragma unroll
          for (int v = 0; v < 4; ++v) st[(ii * 16 + 4 * g4 + v) * EPI_LD + j * 16 + (lane & 15)] = acc[i][j][v];
      }
      // The staging slice is private to this wave and LDS executes a wave's
      // accesses in order, so no barrier is needed between writes and reads.
      constexpr int CPR = WTN / 8;          // 8-column chunks per row
#pragma unroll
      for (int q = lane; q < EPI_ROWS * CPR; q += 64) {
        const int rr = q / CPR, cc = q % CPR;
        const int row = m0 + wm * WTM + pass * EPI_ROWS + rr;
        const int col = n0 + wn * WTN + cc * 8;
        if (row < Mlim && col < p.N) {
          float v[8];
          const f32x4 a = *reinterpret_cast<const f32x4*>(st + rr * EPI_LD + cc * 8);
          const f32x4 b = *reinterpret_cast<const f32x4*>(st + rr * EPI_LD + cc * 8 + 4);
#pragma unroll
          for (int u = 0; u < 4; ++u) { v[u] = a[u]; v[4 + u] = b[u]; }
          const int64_t off = (int64_t)row * p.ldc + col;
          if constexpr (EPI == EPI_FWD1) {
            Vec<uint16_t>::store(C + off, v);
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = act_fwd_t<ACT>(v[u]);
            Vec<uint16_t>::store(C2 + off, v);
          } else if constexpr (EPI == EPI_DACT) {
            float h[8];
            Vec<uint16_t>::load(Aux + off, h);
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] *= act_bwd_t<ACT>(h[u]);
            Vec<uint16_t>::store(C + off, v);
          } else if constexpr (EPI == EPI_RES) {
            float r[8];
            Vec<uint16_t>::load(Aux + off, r);
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] += r[u];
            Vec<uint16_t>::store(C + off, v);
          } else {
            Vec<uint16_t>::store(C + off, v);
          }
        }
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    lds_barrier();  // every wave is done with its staging slice before the next tile's loads land
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
// Tile shape, LDS stages and resident blocks per CU (OCC) of the bf16 kernel.
#ifndef LMOE_GEMM_TILE
#define LMOE_GEMM_TILE 128, 128, 2, 2, 4, 2
#endif
template <int BM_, int BN_, int WGM_, int WGN_, int STAGES_, int OCC_> struct TileCfg {
  static constexpr int BM = BM_, BN = BN_, WGM = WGM_, WGN = WGN_, STAGES = STAGES_, OCC = OCC_;
};
using Tile = TileCfg<LMOE_GEMM_TILE>;
constexpr int kBM = Tile::BM, kBN = Tile::BN;

static int num_cus() {
  static int n = 0;
  if (n == 0) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
  }
  return n;
}

template <bool B_K, bool RAGGED_K, int EPI, int ACT>
static void launch_bf16(int groups, const GemmParams& p, int tilesM, int tilesN, hipStream_t s) {
  constexpr int NT = Tile::WGM * Tile::WGN * 64;
  constexpr size_t shmem = Tile::STAGES * (size_t)(Tile::BM + Tile::BN) * kBKb * sizeof(uint16_t);
  auto kern = gemm_bf16_kernel<Tile::BM, Tile::BN, Tile::WGM, Tile::WGN, Tile::STAGES, Tile::OCC, B_K, RAGGED_K, EPI, ACT>;
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shmem);
    attr_set = true;
  }
  const int64_t max_tiles = (int64_t)tilesM * tilesN * groups;
  int blocks = num_cus() * Tile::OCC;
  if (max_tiles < blocks) blocks = (int)((max_tiles + 7) / 8 * 8);
  blocks = (blocks + 7) / 8 * 8;
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(NT), shmem, s, p, tilesM, tilesN, groups);
}

// groups: experts (or 1 for a dense product); dtype/act as in moe_cfg.
template <bool B_K, bool RAGGED_K, int EPI>
static void run_gemm(int dtype, int act, int groups, const GemmParams& p, int tilesM, int tilesN, hipStream_t s) {
  if (tilesM <= 0 || tilesN <= 0 || groups <= 0) return;
  if (dtype == MOE_BF16) {
    if constexpr (EPI == EPI_STORE || EPI == EPI_RES) {
      launch_bf16<B_K, RAGGED_K, EPI, MOE_ACT_IDENTITY>(groups, p, tilesM, tilesN, s);
    } else {
      switch (act) {
        case MOE_ACT_RELU: launch_bf16<B_K, RAGGED_K, EPI, MOE_ACT_RELU>(groups, p, tilesM, tilesN, s); break;
        case MOE_ACT_GELU_TANH: launch_bf16<B_K, RAGGED_K, EPI, MOE_ACT_GELU_TANH>(groups, p, tilesM, tilesN, s); break;
        case MOE_ACT_GELU_ERF: launch_bf16<B_K, RAGGED_K, EPI, MOE_ACT_GELU_ERF>(groups, p, tilesM, tilesN, s); break;
        default: launch_bf16<B_K, RAGGED_K, EPI, MOE_ACT_IDENTITY>(groups, p, tilesM, tilesN, s); break;
      }
    }
  } else {
    if constexpr (EPI != EPI_RES) {
      dim3 grid((unsigned)tilesN, (unsigned)tilesM, (unsigned)groups);
      hipLaunchKernelGGL((gemm_f32_kernel<B_K, RAGGED_K, EPI>), grid, dim3(256), 0, s, p);
    }
  }
}

template <bool B_K, bool RAGGED_K, int EPI>
static void run_gemm(const moe_cfg& c, const GemmParams& p, int tilesM, int tilesN, hipStream_t s) {
  run_gemm<B_K, RAGGED_K, EPI>(c.dtype, c.act, c.E, p, tilesM, tilesN, s);
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

// Dense bf16 products of the transformer block (one group, every row).
void launch_dense(int64_t M, int N, int K, const void* A, int64_t lda, const void* B, int64_t ldb, bool b_nk,
                  void* C, int64_t ldc, const void* resid, hipStream_t s) {
  GemmParams p{A, lda, 0, B, ldb, 0, C, ldc, 0, nullptr, resid, nullptr, nullptr, 0, N, K, 0, (int)M};
  const int tm = cdiv(M, kBM), tn = cdiv(N, kBN);
  if (b_nk) {
    if (resid) run_gemm<true, false, EPI_RES>(MOE_BF16, 0, 1, p, tm, tn, s);
    else run_gemm<true, false, EPI_STORE>(MOE_BF16, 0, 1, p, tm, tn, s);
  } else {
    if (resid) run_gemm<false, false, EPI_RES>(MOE_BF16, 0, 1, p, tm, tn, s);
    else run_gemm<false, false, EPI_STORE>(MOE_BF16, 0, 1, p, tm, tn, s);
  }
}

void launch_dense_wgrad(int M, int N, int64_t K, const void* A, int64_t lda, const void* B, int64_t ldb, void* C,
                        int64_t ldc, hipStream_t s) {
  GemmParams p{A, lda, 0, B, ldb, 0, C, ldc, 0, nullptr, nullptr, nullptr, nullptr, M, N, 0, 0, (int)K};
  run_gemm<false, true, EPI_STORE>(MOE_BF16, 0, 1, p, cdiv(M, kBM), cdiv(N, kBN), s);
}

}  // namespace lmoe
