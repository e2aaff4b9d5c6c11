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
// BLK: the operand is stored in 16 x 32 blocks; a fragment is one block.
template <int ROWS, int NW, bool BLK>
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
  // Blocked source: row0 (a multiple of 16) is the fragment's first row in
  // the operand, rows at or past rowlim read zeros.  Lane l takes (row l%16,
  // k chunk l/16) of the block, which is its fragment-linear LDS position.
  __device__ static void issue_blk(const uint16_t* base, int64_t ld, int row0, int rowlim, int k0, int klim,
                                   uint16_t* stage, int wid, int lane) {
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int q = i * NW + wid;
      const int rb = (row0 >> 4) + q;
      const int row = 16 * rb + (lane & 15);
      const void* src = (row < rowlim && k0 < klim)
                            ? (const void*)(base + ((int64_t)rb * (ld >> 5) + (k0 >> 5)) * 512 + (lane & 15) * 32 +
                                            (lane >> 4) * 8)
                            : (const void*)g_zero16;
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
  // Split form (NF = 4 or 8): start the reads, later complete them in place.
  template <int NF>
  __device__ static void read_issue(u32x4 (&f)[NF], u32x2 (&)[8], const uint16_t* stage, int r0, int lane) {
    static_assert(NF == 4 || NF == 8, "split reads: 4 or 8 fragments");
    uint32_t a[NF];
#pragma unroll
    for (int u = 0; u < NF; ++u) a[u] = lds_addr(stage + ((r0 >> 4) + u) * 512 + lane * 8);
    Rd128Issue<NF>::run(f, a);
  }
  template <int NF>
  __device__ static void read_finish(u32x4 (&f)[NF], u32x2 (&)[8]) { lds_wait(f); }
};

// MN-contiguous operand: 32 x COLS tile (row = k), one wave instruction fills 64 chunks.
// BLK: the operand is stored in 16 x 32 blocks and the stage keeps them as
// [2][COLS/32] blocks of 16 rows x 4 chunks, chunk c of block row r at c ^ bsw(r):
// the 16 lanes of a transposed read cover rows r..r+3 and the next lane group
// rows r+8..r+11, and this swizzle puts those 8 x 32 bytes on distinct banks.
__device__ __forceinline__ int bsw(int r) { return 2 * (((r >> 1) ^ (r >> 3)) & 1); }
template <int COLS, int NW, bool BLK>
struct TileMN {
  static constexpr int CB = COLS / 32;          // column blocks per stage
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
  // Blocked source: k0 (a multiple of 16) is the stage's first row in the
  // operand; rows outside [klo, khi) and column blocks at or past collim read zeros.
  __device__ static void issue_blk(const uint16_t* base, int64_t ld, int col0, int collim, int k0, int klo, int khi,
                                   uint16_t* stage, int wid, int lane) {
    const int r = lane >> 2;
    const int c = (lane & 3) ^ bsw(r);
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int b = i * NW + wid;
      const int kb = b / CB, cb = b % CB;
      const int krow = k0 + 16 * kb + r;
      const int col = col0 + 32 * cb;
      const void* src = (krow >= klo && krow < khi && col < collim)
                            ? (const void*)(base + ((int64_t)((k0 >> 4) + kb) * (ld >> 5) + (col >> 5)) * 512 +
                                            r * 32 + c * 8)
                            : (const void*)g_zero16;
      dma16(src, stage + b * 512);
    }
  }
  // LDS element offset of (k, col) in a stage.
  __device__ static int lds_off(int k, int col) {
    if constexpr (BLK) {
      const int r = k & 15;
      return ((k >> 4) * CB + (col >> 5)) * 512 + r * 32 + ((((col & 31) >> 3) ^ bsw(r)) << 3) + (col & 7);
    } else {
      return k * COLS + (((col >> 3) ^ hsw(k)) << 3) + (col & 7);
    }
  }
  // Reads NF 16 (m or n) x 32 k fragments at columns c0 + 16 j: lane gets column
  // c0 + 16 j + lane%16, k = 8*(lane/16) .. +7 (two transposed reads: k .. k+3, k+4 .. k+7).
  template <int NF>
  __device__ static void read(u32x4 (&f)[NF], const uint16_t* stage, int c0, int lane) {
    static_assert(NF % 4 == 0, "fragment count");
    const int j = lane & 15;
    const int k = 8 * (lane >> 4) + (j >> 2);
#pragma unroll
    for (int c = 0; c < NF; c += 4) {
      uint32_t a[8];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int col = c0 + 16 * (c + u) + 4 * (j & 3);
        a[2 * u] = lds_addr(stage + lds_off(k, col));
        a[2 * u + 1] = lds_addr(stage + lds_off(k + 4, col));
      }
      u32x2 o[8];
      RdTr<8>::run(o, a);
#pragma unroll
      for (int u = 0; u < 4; ++u) f[c + u] = u32x4{o[2 * u][0], o[2 * u][1], o[2 * u + 1][0], o[2 * u + 1][1]};
    }
  }
  // Split form (NF = 4): the 8 transposed reads land in p; read_finish waits and assembles.
  template <int NF>
  __device__ static void read_issue(u32x4 (&)[NF], u32x2 (&p)[8], const uint16_t* stage, int c0, int lane) {
    static_assert(NF == 4, "split transposed reads: 4 fragments");
    const int j = lane & 15;
    const int k = 8 * (lane >> 4) + (j >> 2);
    uint32_t a[8];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int col = c0 + 16 * u + 4 * (j & 3);
      a[2 * u] = lds_addr(stage + lds_off(k, col));
      a[2 * u + 1] = lds_addr(stage + lds_off(k + 4, col));
    }
    RdTrIssue8::run(p, a);
  }
  template <int NF>
  __device__ static void read_finish(u32x4 (&f)[NF], u32x2 (&p)[8]) {
    lds_wait(p);
#pragma unroll
    for (int u = 0; u < 4; ++u) f[u] = u32x4{p[2 * u][0], p[2 * u][1], p[2 * u + 1][0], p[2 * u + 1][1]};
  }
};

// Persistent grouped GEMM: resident blocks walk the list of real tiles of all
// groups.  Within a group, tiles are numbered panel by panel (kPanelN tile
// columns wide), m-tile by m-tile inside a panel, n fastest.  The list is cut
// into 8 contiguous ranges, one per XCD (workgroups are dealt to XCDs
// round-robin by block index), so the ~64 tiles an XCD has in flight form an
// 8 x 8 patch: each A row-slice and B column-slice it streams is shared by 8
// tiles through that XCD's L2, instead of one A slice shared by a whole row of
// tiles while every B slice of the row is fetched afresh.
#ifndef LMOE_SPLIT_READS
#define LMOE_SPLIT_READS 1
#endif
#ifndef LMOE_PANEL_N
#define LMOE_PANEL_N 8
#endif
constexpr int kPanelN = LMOE_PANEL_N;
// BLK: both operands in 16 x 32 blocks (expert buffers and packed weights),
// ragged row ranges start at the block row containing row_begin; CBLK: the
// output (and the epilogue's auxiliary input) too.  Otherwise row-major.
template <int BM, int BN, int WGM, int WGN, int STAGES, int OCC, bool B_K, bool RAGGED_K, int EPI, int ACT, bool BLK,
          bool CBLK>
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
  using TA = typename std::conditional<A_K, TileK<BM, NW, BLK>, TileMN<BM, NW, BLK>>::type;
  using TB = typename std::conditional<BK_C, TileK<BN, NW, BLK>, TileMN<BN, NW, BLK>>::type;
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
        if (BLK && span > 0) span += lo & 15;  // tiles start at the block row holding row_begin
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
    int lo, span;
    group_rows(p, g, lo, span);
    const int hi = lo + span;
    const int lo_al = BLK ? (lo & ~15) : lo;   // row (or K) origin of this group's tiles
    if (BLK && span > 0) span += lo - lo_al;
    // Panel order: n-panels of kPanelN tile columns, m-tiles within a panel,
    // n fastest, so the tiles in flight on one XCD form a square-ish patch.
    const int tmg = RAGGED_K ? tilesM : (span + BM - 1) / BM;
    const int pnl = local / (tmg * kPanelN);
    const int rem = local - pnl * tmg * kPanelN;
    const int pw = min(kPanelN, tilesN - pnl * kPanelN);
    const int m0 = (rem / pw) * BM;
    const int n0 = (pnl * kPanelN + rem % pw) * BN;
    const int Mlim = RAGGED_K ? p.M : span;
    const int Klim = RAGGED_K ? span : p.K;
    const uint16_t* Ab = (const uint16_t*)p.A + g * p.sA + (BLK ? 0 : (int64_t)lo * p.lda);
    const uint16_t* Bb = (const uint16_t*)p.B + g * p.sB + (RAGGED_K && !BLK ? (int64_t)lo * p.ldb : 0);

    f32x4 acc[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nk = (Klim + BK - 1) / BK;
    auto issue = [&](int kt) {
      uint16_t* st = lds + (kt % STAGES) * STAGE;
      if constexpr (!BLK) {
        TA::issue(Ab, p.lda, m0, Mlim, kt * BK, Klim, st, wid, lane);
        TB::issue(Bb, p.ldb, n0, p.N, kt * BK, Klim, st + BM * BK, wid, lane);
      } else {
        if constexpr (A_K) TA::issue_blk(Ab, p.lda, lo_al + m0, (int)pad16(p.cap), kt * BK, Klim, st, wid, lane);
        else TA::issue_blk(Ab, p.lda, m0, p.M, lo_al + kt * BK, lo, hi, st, wid, lane);
        if constexpr (BK_C) TB::issue_blk(Bb, p.ldb, n0, p.N, kt * BK, Klim, st + BM * BK, wid, lane);
        else if constexpr (RAGGED_K) TB::issue_blk(Bb, p.ldb, n0, p.N, lo_al + kt * BK, lo, hi, st + BM * BK, wid, lane);
        else TB::issue_blk(Bb, p.ldb, n0, p.N, kt * BK, 0, p.K, st + BM * BK, wid, lane);
      }
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
    // With split reads the fragment reads of tile kt+1 are started before a
    // half of tile kt's MFMAs and completed after it, so their latency hides
    // under those MFMAs.
    constexpr bool kSplit = LMOE_SPLIT_READS && (A_K ? (FM == 4 || FM == 8) : FM == 4) &&
                            (BK_C ? (FN == 4 || FN == 8) : FN == 4);
    u32x2 pa[8], pb[8];
    auto step = [&](int kt, u32x4 (&ca)[FM], u32x4 (&cb)[FN], u32x4 (&na)[FM], u32x4 (&nb)[FN]) {
      const bool more = kt + 1 < nk;
      const uint16_t* st = lds + ((kt + 1) % STAGES) * STAGE;
      if (more) {
        // tile kt+1 has landed once only tiles kt+2 .. min(kt+STAGES-1, nk-1) are pending
        wait_vm_tiles<LPS, STAGES - 2>(min(STAGES - 2, nk - 2 - kt));
        lds_barrier();  // tile kt+1 is in LDS for every wave; no wave reads tile kt's stage any more
        if (kt + STAGES < nk) issue(kt + STAGES);
      }
      // Split reads are unconditional (branch-free, so the pending registers
      // are never copied): after the last tile they read a stale stage that
      // no load is writing, and the values are discarded.
      if constexpr (kSplit) TA::template read_issue<FM>(na, pa, st, wm * WTM, lane);
      else if (more) read_a(kt + 1, na);
      __builtin_amdgcn_sched_barrier(0);
      mfma_rows(0, FM / 2, ca, cb);
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (kSplit) {
        TA::template read_finish<FM>(na, pa);
        TB::template read_issue<FN>(nb, pb, st + BM * BK, wn * WTN, lane);
      } else if (more) {
        read_b(kt + 1, nb);
      }
      __builtin_amdgcn_sched_barrier(0);
      mfma_rows(FM / 2, FM, ca, cb);
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (kSplit) {
        TB::template read_finish<FN>(nb, pb);
        __builtin_amdgcn_sched_barrier(0);
      }
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
    // Output rows are relative to lo_al; a row-major output starts at row lo_al.
    const int64_t cofs = (int64_t)g * p.sC + (RAGGED_K || CBLK ? 0 : (int64_t)lo_al * p.ldc);
    uint16_t* C = (uint16_t*)p.C + cofs;
    uint16_t* C2 = EPI == EPI_FWD1 ? (uint16_t*)p.C2 + cofs : nullptr;
    const uint16_t* Aux = (EPI == EPI_DACT || EPI == EPI_RES) ? (const uint16_t*)p.Aux + cofs : nullptr;
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
        if (row < Mlim && col < p.N && (RAGGED_K || lo_al + row >= lo)) {
          float v[8];
          const f32x4 a = *reinterpret_cast<const f32x4*>(st + rr * EPI_LD + cc * 8);
          const f32x4 b = *reinterpret_cast<const f32x4*>(st + rr * EPI_LD + cc * 8 + 4);
#pragma unroll
          for (int u = 0; u < 4; ++u) { v[u] = a[u]; v[4 + u] = b[u]; }
          const int64_t off = CBLK ? blk_off(lo_al + row, col, p.ldc) : (int64_t)row * p.ldc + col;
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

template <bool B_K, bool RAGGED_K, int EPI, int ACT, bool BLK, bool CBLK>
static void launch_bf16(int groups, const GemmParams& p, int tilesM, int tilesN, hipStream_t s) {
  constexpr int NT = Tile::WGM * Tile::WGN * 64;
  constexpr size_t shmem = Tile::STAGES * (size_t)(Tile::BM + Tile::BN) * kBKb * sizeof(uint16_t);
  auto kern = gemm_bf16_kernel<Tile::BM, Tile::BN, Tile::WGM, Tile::WGN, Tile::STAGES, Tile::OCC, B_K, RAGGED_K, EPI,
                               ACT, BLK, CBLK>;
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

// groups: experts (or 1 for a dense product); dtype/act as in moe_cfg.  BLK,
// CBLK (bf16 only): operands / output in the blocked layout.
template <bool B_K, bool RAGGED_K, int EPI, bool BLK = false, bool CBLK = false>
static void run_gemm(int dtype, int act, int groups, const GemmParams& p, int tilesM, int tilesN, hipStream_t s) {
  if (tilesM <= 0 || tilesN <= 0 || groups <= 0) return;
  if (dtype == MOE_BF16) {
    if constexpr (EPI == EPI_STORE || EPI == EPI_RES) {
      launch_bf16<B_K, RAGGED_K, EPI, MOE_ACT_IDENTITY, BLK, CBLK>(groups, p, tilesM, tilesN, s);
    } else {
      switch (act) {
        case MOE_ACT_RELU: launch_bf16<B_K, RAGGED_K, EPI, MOE_ACT_RELU, BLK, CBLK>(groups, p, tilesM, tilesN, s); break;
        case MOE_ACT_GELU_TANH:
          launch_bf16<B_K, RAGGED_K, EPI, MOE_ACT_GELU_TANH, BLK, CBLK>(groups, p, tilesM, tilesN, s);
          break;
        case MOE_ACT_GELU_ERF:
          launch_bf16<B_K, RAGGED_K, EPI, MOE_ACT_GELU_ERF, BLK, CBLK>(groups, p, tilesM, tilesN, s);
          break;
        default: launch_bf16<B_K, RAGGED_K, EPI, MOE_ACT_IDENTITY, BLK, CBLK>(groups, p, tilesM, tilesN, s); break;
      }
    }
  } else {
    if constexpr (EPI != EPI_RES) {
      dim3 grid((unsigned)tilesN, (unsigned)tilesM, (unsigned)groups);
      hipLaunchKernelGGL((gemm_f32_kernel<B_K, RAGGED_K, EPI>), grid, dim3(256), 0, s, p);
    }
  }
}

// Expert products: bf16 operands and outputs in the blocked layout (dW outputs
// row-major), float ones row-major.
template <bool B_K, bool RAGGED_K, int EPI, bool CBLK>
static void run_expert(const moe_cfg& c, const GemmParams& p, int tilesM, int tilesN, hipStream_t s) {
  run_gemm<B_K, RAGGED_K, EPI, true, CBLK>(c.dtype, c.act, c.E, p, tilesM, tilesN, s);
}

static int tile_m(const moe_cfg& c) { return c.dtype == MOE_BF16 ? kBM : 64; }
static int tile_n(const moe_cfg& c) { return c.dtype == MOE_BF16 ? kBN : 64; }
static int cdiv(int64_t a, int b) { return (int)((a + b - 1) / b); }
// Rows per expert block of an [E][C][*] buffer (C rounded up to 16 for bf16).
static int64_t rows_alloc(const moe_cfg& c) { return c.dtype == MOE_BF16 ? pad16(c.C) : c.C; }

void launch_expert_fwd(const moe_cfg& c, const void* X, const int32_t* rb, const int32_t* re, const void* W1,
                       const void* W2, void* H, void* A, void* O, hipStream_t s) {
  const int64_t d = c.d_model, f = c.d_ff, C = c.C, Cp = rows_alloc(c);
  const int tm = cdiv(C + 15, tile_m(c));
  GemmParams p1{X, d, Cp * d, W1, d, f * d, H, f, Cp * f, A, nullptr, rb, re, 0, (int)f, (int)d, c.act, (int)C};
  run_expert<true, false, EPI_FWD1, true>(c, p1, tm, cdiv(f, tile_n(c)), s);
  GemmParams p2{A, f, Cp * f, W2, f, d * f, O, d, Cp * d, nullptr, nullptr, rb, re, 0, (int)d, (int)f, c.act, (int)C};
  run_expert<true, false, EPI_STORE, true>(c, p2, tm, cdiv(d, tile_n(c)), s);
}

void launch_expert_bwd_dx(const moe_cfg& c, const void* dO, const int32_t* rb, const int32_t* re, const void* H,
                          const void* W1, const void* W2, void* dH, void* dXe, hipStream_t s) {
  const int64_t d = c.d_model, f = c.d_ff, C = c.C, Cp = rows_alloc(c);
  const int tm = cdiv(C + 15, tile_m(c));
  // dA = dO W2_e  (B(k=i, n=j) = W2[e][i][j], N contiguous), epilogue dH = dA * act'(H)
  GemmParams p1{dO, d, Cp * d, W2, f, d * f, dH, f, Cp * f, nullptr, H, rb, re, 0, (int)f, (int)d, c.act, (int)C};
  run_expert<false, false, EPI_DACT, true>(c, p1, tm, cdiv(f, tile_n(c)), s);
  // dXe = dH W1_e  (B(k=i, n=j) = W1[e][i][j])
  GemmParams p2{dH, f, Cp * f, W1, d, f * d, dXe, d, Cp * d, nullptr, nullptr, rb, re, 0, (int)d, (int)f, c.act, (int)C};
  run_expert<false, false, EPI_STORE, true>(c, p2, tm, cdiv(d, tile_n(c)), s);
}

void launch_expert_bwd_dw(const moe_cfg& c, const void* X, const void* A, const void* dO, const void* dH,
                          const int32_t* rb, const int32_t* re, void* dW1, void* dW2, hipStream_t s) {
  const int64_t d = c.d_model, f = c.d_ff, C = c.C, Cp = rows_alloc(c);
  // dW2_e [d][f] = dO_e^T A_e : A-operand(m, k) = dO[e][k][m], B(k, n) = A[e][k][n]
  GemmParams p2{dO, d, Cp * d, A, f, Cp * f, dW2, f, d * f, nullptr, nullptr, rb, re, (int)d, (int)f, 0, c.act, (int)C};
  run_expert<false, true, EPI_STORE, false>(c, p2, cdiv(d, tile_m(c)), cdiv(f, tile_n(c)), s);
  // dW1_e [f][d] = dH_e^T X_e
  GemmParams p1{dH, f, Cp * f, X, d, Cp * d, dW1, d, f * d, nullptr, nullptr, rb, re, (int)f, (int)d, 0, c.act, (int)C};
  run_expert<false, true, EPI_STORE, false>(c, p1, cdiv(f, tile_m(c)), cdiv(d, tile_n(c)), s);
}

// Dense bf16 products of the transformer block (one group, every row, row-major).
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
