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
// store, dA * act'(H) for the backward, a residual add, and float partials of
// a K-split dense weight gradient.
// The same kernel serves dense products (one group, no row ranges): the
// block's projections and, with row-major operands split into token ranges,
// their weight gradients.
// f32 path: a plain LDS-tiled FMA GEMM with the same addressing.
#include "internal.h"
#include "lds_ops.h"

#include <utility>
#include <vector>

namespace lmoe {

// EPI_WGF32: the dense weight-gradient product C = A^T B of the block, both
// operands row-major [K][*] (not blocked), K split into groups of kchunk rows
// (group g: rows [g kchunk, (g + 1) kchunk)), each group's float partial C at
// C + g sC; gemm_wgrad_reduce_kernel adds the partials in group order.
enum { EPI_STORE = 0, EPI_FWD1 = 1, EPI_DACT = 2, EPI_RES = 3, EPI_WGF32 = 4 };

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
  float* part;      // wide ragged-M products: partial tiles of the K-split (stream-K) schedule
  int ksplit;       // wide plain-store ragged-M products: 1 = a short last round may be K-split
  int kchunk;       // rb == re == NULL and kchunk > 0: group g's rows are [g kchunk, (g + 1) kchunk)
};

// Row range of group g, clamped to the buffer so bad ranges cannot reach outside it.
__device__ __forceinline__ void group_rows(const GemmParams& p, int g, int& lo, int& span) {
  int a = p.rb ? p.rb[g] : (p.kchunk > 0 ? g * p.kchunk : 0);
  int b = p.re ? p.re[g] : (p.kchunk > 0 ? (g + 1) * p.kchunk : p.cap);
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
// Operand tiles (BK = 32, one MFMA K step) move global -> LDS with buffer
// loads into LDS (each lane's 16 bytes land at LDS base + 16 * lane) into a
// multi-stage ring; a lane whose element lies outside the operand reads zeros.
//
// LDS layouts of a stage:
//  * K-contiguous operand, ROWS x 32: fragment-linear.  The 16 x 32 MFMA
//    fragment of rows 16f..16f+15 is 1 KB at offset 1 KB * f, lane L's 16
//    bytes (row 16f + L%16, k = 8*(L/16) .. +7) at 16 * L: one DMA instruction
//    fills one fragment and one ds_read_b128 reads it, both linear.
//  * MN-contiguous operand, 32 x COLS (row = k): [2][COLS/32] blocks of 16
//    rows x 4 chunks of 16 bytes, chunk c of block row r at c ^ bsw(r): the 16
//    lanes of a transposed read cover rows r..r+3 and the next lane group rows
//    r+8..r+11, and this swizzle puts those 8 x 32 bytes on distinct banks.
//    Fragments are read with ds_read_b64_tr_b16: within each 16-lane group,
//    lane j addresses row k0 + j/4, columns n0 + 4*(j%4) .. +3, and receives
//    column n0 + j of rows k0 .. k0+3 -- two such reads give the 8-element K
//    run of the MFMA operand.
constexpr int kBKb = 32;

// K-contiguous operand: ROWS x 32 tile, one wave instruction fills one fragment.
template <int ROWS, int NW>
struct TileK {
  static constexpr int NI = ROWS / 16 / NW;     // loads per wave per tile
  static_assert(NI >= 1 && ROWS % (16 * NW) == 0, "tile/waves mismatch");
  // Split reads (NF = 4 or 8): start the reads, later complete them in place.
  template <int NF>
  __device__ static void read_issue(u32x4 (&f)[NF], u32x2 (&)[8], const uint16_t* stage, int r0, int lane) {
    static_assert(NF == 4 || NF == 8, "split reads: 4 or 8 fragments");
    uint32_t a[NF];
#pragma unroll
    for (int u = 0; u < NF; ++u) a[u] = lds_addr(stage + ((r0 >> 4) + u) * 512 + lane * 8);
    Rd128Issue<NF>::run(f, a);
  }
};

// MN-contiguous operand: 32 x COLS tile (row = k), one wave instruction fills 64 chunks.
__device__ __forceinline__ int bsw(int r) { return 2 * (((r >> 1) ^ (r >> 3)) & 1); }
template <int COLS, int NW>
struct TileMN {
  static constexpr int CB = COLS / 32;          // column blocks per stage
  static constexpr int CPR = COLS / 8;          // 16-byte chunks per row
  static constexpr int NI = kBKb * CPR / 64 / NW;
  static_assert(NI >= 1 && (kBKb * CPR) % (64 * NW) == 0 && CPR >= 16, "tile/waves mismatch");
  // LDS element offset of (k, col) in a stage.
  __device__ static int lds_off(int k, int col) {
    const int r = k & 15;
    return ((k >> 4) * CB + (col >> 5)) * 512 + r * 32 + ((((col & 31) >> 3) ^ bsw(r)) << 3) + (col & 7);
  }
};


// Tiles of a group are numbered panel by panel (kPanelN tile columns wide),
// m-tile by m-tile inside a panel, n fastest, so the tiles an XCD has in
// flight form a square-ish patch whose operand slices are shared through that
// XCD's L2.
constexpr int kPanelN = 8;

// ------------------------------------------------------ wide bf16 MFMA tiles
// The expert products at full size.  256 x 256 block tiles, one block per CU,
// eight waves in a 2 x 4 grid, each owning a 128 x 64 tile (32 accumulator
// fragments) -- two waves per SIMD, so one wave's MFMAs issue while the other
// waits on memory (a four-wave 128 x 128 variant is kept for comparison).
// Against 128 x 128 block tiles this halves the operand bytes a CU moves
// global -> LDS per flop; the per-CU load path is what limits the smaller
// tile.
//
// Operands reach LDS through raw buffer loads with the LDS flag: a scalar
// buffer descriptor covers the operand's group from the current K-step on, so
// a K-step only moves the descriptor, and an out-of-range lane sets bit 31 of
// its offset, which the buffer range check turns into zeros.  Each K-step's
// fragment reads for the next step and the loads refilling the stage just
// consumed are interleaved one instruction at a time between the step's
// MFMAs, so the wave keeps issuing MFMAs while memory operations queue.
//
// The K loop runs continuously over every tile a block owns: the load cursor
// runs STAGES K-steps ahead of the compute cursor and crosses into the block's
// next tile while the current one finishes, so that tile's first stages land
// while the epilogue stores.  After an epilogue the first wait is a full
// vmcnt(0): stores and loads share the counter, and the order in which they
// complete is not relied on.
//
// The accumulators live in AGPRs through inline-asm MFMAs ("+a"), which keeps
// every fragment in one register quad for the whole tile.  The compiler does
// not see those MFMAs, so the hazards it would otherwise cover are fenced by
// hand: s_nop after VALU writes of fragment registers an MFMA reads next, and
// after the last MFMA of a tile before the accumulators are read.
//
// The product is computed transposed (MFMA A operand = a B fragment, B operand
// = an A fragment), so each lane's four accumulator values are four
// consecutive output columns of one row: the epilogue converts them with
// v_cvt_pk_bf16_f32 and stores 8-byte vectors straight from registers.
//
// LDS stages: four with one block barrier per K-step; five (the whole LDS)
// with one barrier per two K-steps (PAIR: the barrier before an even step
// covers the stages of both steps of the pair).  The products whose B operand
// is MN-contiguous (read transposed) run PAIR -- measured faster there (the
// ragged-K weight-gradient products -7 % at d_model 2048) -- and the
// K-contiguous ones four stages (PAIR measured +4 % there).
constexpr int kWB = 256;       // block tile (rows and columns)

// Immediate byte offset of fragment read r from its base (see read_base in the
// kernel): K-contiguous fragment r sits r KB on; an MN-contiguous half r % 2
// of fragment r / 2 sits (r / 4) blocks and (r % 2) * 4 rows on.
template <bool KC, int R>
constexpr int wide_read_imm() {
  return KC ? R * 1024 : ((R >> 2) * 512 + (R & 1) * 128) * 2;
}

// Compile-time loop: f(std::integral_constant<int, I>) for I in [B, E).
template <int B, int E, typename Fn>
__device__ __forceinline__ void static_for(Fn&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

struct WGeo {
  int g;        // group (expert)
  int m0, n0;   // tile origin (rows relative to lo_al for ragged-M products)
  int lo, hi;   // the group's row range in its [C][*] block
  int lo_al;    // lo rounded down to the 16-row block: origin of the tile rows (ragged-M) or of K (ragged-K)
  int Mlim, Klim, nk;
};

__device__ __forceinline__ uint32_t cvt_pk_bf16(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{lo, hi}), bf16x2_t));
}
__device__ __forceinline__ u32x2 pack4_bf16(const float (&v)[4]) {
  return u32x2{cvt_pk_bf16(v[0], v[1]), cvt_pk_bf16(v[2], v[3])};
}

__device__ __forceinline__ void mfma_acc(f32x4& acc, const u32x4& a, const u32x4& b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
// Wait states between VALU writes of fragment registers and the MFMAs that read them.
__device__ __forceinline__ void valu_to_mfma_fence(u32x4 (&f)[8]) {
  asm volatile("s_nop 4" : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]), "+v"(f[4]), "+v"(f[5]), "+v"(f[6]),
               "+v"(f[7]));
}
__device__ __forceinline__ void valu_to_mfma_fence(u32x4 (&f)[4]) {
  asm volatile("s_nop 4" : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]));
}
// Pins a row of accumulators in AGPRs at this point of the instruction stream.
__device__ __forceinline__ void acc_pin(f32x4 (&a)[8]) {
  asm volatile("" : "+a"(a[0]), "+a"(a[1]), "+a"(a[2]), "+a"(a[3]), "+a"(a[4]), "+a"(a[5]), "+a"(a[6]), "+a"(a[7]));
}
__device__ __forceinline__ void acc_pin(f32x4 (&a)[4]) {
  asm volatile("" : "+a"(a[0]), "+a"(a[1]), "+a"(a[2]), "+a"(a[3]));
}
// The same, ordered after every earlier memory operation.
__device__ __forceinline__ void acc_pin_mem(f32x4 (&a)[8]) {
  asm volatile("" : "+a"(a[0]), "+a"(a[1]), "+a"(a[2]), "+a"(a[3]), "+a"(a[4]), "+a"(a[5]), "+a"(a[6]), "+a"(a[7])
               :: "memory");
}
__device__ __forceinline__ void acc_pin_mem(f32x4 (&a)[4]) {
  asm volatile("" : "+a"(a[0]), "+a"(a[1]), "+a"(a[2]), "+a"(a[3])::"memory");
}

// One operand's loads for the K-steps of a tile (256 rows or columns x 32 K
// per stage, blocked source), as raw buffer loads into LDS.  The buffer
// descriptor spans the operand's group (expert) from the current K-step on, so
// a K-step only moves the descriptor (scalar adds), and a lane whose chunk is
// out of range carries bit 31 in its offset, which the buffer range check
// turns into zeros.  K-contiguous (KC): the chunk of fragment q is a whole
// 16 x 32 block, rows past `lim` read zeros.  MN-contiguous: 32 K rows x 256
// columns as 2 x 8 blocks, each lane's chunk placed at its swizzled position;
// columns past `lim` and, with KCHK, K rows outside [klo, khi) read zeros.
constexpr int kBufCfg = 0x00020000;   // buffer descriptor word 3: raw 32-bit data, gfx9 family
constexpr uint32_t kOob = 0x80000000u;
// RM (MN-contiguous only): the operand is row-major [K][ld] instead of blocked;
// a lane loads the same 16-byte chunk (K row, 8 columns) that it would take
// from the blocked layout, so the stage's LDS layout is the same.
template <bool KC, bool KCHK, int NW, bool RM = false>
struct WOp {
  static constexpr int kWNI = 16 / NW;   // loads per wave per stage (16 blocks of 1 KB)
  const char* base;      // the group's operand (uniform)
  uint32_t bytes;        // its extent in bytes (uniform)
  uint32_t stride;       // bytes per K-step (uniform)
  uint32_t voff[kWNI];   // byte offset of the lane's chunk at K-step 0, | kOob if out of range
  int kr[kWNI];          // KCHK: K row of the lane's chunk at K-step 0
  int klo, khi;

  // KC: row0 = first row of the tile (multiple of 16), lim = row limit.
  // MN: row0 = first column of the tile, lim = column limit, korg = K origin (multiple of 16).
  __device__ __forceinline__ void plan(const uint16_t* b, int64_t extent, int64_t ld, int row0, int lim, int korg,
                                       int lo, int hi, int wid, int lane) {
    base = (const char*)b;
    bytes = (uint32_t)(extent * 2);
    klo = lo;
    khi = hi;
    if constexpr (KC) {
      stride = 1024;
#pragma unroll
      for (int i = 0; i < kWNI; ++i) {
        const int rb = (row0 >> 4) + i * NW + wid;
        const uint32_t off = (uint32_t)(rb * (int)(ld >> 5) * 512 + (lane & 15) * 32 + (lane >> 4) * 8) * 2u;
        voff[i] = (16 * rb + (lane & 15) < lim) ? off : (off | kOob);
        kr[i] = 0;
      }
    } else {
      const int nb = (int)(ld >> 5);
      stride = RM ? (uint32_t)(32 * ld * 2) : (uint32_t)nb * 2048u;
      const int r = lane >> 2;
      const int c = (lane & 3) ^ bsw(r);
#pragma unroll
      for (int i = 0; i < kWNI; ++i) {
        const int b2 = i * NW + wid;
        const int kb = b2 / 8, cb = b2 % 8;
        const int col = row0 + 32 * cb;
        const uint32_t off =
            RM ? (uint32_t)(((int64_t)(korg + 16 * kb + r) * ld + col + c * 8) * 2)
               : (uint32_t)((((korg >> 4) + kb) * nb + (col >> 5)) * 512 + r * 32 + c * 8) * 2u;
        voff[i] = col < lim ? off : (off | kOob);
        kr[i] = korg + 16 * kb + r;
      }
    }
  }
  // Load i (0 .. kWNI-1) of K-step kk into its place in the stage.
  __device__ __forceinline__ void issue(int i, int kk, uint16_t* stage, int wid) const {
    const uint32_t adv = (uint32_t)kk * stride;
    const __amdgpu_buffer_rsrc_t r =
        __builtin_amdgcn_make_buffer_rsrc((void*)(base + adv), (short)0, (int)(bytes - adv), kBufCfg);
    uint32_t vo = voff[i];
    if constexpr (KCHK) {
      const int k = kr[i] + 32 * kk;
      if (k < klo || k >= khi) vo |= kOob;
    }
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)(stage + (i * NW + wid) * 512), 16, vo, 0, 0, 0);
  }
  // The same, branch-free, with the K-step's descriptor made once per step:
  // with live false the descriptor is empty, so the load writes zeros into
  // the stage (a stage no later step reads).
  __device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(int kk, bool live) const {
    const uint32_t adv = (uint32_t)kk * stride;
    return __builtin_amdgcn_make_buffer_rsrc((void*)(base + adv), (short)0, live ? (int)(bytes - adv) : 0, kBufCfg);
  }
  __device__ __forceinline__ void issue_r(int i, __amdgpu_buffer_rsrc_t r, int kk, uint16_t* stage, int wid) const {
    uint32_t vo = voff[i];
    if constexpr (KCHK) {
      const int k = kr[i] + 32 * kk;
      if (k < klo || k >= khi) vo |= kOob;
    }
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)(stage + (i * NW + wid) * 512), 16, vo, 0, 0, 0);
  }
};

// Schedule of one XCD's n tiles xtile(0 .. n-1) over its nslot blocks.  Rounds
// of whole tiles run in lock step (block s takes tiles xtile(q nslot + s)), so the
// tiles in flight share their K position and their operand slices in L2.  A
// last round that would leave most blocks idle (r <= nslot / 4 tiles) is
// split instead: the r tiles' K-steps go to all nslot blocks, each tile to a
// contiguous group of blocks, each block a contiguous K range of one tile;
// the partial sums are added by gemm_wide_fixup_kernel.
struct WSched {
  int R, r;      // full rounds; tiles left for the last round
  bool split;    // the last round is K-split
  // K-split: the remainder tile of block `slot`, the first block of that tile,
  // its number of blocks, and the block's K range [k0, k1).
  __device__ __forceinline__ void split_part(int slot, int nslot, int nk, int& q, int& first, int& cnt, int& k0,
                                             int& k1) const {
    q = slot * r / nslot;
    first = (q * nslot + r - 1) / r;
    cnt = ((q + 1) * nslot + r - 1) / r - first;
    const int rank = slot - first;
    k0 = rank * nk / cnt;
    k1 = (rank + 1) * nk / cnt;
  }
};
__device__ __forceinline__ WSched wide_sched(int n, int nslot, bool allow_split) {
  WSched w;
  w.R = n / nslot;
  w.r = n - w.R * nslot;
  w.split = allow_split && w.r > 0 && 4 * w.r <= nslot;
  return w;
}

// Lane-per-group tile counts of a wide product and their prefixes (groups <= 64).
// Ragged-K, or ragged-M without SEP: every tile of a group (with rows).
// Ragged-M with SEP: the full M-tiles (256 rows) and, separately, the short
// last M-tile of a group whose rows are not a multiple of 256; tile numbers
// [0, NF) are the full tiles, [NF, NF + NP) the short ones, so a schedule can
// place the short (cheaper) tiles last.
struct WPrefix {
  int incl, excl;     // full tiles (ragged-K: all tiles), lane = group
  int inclP, exclP;   // ragged-M short tiles, lane = group
  int NF, NP;         // totals (uniform)
  int lo, span;       // the group's clamped row range (group_rows), lane = group: read once, so a
                      // tile change never waits on a memory load (which would drain the wave's
                      // in-flight operand loads and epilogue stores)
};
template <bool RAGGED_K, bool SEP>
__device__ __forceinline__ WPrefix wide_tile_prefix(const GemmParams& p, int lane, int groups, int tilesM,
                                                    int tilesN) {
  int cnt = 0, cntP = 0;
  int lo = 0, span = 0;
  if (lane < groups) {
    group_rows(p, lane, lo, span);
    if constexpr (RAGGED_K) {
      cnt = span > 0 ? tilesM * tilesN : 0;   // an empty group's output is zeroed in the prologue
    } else {
      const int rows = span > 0 ? span + (lo & 15) : 0;   // from the 16-row block holding the first row
      const int tm = (rows + kWB - 1) / kWB;
      const int sh = (SEP && (rows % kWB) != 0) ? 1 : 0;
      cnt = (tm - sh) * tilesN;
      cntP = sh * tilesN;
    }
  }
  WPrefix P;
  P.incl = cnt;
  P.inclP = cntP;
  P.lo = lo;
  P.span = span;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(P.incl, o, 64);
    const int v = __shfl_up(P.inclP, o, 64);
    if (lane >= o) {
      P.incl += u;
      P.inclP += v;
    }
  }
  P.excl = P.incl - cnt;
  P.exclP = P.inclP - cntP;
  P.NF = __builtin_amdgcn_readfirstlane(__shfl(P.incl, groups - 1, 64));
  P.NP = __builtin_amdgcn_readfirstlane(__shfl(P.inclP, groups - 1, 64));
  return P;
}

// Geometry of tile t of a wide product.  Within a group, tiles (with SEP: the
// full tiles) are numbered panel by panel (kPanelN tile columns), m-tiles
// within a panel, n fastest, so the tiles one XCD has in flight form a
// square-ish patch; with SEP a group's short last M-tile has its own numbers
// (t >= NF), n order.
template <bool RAGGED_K, bool SEP>
__device__ __forceinline__ WGeo wide_geo(const GemmParams& p, int t, int lane, int groups, const WPrefix& P,
                                         int tilesM, int tilesN) {
  WGeo G;
  const bool shrt = SEP && !RAGGED_K && t >= P.NF;
  const int tt = shrt ? t - P.NF : t;
  const int inc = shrt ? P.inclP : P.incl;
  const int exc = shrt ? P.exclP : P.excl;
  G.g = __builtin_amdgcn_readfirstlane(__popcll(__ballot(lane < groups && inc <= tt)));
  const int local = tt - __builtin_amdgcn_readlane(exc, G.g);
  const int lo = __builtin_amdgcn_readlane(P.lo, G.g);
  int span = __builtin_amdgcn_readlane(P.span, G.g);
  G.lo = lo;
  G.hi = lo + span;
  G.lo_al = lo & ~15;
  if (span > 0) span += lo - G.lo_al;
  if (shrt) {
    G.m0 = ((span + kWB - 1) / kWB - 1) * kWB;
    G.n0 = local * kWB;
  } else {
    const int tmg = RAGGED_K ? tilesM : (SEP ? span / kWB : (span + kWB - 1) / kWB);   // (full) M-tiles
    const int pnl = local / (tmg * kPanelN);
    const int rem = local - pnl * tmg * kPanelN;
    const int pw = min(kPanelN, tilesN - pnl * kPanelN);
    G.m0 = (rem / pw) * kWB;
    G.n0 = (pnl * kPanelN + rem % pw) * kWB;
  }
  G.Mlim = RAGGED_K ? p.M : span;
  G.Klim = RAGGED_K ? span : p.K;
  G.nk = max(1, (G.Klim + kBKb - 1) / kBKb);
  return G;
}

// One XCD's tiles of a ragged-M product: an even share of the full tiles, as
// one contiguous range (neighbouring operand panels in the XCD's L2), then an
// even share of the short tiles.  tile(j) = the XCD's j-th tile.
struct WRange {
  int f0, nf, p0, np, NF;
  __device__ __forceinline__ int tile(int j) const { return j < nf ? f0 + j : NF + p0 + (j - nf); }
};
__device__ __forceinline__ WRange wide_range(const WPrefix& P, int xcd) {
  WRange r;
  const int perF = (P.NF + 7) / 8, perP = (P.NP + 7) / 8;
  r.f0 = xcd * perF;
  r.nf = max(min(P.NF, r.f0 + perF) - r.f0, 0);
  r.p0 = xcd * perP;
  r.np = max(min(P.NP, r.p0 + perP) - r.p0, 0);
  r.NF = P.NF;
  return r;
}

// Epilogue of one wave's tile from its accumulators: bf16 conversion and the
// EPI-specific store (plain, (H, act(H)), or dA * act'(H) with H read back).
// acc[i][j] holds output row 16 i + l % 16, columns 16 j + 4 (l / 16) .. +3 of
// the wave tile at (G.m0 + wm WTM, G.n0 + wn WTN).
template <int FM, int FN, int WTM, int WTN, bool RAGGED_K, int EPI, int ACT, bool CBLK>
__device__ __forceinline__ void wide_epilogue(const GemmParams& p, const WGeo& G, f32x4 (&acc)[FM][FN], int wm,
                                              int wn, int lane, int i_lo = 0, int i_hi = FM) {
  // Buffer stores and loads over the group's output: a lane outside the
  // product carries an out-of-range offset (store dropped, load zero), so
  // the epilogue is branch-free and dA * act'(H) issues all of a half's H
  // loads together.  Group offsets fit 31 bits (validated on the host).
  const int64_t cofs = (int64_t)G.g * p.sC + (RAGGED_K || CBLK ? 0 : (int64_t)G.lo_al * p.ldc);
  constexpr int ESZ = EPI == EPI_WGF32 ? 4 : 2;   // bytes per output element
  void* const cbase = EPI == EPI_WGF32 ? (void*)((float*)p.C + cofs) : (void*)((uint16_t*)p.C + cofs);
  const __amdgpu_buffer_rsrc_t rC = __builtin_amdgcn_make_buffer_rsrc(cbase, (short)0, 0x7fffffff, kBufCfg);
  __amdgpu_buffer_rsrc_t rC2 = rC, rAux = rC;
  if constexpr (EPI == EPI_FWD1)
    rC2 = __builtin_amdgcn_make_buffer_rsrc((uint16_t*)p.C2 + cofs, (short)0, 0x7fffffff, kBufCfg);
  if constexpr (EPI == EPI_DACT || EPI == EPI_RES)
    rAux = __builtin_amdgcn_make_buffer_rsrc((uint16_t*)p.Aux + cofs, (short)0, 0x7fffffff, kBufCfg);
  const int rl = lane & 15, cq = 4 * (lane >> 4);
  auto voff = [&](bool ok, int row, int col) __attribute__((always_inline)) -> uint32_t {
    const int64_t e = CBLK ? blk_off((RAGGED_K ? 0 : G.lo_al) + row, col, p.ldc) : (int64_t)row * p.ldc + col;
    return ok ? (uint32_t)(e * ESZ) : kOob;
  };
#pragma unroll
  for (int h = 0; h < 2; ++h) {          // two halves of four fragment rows
    u32x2 aux[4][FN];
    if constexpr (EPI == EPI_DACT || EPI == EPI_RES) {   // all loads of the half first, then the math
#pragma unroll
      for (int ii = 0; ii < 4; ++ii) {
        const int row = G.m0 + wm * WTM + 16 * (4 * h + ii) + rl;
        const bool rok = row < G.Mlim && (RAGGED_K || G.lo_al + row >= G.lo) && 4 * h + ii >= i_lo && 4 * h + ii < i_hi;
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int col = G.n0 + wn * WTN + 16 * j + cq;
          aux[ii][j] = __builtin_amdgcn_raw_buffer_load_b64(rAux, (int)voff(rok && col < p.N, row, col), 0, 0);
        }
      }
    }
#pragma unroll
    for (int ii = 0; ii < 4; ++ii) {
      const int i = 4 * h + ii;
      if (i < i_lo || i >= i_hi) continue;
      const int row = G.m0 + wm * WTM + 16 * i + rl;
      const bool rok = row < G.Mlim && (RAGGED_K || G.lo_al + row >= G.lo);
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int col = G.n0 + wn * WTN + 16 * j + cq;
        const int vo = (int)voff(rok && col < p.N, row, col);
        float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
        if constexpr (EPI == EPI_FWD1) {
          __builtin_amdgcn_raw_buffer_store_b64(pack4_bf16(v), rC, vo, 0, 0);
#pragma unroll
          for (int u = 0; u < 4; ++u) v[u] = act_fwd_t<ACT>(v[u]);
          __builtin_amdgcn_raw_buffer_store_b64(pack4_bf16(v), rC2, vo, 0, 0);
        } else if constexpr (EPI == EPI_DACT) {
          const u32x2 hv = aux[ii][j];
          const float hh[4] = {__uint_as_float(hv[0] << 16), __uint_as_float(hv[0] & 0xffff0000u),
                               __uint_as_float(hv[1] << 16), __uint_as_float(hv[1] & 0xffff0000u)};
#pragma unroll
          for (int u = 0; u < 4; ++u) v[u] *= act_bwd_t<ACT>(hh[u]);
          __builtin_amdgcn_raw_buffer_store_b64(pack4_bf16(v), rC, vo, 0, 0);
        } else if constexpr (EPI == EPI_WGF32) {
          __builtin_amdgcn_raw_buffer_store_b128(
              u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3])}, rC, vo,
              0, 0);
        } else if constexpr (EPI == EPI_RES) {
          const u32x2 rv = aux[ii][j];
          v[0] += __uint_as_float(rv[0] << 16);
          v[1] += __uint_as_float(rv[0] & 0xffff0000u);
          v[2] += __uint_as_float(rv[1] << 16);
          v[3] += __uint_as_float(rv[1] & 0xffff0000u);
          __builtin_amdgcn_raw_buffer_store_b64(pack4_bf16(v), rC, vo, 0, 0);
        } else {
          __builtin_amdgcn_raw_buffer_store_b64(pack4_bf16(v), rC, vo, 0, 0);
        }
      }
    }
  }
}

// NW = 4: waves 2 x 2, wave tile 128 x 128, one wave per SIMD.
// NW = 8: waves 2 x 4, wave tile 128 x 64, two waves per SIMD, which lets the
// SIMD issue one wave's MFMAs while the other waits on memory.
template <int NW, int STAGES, bool B_K, bool RAGGED_K, int EPI, int ACT, bool CBLK>
__global__ __attribute__((amdgpu_flat_work_group_size(NW * 64, NW * 64), amdgpu_waves_per_eu(NW / 4, NW / 4))) void
gemm_wide_kernel(GemmParams p, int tilesM, int tilesN, int groups) {
  constexpr int BK = kBKb;
  constexpr int WGN = NW / 2;                   // wave grid 2 x WGN
  constexpr int WTM = 128, WTN = kWB / WGN;     // wave tile
  constexpr int FM = WTM / 16, FN = WTN / 16;   // fragments per wave tile side
  constexpr int kWNI = 16 / NW;
  constexpr int STAGE = (kWB + kWB) * BK;       // elements per pipeline stage
  constexpr bool A_K = !RAGGED_K;
  constexpr bool BK_C = B_K && !RAGGED_K;
  using TA = typename std::conditional<A_K, TileK<kWB, NW>, TileMN<kWB, NW>>::type;
  using TB = typename std::conditional<BK_C, TileK<kWB, NW>, TileMN<kWB, NW>>::type;
  static_assert(TA::NI == kWNI && TB::NI == kWNI, "load plan");
  constexpr int LPS = 2 * kWNI;                  // loads per wave per stage
  static_assert(STAGES >= 2 && LPS * (STAGES - 1) < 64, "vmcnt range");
  constexpr bool PAIR = STAGES >= 5;
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];

  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wid / WGN, wn = wid % WGN;

  // Tile counts per group and their prefix (every wave computes the same values).
  // Only the plain-store ragged-M products may K-split their last round (the
  // narrow-N products where a ragged last round idles most of the GPU); the
  // others keep the simpler whole-tile schedule and its register budget.
  // The K-split products place their short tiles last (SEP), so the split
  // round holds the short tiles, whose partial sums stop at the group's rows.
  constexpr bool SPLIT = !RAGGED_K && EPI == EPI_STORE;
  const WPrefix P = wide_tile_prefix<RAGGED_K, SPLIT>(p, lane, groups, tilesM, tilesN);
  const int total = P.NF + P.NP;
  if constexpr (RAGGED_K) {
    // Groups without rows have no tiles: their [M][N] outputs are zeroed here,
    // spread over the whole grid (16-byte stores; no tile writes them).
    uint64_t empty = __ballot(lane < groups && P.incl == P.excl);
    const int64_t chunks = (int64_t)p.M * p.N / (EPI == EPI_WGF32 ? 4 : 8);
    const int64_t gtid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x, gstride = (int64_t)gridDim.x * blockDim.x;
    while (empty) {
      const int g = __builtin_ctzll(empty);
      empty &= empty - 1;
      u32x4* o = EPI == EPI_WGF32 ? reinterpret_cast<u32x4*>((float*)p.C + (int64_t)g * p.sC)
                                  : reinterpret_cast<u32x4*>((uint16_t*)p.C + (int64_t)g * p.sC);
      for (int64_t i = gtid; i < chunks; i += gstride) o[i] = u32x4{0u, 0u, 0u, 0u};
    }
  }
  const int nslot = gridDim.x / 8;
  const int xcd = blockIdx.x % 8, slot = blockIdx.x / 8;
  // The XCD's tiles: ragged-M products (one K length) take a contiguous range
  // of the (full) tiles, so the XCD's L2 holds neighbouring operand panels,
  // then with SEP their share of the short last M-tiles;
  // ragged-K products, whose tiles cost as many K-steps as their group has
  // rows, take every eighth tile, so each XCD gets an even share of every
  // group (with skewed routing, a contiguous range could hold the few large
  // groups).  xtile(j) = the XCD's j-th tile.
  // The block's segments (see WSched): nd whole tiles xtile(e nslot + slot),
  // then, if the last round is K-split (ragged-M products, one K length), the
  // K range [sk0, sk1) of remainder tile xtile(R nslot + sq).
  const WRange XR = wide_range(P, xcd);
  const int nx = RAGGED_K ? (total > xcd ? (total - xcd + 7) / 8 : 0) : XR.nf + XR.np;
  auto xtile = [&](int j) __attribute__((always_inline)) { return RAGGED_K ? xcd + 8 * j : XR.tile(j); };
  const int nkU = (p.K + BK - 1) / BK;
  const WSched W = wide_sched(nx, nslot, SPLIT && p.ksplit != 0);
  int sq = 0, sfirst = 0, scnt = 0, sk0 = 0, sk1 = 0;
  if (SPLIT && W.split) W.split_part(slot, nslot, nkU, sq, sfirst, scnt, sk0, sk1);
  // (uniform values: keep them in scalar registers)
  const int WR = __builtin_amdgcn_readfirstlane(W.R);
  sq = __builtin_amdgcn_readfirstlane(sq);
  sk0 = __builtin_amdgcn_readfirstlane(sk0);
  sk1 = __builtin_amdgcn_readfirstlane(sk1);
  const int nd = __builtin_amdgcn_readfirstlane(W.R + (!W.split && slot < W.r ? 1 : 0));
  const int nseg = __builtin_amdgcn_readfirstlane(nd + (SPLIT && W.split && sk0 < sk1 ? 1 : 0));
  if (nseg == 0) return;

  auto geo = [&](int t) __attribute__((always_inline)) {
    return wide_geo<RAGGED_K, SPLIT>(p, t, lane, groups, P, tilesM, tilesN);
  };

  // Segment e: tile, first K-step, end K-step (0 = the tile's own count).
  auto seg = [&](int e, int& t, int& k0, int& k1) __attribute__((always_inline)) {
    if (e < nd) {
      t = xtile(e * nslot + slot);
      k0 = 0;
      k1 = 0;
    } else {
      t = xtile(WR * nslot + sq);
      k0 = sk0;
      k1 = sk1;
    }
  };
  // Load cursor: segment le, its tile lt, K-step lk, end lkend; ls = stages
  // issued so far.
  // EPI_WGF32: both operands row-major and shared by every group (each group
  // a K range of them), so the extent is the whole operand.
  constexpr bool RMO = EPI == EPI_WGF32;
  static_assert(!RMO || RAGGED_K, "row-major operands: ragged-K products only");
  WOp<A_K, RAGGED_K, NW, RMO> opA;
  WOp<BK_C, RAGGED_K, NW, RMO> opB;
  int le = 0, lt = 0, lk = 0, lkend = 0, ls = 0;
  auto plan = [&](int t) __attribute__((always_inline)) {
    const WGeo G = geo(t);
    const uint16_t* Ab = (const uint16_t*)p.A + (RMO ? 0 : G.g * p.sA);
    const uint16_t* Bb = (const uint16_t*)p.B + (RMO ? 0 : G.g * p.sB);
    const int64_t extA = RMO ? (int64_t)p.cap * p.lda : p.sA, extB = RMO ? (int64_t)p.cap * p.ldb : p.sB;
    if constexpr (A_K) opA.plan(Ab, p.sA, p.lda, G.lo_al + G.m0, (int)pad16(p.cap), 0, 0, 0, wid, lane);
    else opA.plan(Ab, extA, p.lda, G.m0, p.M, G.lo_al, G.lo, G.hi, wid, lane);
    if constexpr (BK_C) opB.plan(Bb, p.sB, p.ldb, G.n0, p.N, 0, 0, 0, wid, lane);
    else if constexpr (RAGGED_K) opB.plan(Bb, extB, p.ldb, G.n0, p.N, G.lo_al, G.lo, G.hi, wid, lane);
    else opB.plan(Bb, p.sB, p.ldb, G.n0, p.N, 0, 0, p.K, wid, lane);
    if (lkend == 0) lkend = G.nk;
  };
  auto enter = [&]() __attribute__((always_inline)) {   // load cursor onto segment le
    seg(le, lt, lk, lkend);
    plan(lt);
  };
  enter();
  auto loads_left = [&]() __attribute__((always_inline)) { return le < nseg; };
  // Load q (0 .. 2 kWNI - 1; even: A, odd: B) of the next stage.
  auto issue_load = [&](int q) __attribute__((always_inline)) {
    if (!loads_left()) return;
    uint16_t* st = lds + ((unsigned)ls % STAGES) * STAGE;
    if (q & 1) opB.issue(q >> 1, lk, st + kWB * BK, wid);
    else opA.issue(q >> 1, lk, st, wid);
  };
  // Moves the load cursor past the stage just issued.
  auto advance = [&]() __attribute__((always_inline)) {
    if (!loads_left()) return;
    ++ls;
    if (++lk == lkend) {
      ++le;
      if (loads_left()) enter();
    }
  };

  // Fragment reads.  K-contiguous operands: 8 ds_read_b128 (one per
  // fragment).  MN-contiguous: 16 ds_read_b64_tr_b16, two per fragment.
  using Pend = u32x2[8];
  auto read_issue = [&](auto tile, auto& f, Pend& p0, Pend& p1, const uint16_t* st, int c0)
                        __attribute__((always_inline)) {
    using T = decltype(tile);
    constexpr int NF = sizeof(f) / sizeof(u32x4);
    if constexpr (std::is_same<T, TileK<kWB, NW>>::value) {
      T::template read_issue<NF>(f, p0, st, c0, lane);
    } else {
      const int j = lane & 15;
      const int k = 8 * (lane >> 4) + (j >> 2);
      uint32_t a0[8], a1[8];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int col0 = c0 + 16 * u + 4 * (j & 3), col1 = col0 + 64;
        a0[2 * u] = lds_addr(st + T::lds_off(k, col0));
        a0[2 * u + 1] = lds_addr(st + T::lds_off(k + 4, col0));
        a1[2 * u] = lds_addr(st + T::lds_off(k, col1));
        a1[2 * u + 1] = lds_addr(st + T::lds_off(k + 4, col1));
      }
      RdTrIssue8::run(p0, a0);
      if constexpr (NF == 8) RdTrIssue8::run(p1, a1);
    }
  };
  auto read_finish = [&](auto tile, auto& f, Pend& p0, Pend& p1) __attribute__((always_inline)) {
    using T = decltype(tile);
    constexpr int NF = sizeof(f) / sizeof(u32x4);
    if constexpr (std::is_same<T, TileK<kWB, NW>>::value) {
      lds_wait(f);
    } else {
      lds_wait(p0);
      if constexpr (NF == 8) lds_retired(p1);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        f[u] = u32x4{p0[2 * u][0], p0[2 * u][1], p0[2 * u + 1][0], p0[2 * u + 1][1]};
        if constexpr (NF == 8) f[4 + u] = u32x4{p1[2 * u][0], p1[2 * u][1], p1[2 * u + 1][0], p1[2 * u + 1][1]};
      }
      valu_to_mfma_fence(f);
    }
  };

  f32x4 acc[FM][FN];
  auto zero_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    asm volatile("s_nop 4" ::: "memory");
#pragma unroll
    for (int i = 0; i < FM; ++i) acc_pin(acc[i]);
  };
  // acc[i][j] holds the transposed 16 x 16 product: lane l has output row
  // 16 i + l % 16, columns 16 j + 4 (l / 16) .. +3 of the wave tile.
  auto mfma_rows = [&](int i0, int i1, u32x4 (&ca)[FM], u32x4 (&cb)[FN]) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      if (i < i0 || i >= i1) continue;
#pragma unroll
      for (int j = 0; j < FN; ++j) mfma_acc(acc[i][j], cb[j], ca[i]);
    }
  };

  auto epilogue = [&](const WGeo& G) __attribute__((always_inline)) {
    // Wait states between the last MFMA and the first read of its accumulator.
    asm volatile("s_nop 15\n s_nop 15" ::: "memory");
#pragma unroll
    for (int i = 0; i < FM; ++i) acc_pin(acc[i]);
    wide_epilogue<FM, FN, WTM, WTN, RAGGED_K, EPI, ACT, CBLK>(p, G, acc, wm, wn, lane);
  };

  // Prologue: fill the ring (PAIR: all but one stage, the slot the first
  // step refills), wait for the first stage, read its fragments.
#pragma unroll
  for (int s = 0; s < (PAIR ? STAGES - 1 : STAGES); ++s) {
#pragma unroll
    for (int q = 0; q < 2 * kWNI; ++q) issue_load(q);
    advance();
  }
  wait_vm_tiles<LPS, STAGES - 1>(ls - 1);
  lds_barrier();
  u32x4 fa0[FM], fb0[FN], fa1[FM], fb1[FN];
  Pend pa0, pa1, pb0, pb1;
  read_issue(TA{}, fa0, pa0, pa1, lds, wm * WTM);
  read_finish(TA{}, fa0, pa0, pa1);
  read_issue(TB{}, fb0, pb0, pb1, lds + kWB * BK, wn * WTN);
  read_finish(TB{}, fb0, pb0, pb1);
  zero_acc();

  int cs = 0;                // compute steps done (over all of the block's tiles)
  // The first step after an epilogue drains every store before its barrier
  // (measured faster than letting the stores overlap the next tile's loads).
  bool stores_pending = false;
  // One K-step: multiply the fragments in (ca, cb) while the next stage's
  // loads are issued and its fragments read into (na, nb).
  // Fragment read plan of the next stage: NRA reads for A, NRB for B (one
  // ds_read_b128 per K-contiguous fragment, two ds_read_b64_tr_b16 per
  // MN-contiguous one), each landing in its fragment or in a half-fragment
  // pending register.
  constexpr bool AK = std::is_same<TA, TileK<kWB, NW>>::value;
  constexpr bool BKK = std::is_same<TB, TileK<kWB, NW>>::value;
  constexpr int NRA = AK ? FM : 2 * FM, NRB = BKK ? FN : 2 * FN, NRD = NRA + NRB;
  constexpr int NMF = FM * FN, NDMA = 2 * kWNI;
  // PRE: MFMAs of a step issued before its wait and barrier (they use the
  // fragments read in the previous step), at the low wave priority; the rest
  // of the step, with the reads and refills, follows the barrier at the raised
  // priority.  Of the two waves on a SIMD the older one wins every tie for the
  // matrix core, so it finishes its MFMAs first and then waits at the barrier
  // while the other still issues; the early wave's PRE MFMAs of the next step
  // fill the matrix core while the late wave finishes its step, waits and
  // passes the barrier.  Measured (16384-token layer, one MI355X, per-wave
  // cycle counters): FWD2 1750 -> 1564 cycles per K-step, dXe 1773 -> 1505;
  // the layer's ragged-M calls -4 to -7 %, 12 and 16 equal, 20 and 24 slower.
  // The ragged-K (dW) products were measured slower with it (+2 %) and keep 0.
  constexpr int PRE = RAGGED_K ? 0 : 16;
  constexpr int RSPAN = (NMF - PRE) * 3 / 4;  // reads issued within the first 3/4 of the MFMAs after PRE
  u32x2 qa[2 * FM], qb[2 * FN];               // pending halves of MN-contiguous fragments
  // LDS byte address of read r of an operand = base(par) + imm(r), with a
  // compile-time immediate, so a step needs one or two base registers per
  // operand.  K-contiguous: fragment r, base at fragment 0, imm = r KB.
  // MN-contiguous: half h = r % 2 of fragment u = r / 2; within the swizzled
  // 16 x 32 blocks the lane's chunk depends on u % 2 (par) and on the lane,
  // while the block (u / 2) and the +4 rows of the second half are constant
  // offsets (rows k and k + 4 share their swizzle).
  auto read_base = [&](auto tile, const uint16_t* st, int c0, int par) __attribute__((always_inline)) -> uint32_t {
    using T = decltype(tile);
    if constexpr (std::is_same<T, TileK<kWB, NW>>::value) {
      return lds_addr(st + (c0 >> 4) * 512 + lane * 8);
    } else {
      const int j = lane & 15;
      const int k = 8 * (lane >> 4) + (j >> 2);
      return lds_addr(st + T::lds_off(k, c0 + 16 * par + 4 * (j & 3)));
    }
  };
  // One K-step: the MFMAs of (ca, cb), with the next stage's fragment reads
  // into (na, nb) and the refill of this step's stage interleaved between
  // them one instruction at a time, so the wave keeps issuing MFMAs while the
  // memory operations queue.
  // MMA false: a wave whose rows of the tile are all past the group's last
  // row keeps its share of the loads and reads but issues no MFMAs, leaving
  // the matrix core to the other wave on its SIMD.
  auto step = [&](auto mmac, u32x4 (&ca)[FM], u32x4 (&cb)[FN], u32x4 (&na)[FM], u32x4 (&nb)[FN])
                  __attribute__((always_inline)) {
    constexpr bool MMA = decltype(mmac)::value;
    const uint16_t* st = lds + ((unsigned)(cs + 1) % STAGES) * STAGE;
    // This step's refill: stage ls, K-step lk of the load cursor (issued
    // unconditionally; past the block's last load it writes zeros into the
    // ring slot of a K-step already consumed, which no later step reads).
    uint16_t* const dst = lds + ((unsigned)ls % STAGES) * STAGE;
    const bool live = loads_left();
    const int kdma = lk;
    const __amdgpu_buffer_rsrc_t rsa = opA.rsrc(kdma, live), rsb = opB.rsrc(kdma, live);
    const bool more = cs + 1 < ls;
    auto sync = [&]() __attribute__((always_inline)) {
    if constexpr (PAIR) {
      // Even step: stages cs+1 and cs+2 have landed (at most stage cs+3 is
      // pending) and, after the barrier, are in LDS for every wave; every wave
      // is past step cs-1, so no wave reads the stages of K-steps cs-1 and cs
      // any more -- the refills of steps cs and cs+1 (ls <= cs+4 and ls+1:
      // ring slots of K-steps ls-5 <= cs-1 and cs).  Odd step: nothing to wait
      // for but this wave's epilogue stores.
      if ((cs & 1) == 0) {
        if (more) {
          if (stores_pending) {
            wait_vm<0>();
            stores_pending = false;
          } else {
            wait_vm_tiles<LPS, STAGES - 4>(ls - cs - 3);
          }
          lds_barrier();
        }
      } else if (stores_pending) {
        wait_vm<0>();
        stores_pending = false;
      }
    } else if (more) {
      if (stores_pending) {
        wait_vm<0>();
        stores_pending = false;
      } else {
        wait_vm_tiles<LPS, STAGES - 2>(ls - cs - 2);   // stage cs+1 has landed
      }
      lds_barrier();   // stage cs+1 is in LDS for every wave; no wave reads stage cs any more
    }
    };
    if constexpr (PRE == 0) sync();
    // The reads are unconditional (branch-free, so pending registers are never
    // copied); after the last step they read a stage no load is writing.
    const uint32_t ra0 = read_base(TA{}, st, wm * WTM, 0);
    const uint32_t ra1 = AK ? ra0 : read_base(TA{}, st, wm * WTM, 1);
    const uint32_t rb0 = read_base(TB{}, st + kWB * BK, wn * WTN, 0);
    const uint32_t rb1 = BKK ? rb0 : read_base(TB{}, st + kWB * BK, wn * WTN, 1);
    __builtin_amdgcn_sched_barrier(0);
    // Raised wave priority while this step's MFMAs after the barrier and the
    // reads issue: of the two waves on a SIMD, the one past the barrier keeps
    // the matrix core fed while the other waits (measured: FWD2 -3 %, the
    // layer step -1 %).  PRE MFMAs before the barrier issue at the low priority.
    if constexpr (PRE == 0) __builtin_amdgcn_s_setprio(1);
    static_for<0, NMF>([&](auto mc) __attribute__((always_inline)) {
      constexpr int m = decltype(mc)::value;
      if constexpr (PRE > 0 && m == PRE) {
        __builtin_amdgcn_sched_barrier(0);
        sync();
        __builtin_amdgcn_s_setprio(1);
        __builtin_amdgcn_sched_barrier(0);
      }
      if constexpr (MMA) mfma_acc(acc[m / FN][m % FN], cb[m % FN], ca[m / FN]);
      static_for<0, NRD>([&](auto rc) __attribute__((always_inline)) {
        constexpr int r = decltype(rc)::value;
        if constexpr (m >= PRE && (r * RSPAN) / NRD == m - PRE) {
          if constexpr (r < NRA) {
            constexpr int imm = wide_read_imm<AK, r>();
            if constexpr (AK) rd128_issue_at<imm>(na[r], ra0);
            else rdtr_issue_at<imm>(qa[r], ((r >> 1) & 1) ? ra1 : ra0);
          } else {
            constexpr int rr = r - NRA;
            constexpr int imm = wide_read_imm<BKK, rr>();
            if constexpr (BKK) rd128_issue_at<imm>(nb[rr], rb0);
            else rdtr_issue_at<imm>(qb[rr], ((rr >> 1) & 1) ? rb1 : rb0);
          }
          if constexpr (r % 8 == 7 && r + 1 < NRD) lds_wait_le<7>();
        }
      });
      // The step's refills: the ragged-K (dW) products spread them over the
      // MFMAs after the barrier; the others issue them at the last MFMA
      // slots, after the fragment reads (measured: the dX call -18 us, the
      // forward -7 us on the 16384-token layer; the dW products +5 % that way).
      static_for<0, NDMA>([&](auto dc) __attribute__((always_inline)) {
        constexpr int d = decltype(dc)::value;
        constexpr int slot = RAGGED_K ? (d * (NMF - PRE)) / NDMA + 1 + PRE : NMF - NDMA - 1 + d;
        static_assert(slot > PRE, "refills follow the step's barrier");
        if constexpr (slot == m) {
          __builtin_amdgcn_sched_barrier(0);
          if constexpr (d & 1) opB.issue_r(d >> 1, rsb, kdma, dst + kWB * BK, wid);
          else opA.issue_r(d >> 1, rsa, kdma, dst, wid);
          __builtin_amdgcn_sched_barrier(0);
        }
      });
    });
    __builtin_amdgcn_s_setprio(0);
    lds_wait_all();
    if constexpr (AK) {
      lds_mark(na);
    } else {
      lds_mark(qa);
#pragma unroll
      for (int u = 0; u < FM; ++u) na[u] = u32x4{qa[2 * u][0], qa[2 * u][1], qa[2 * u + 1][0], qa[2 * u + 1][1]};
      valu_to_mfma_fence(na);
    }
    if constexpr (BKK) {
      lds_mark(nb);
    } else {
      lds_mark(qb);
#pragma unroll
      for (int u = 0; u < FN; ++u) nb[u] = u32x4{qb[2 * u][0], qb[2 * u][1], qb[2 * u + 1][0], qb[2 * u + 1][1]};
      valu_to_mfma_fence(nb);
    }
    __builtin_amdgcn_sched_barrier(0);
    if (more) advance();
    ++cs;
  };
  // Partial tile of a K-split remainder tile: stored to this block's slot in
  // accumulator order -- wave w, fragment (i, j), lane l at
  // ((w FM + i) FN + j) 64 + l -- for the fix-up kernel to add.
  // Fragment rows past the group's rows are not stored (the fix-up never
  // reads them).
  auto partial = [&](const WGeo& Cg) __attribute__((always_inline)) {
    asm volatile("s_nop 15\n s_nop 15" ::: "memory");   // last MFMA -> accumulator reads
    float* mine = p.part + (int64_t)blockIdx.x * (kWB * kWB) + ((int64_t)wid * FM * FN * 64 + lane) * 4;
    const int rows = Cg.Mlim - (Cg.m0 + wm * WTM);   // the wave's rows in the group (uniform)
    // One fragment row at a time (the pin orders each row's register moves
    // after the previous row's stores, so only a row is ever out of AGPRs).
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      acc_pin_mem(acc[i]);
      if (16 * i < rows) {
#pragma unroll
        for (int j = 0; j < FN; ++j) *reinterpret_cast<f32x4*>(mine + (i * FN + j) * 256) = acc[i][j];
      }
    }
  };

  auto run_steps_t = [&](int n, auto mmac) __attribute__((always_inline)) {
    int kk = 0;
    for (; kk + 2 <= n; kk += 2) {
      step(mmac, fa0, fb0, fa1, fb1);
      step(mmac, fa1, fb1, fa0, fb0);
    }
    if (kk < n) {   // odd step count: the next fragments are in set 1
      step(mmac, fa0, fb0, fa1, fb1);
#pragma unroll
      for (int u = 0; u < FM; ++u) fa0[u] = fa1[u];
#pragma unroll
      for (int u = 0; u < FN; ++u) fb0[u] = fb1[u];
      valu_to_mfma_fence(fa0);
      valu_to_mfma_fence(fb0);
    }
  };
  auto run_steps = [&](int n, bool mma) __attribute__((always_inline)) {
    if (mma) run_steps_t(n, std::true_type{});
    else run_steps_t(n, std::false_type{});
  };
  for (int e = 0; e < nseg; ++e) {
    int ct, k0, k1;
    seg(e, ct, k0, k1);
    const WGeo Cg = geo(ct);
    // Ragged-M: does the wave hold any of the group's rows in this tile?
    const bool mma = RAGGED_K || __builtin_amdgcn_readfirstlane((int)(Cg.m0 + wm * WTM < Cg.Mlim));
    if constexpr (SPLIT) {
      run_steps(e < nd ? Cg.nk : k1 - k0, mma);
      if (e < nd) epilogue(Cg);
      else partial(Cg);
    } else {
      run_steps(Cg.nk, mma);
      epilogue(Cg);
    }
    zero_acc();
    stores_pending = true;
  }
  wait_vm<0>();
}

// Adds the partial sums of the K-split remainder tiles -- in block order, so
// the result does not depend on timing -- and applies the epilogue.  Block b
// takes fragment row i = (b / 8) % FM of remainder tile (b / 8) / FM of XCD
// b % 8 (both waves rows of the tile's 2 x WGN wave grid), so a tile's sum is
// spread over FM blocks.  The schedule is recomputed exactly as the product
// made it (nslot blocks per XCD).
template <int NW, int EPI, int ACT, bool CBLK>
__global__ __launch_bounds__(NW * 64) void gemm_wide_fixup_kernel(GemmParams p, int tilesM, int tilesN, int groups,
                                                                   int nslot) {
  constexpr int WGN = NW / 2, WTM = 128, WTN = kWB / WGN, FM = WTM / 16, FN = WTN / 16;
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wid / WGN, wn = wid % WGN;
  const WPrefix P = wide_tile_prefix<false, true>(p, lane, groups, tilesM, tilesN);
  const int xcd = blockIdx.x % 8, q = (blockIdx.x / 8) / FM, i = (blockIdx.x / 8) % FM;
  const WRange XR = wide_range(P, xcd);
  const int nkU = (p.K + kBKb - 1) / kBKb;
  const WSched W = wide_sched(XR.nf + XR.np, nslot, p.ksplit != 0);
  if (!W.split || q >= W.r) return;
  const WGeo G = wide_geo<false, true>(p, XR.tile(W.R * nslot + q), lane, groups, P, tilesM, tilesN);
  // fragment row i of the wave's rows: nothing to add past the group's rows
  const bool live = 16 * i < G.Mlim - (G.m0 + wm * WTM);
  // the blocks of remainder tile q: [first, first + cnt); an empty K range wrote nothing
  int q0, first, cnt, k0, k1;
  W.split_part((q * nslot + W.r - 1) / W.r, nslot, nkU, q0, first, cnt, k0, k1);
  const int64_t lane_off = ((int64_t)wid * FM * FN * 64 + lane) * 4 + (int64_t)i * FN * 256;
  f32x4 sum[FN];
  bool any = false;
  for (int sl = first; sl < first + cnt; ++sl) {
    int qq, ff, cc, a0, a1;
    W.split_part(sl, nslot, nkU, qq, ff, cc, a0, a1);
    if (a0 >= a1 || !live) continue;
    const float* src = p.part + (int64_t)(sl * 8 + xcd) * (kWB * kWB) + lane_off;
    f32x4 v[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j) v[j] = *reinterpret_cast<const f32x4*>(src + j * 256);
#pragma unroll
    for (int j = 0; j < FN; ++j) sum[j] = any ? sum[j] + v[j] : v[j];
    any = true;
  }
  if (!any) {   // rows past the group, or an empty K range everywhere: nothing stored
#pragma unroll
    for (int j = 0; j < FN; ++j) sum[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  f32x4 acc[FM][FN];
  static_for<0, FM>([&](auto ic) {   // row i of acc (compile-time index), the others unused
    constexpr int I = decltype(ic)::value;
    if (I == i) {
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[I][j] = sum[j];
      wide_epilogue<FM, FN, WTM, WTN, false, EPI, ACT, CBLK>(p, G, acc, wm, wn, lane, I, I + 1);
    }
  });
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
constexpr int kSkMaxBlocks = 256;   // most blocks of a stream-K launch (partial slots per block: 2)
template <bool B_K, bool RAGGED_K, int EPI, int ACT, bool CBLK>
static void launch_wide(int groups, const GemmParams& p, int tilesM, int tilesN, hipStream_t s) {
  constexpr int S = B_K ? 4 : 5, NW = 8;
  constexpr size_t shmem = S * (size_t)(2 * kWB) * kBKb * sizeof(uint16_t);
  auto kern = gemm_wide_kernel<NW, S, B_K, RAGGED_K, EPI, ACT, CBLK>;
  static std::atomic<uint64_t> lds_ok{0};
  allow_dyn_lds((const void*)kern, (int)shmem, lds_ok);
  const int64_t max_tiles = (int64_t)tilesM * tilesN * groups;
  int blocks = num_cus();
  if (!RAGGED_K && blocks > kSkMaxBlocks) blocks = kSkMaxBlocks;   // partial slots in the workspace
  if (max_tiles < blocks) blocks = (int)max_tiles;
  blocks = (blocks + 7) / 8 * 8;
  hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(NW * 64), shmem, s, p, tilesM, tilesN, groups);
  if constexpr (!RAGGED_K && EPI == EPI_STORE) {
    const int nslot = blocks / 8;   // a K-split last round has at most nslot / 4 tiles per XCD
    constexpr int FM = 128 / 16;
    if (nslot >= 4 && p.ksplit)
      hipLaunchKernelGGL((gemm_wide_fixup_kernel<NW, EPI, ACT, CBLK>), dim3((unsigned)(8 * (nslot / 4) * FM)),
                         dim3(NW * 64), 0, s, p, tilesM, tilesN, groups, nslot);
  }
}

// Workspace of the ragged-M bf16 expert products: one partial 256 x 256 float
// tile per block, for a K-split last round.
static constexpr int64_t kSkPartBytes = (int64_t)kSkMaxBlocks * kWB * kWB * sizeof(float);
size_t expert_sk_ws_bytes(const moe_cfg& c) { return c.dtype == MOE_BF16 ? (size_t)kSkPartBytes : 0; }

// Expert products.  bf16: blocked operands, wide tiles; outputs that a later
// product reads (H, A, dH) blocked (CBLK), the others (expert_out, dXe, which
// only the gathers read, and the dW products) row-major.  float: the FMA
// kernel, row-major.
// rows: rows of the output per group (ragged-M: the capacity C, with up to 15
// alignment rows; ragged-K: M); cols: N.
template <bool B_K, bool RAGGED_K, int EPI, bool CBLK>
static void run_expert(const moe_cfg& c, const GemmParams& p, int64_t rows, int cols, hipStream_t s) {
  if (rows <= 0 || cols <= 0 || c.E <= 0) return;
  if (c.dtype != MOE_BF16) {
    dim3 grid((unsigned)((cols + 63) / 64), (unsigned)((rows + 63) / 64), (unsigned)c.E);
    if constexpr (EPI != EPI_RES) hipLaunchKernelGGL((gemm_f32_kernel<B_K, RAGGED_K, EPI>), grid, dim3(256), 0, s, p);
    return;
  }
  const int tm = (int)((rows + (RAGGED_K ? 0 : 15) + kWB - 1) / kWB), tn = (cols + kWB - 1) / kWB;
  if constexpr (EPI == EPI_STORE) {
    launch_wide<B_K, RAGGED_K, EPI, MOE_ACT_IDENTITY, CBLK>(c.E, p, tm, tn, s);
  } else {
    switch (c.act) {
      case MOE_ACT_RELU: launch_wide<B_K, RAGGED_K, EPI, MOE_ACT_RELU, CBLK>(c.E, p, tm, tn, s); break;
      case MOE_ACT_GELU_TANH: launch_wide<B_K, RAGGED_K, EPI, MOE_ACT_GELU_TANH, CBLK>(c.E, p, tm, tn, s); break;
      case MOE_ACT_GELU_ERF: launch_wide<B_K, RAGGED_K, EPI, MOE_ACT_GELU_ERF, CBLK>(c.E, p, tm, tn, s); break;
      default: launch_wide<B_K, RAGGED_K, EPI, MOE_ACT_IDENTITY, CBLK>(c.E, p, tm, tn, s); break;
    }
  }
}

// Rows per expert block of an [E][C][*] buffer (C rounded up to 16 for bf16).
static int64_t rows_alloc(const moe_cfg& c) { return c.dtype == MOE_BF16 ? pad16(c.C) : c.C; }

// Per-product timing (moe_product_timing): while on, each expert product
// launch of this thread is bracketed by a pair of events on its stream (the
// K-split fix-up launch inside the pair); product_times sums them per product.
namespace {
struct ProductTimer {
  bool on = false;
  int dev = -1;
  bool failed = false;
  std::vector<hipEvent_t> pool;      // events of this device, reused after each readout
  size_t next = 0;
  std::vector<std::pair<int, size_t>> rec;   // (product, index of its first event)
};
thread_local ProductTimer g_ptimer;

hipEvent_t ptimer_event() {
  ProductTimer& t = g_ptimer;
  if (t.next == t.pool.size()) {
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) {
      t.failed = true;
      return nullptr;
    }
    t.pool.push_back(e);
  }
  return t.pool[t.next++];
}
// Records the opening event of product `prod` on s; returns false when timing is off.
bool ptimer_begin(int prod, hipStream_t s) {
  ProductTimer& t = g_ptimer;
  if (!t.on) return false;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev != t.dev) {   // events belong to the device timing was started on
    t.failed = true;
    return false;
  }
  const size_t i = t.next;
  hipEvent_t a = ptimer_event(), b = ptimer_event();
  if (!a || !b || hipEventRecord(a, s) != hipSuccess) {
    t.failed = true;
    return false;
  }
  t.rec.push_back({prod, i});
  return true;
}
void ptimer_end(bool begun, hipStream_t s) {
  if (!begun) return;
  ProductTimer& t = g_ptimer;
  if (hipEventRecord(t.pool[t.rec.back().second + 1], s) != hipSuccess) t.failed = true;
}
}  // namespace

hipError_t product_timing(bool on) {
  ProductTimer& t = g_ptimer;
  int dev = 0;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev != t.dev) {   // a different device: the pool's events belong to the old one (left, not destroyed)
    t.pool.clear();
    t.dev = dev;
  }
  t.on = on;
  t.failed = false;
  t.next = 0;
  t.rec.clear();
  return hipSuccess;
}

hipError_t product_times(double* ms, int32_t* counts) {
  ProductTimer& t = g_ptimer;
  for (int q = 0; q < kProducts; ++q) {
    ms[q] = 0.0;
    counts[q] = 0;
  }
  if (t.failed) return hipErrorUnknown;
  for (const auto& r : t.rec) {
    hipError_t e = hipEventSynchronize(t.pool[r.second + 1]);
    float v = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&v, t.pool[r.second], t.pool[r.second + 1]);
    if (e != hipSuccess) return e;
    ms[r.first] += v;
    counts[r.first] += 1;
  }
  t.next = 0;
  t.rec.clear();
  return hipSuccess;
}

void launch_expert_fwd(const moe_cfg& c, const void* X, const int32_t* rb, const int32_t* re, const void* W1,
                       const void* W2, void* H, void* A, void* O, void* ws, hipStream_t s) {
  const int64_t d = c.d_model, f = c.d_ff, C = c.C, Cp = rows_alloc(c);
  GemmParams p1{X, d, Cp * d, W1, d, f * d, H, f, Cp * f, A, nullptr, rb, re, 0, (int)f, (int)d, c.act, (int)C};
  p1.part = (float*)ws;
  p1.ksplit = c.ksplit;
  bool tb = ptimer_begin(kProdFwd1, s);
  run_expert<true, false, EPI_FWD1, true>(c, p1, C, (int)f, s);
  ptimer_end(tb, s);
  GemmParams p2{A, f, Cp * f, W2, f, d * f, O, d, Cp * d, nullptr, nullptr, rb, re, 0, (int)d, (int)f, c.act, (int)C};
  p2.part = (float*)ws;
  p2.ksplit = c.ksplit;
  tb = ptimer_begin(kProdFwd2, s);
  run_expert<true, false, EPI_STORE, false>(c, p2, C, (int)d, s);   // expert_out row-major
  ptimer_end(tb, s);
}

void launch_expert_bwd_dx(const moe_cfg& c, const void* dO, const int32_t* rb, const int32_t* re, const void* H,
                          const void* W1, const void* W2, void* dH, void* dXe, void* ws, hipStream_t s) {
  const int64_t d = c.d_model, f = c.d_ff, C = c.C, Cp = rows_alloc(c);
  // dA = dO W2_e  (B(k=i, n=j) = W2[e][i][j], N contiguous), epilogue dH = dA * act'(H)
  GemmParams p1{dO, d, Cp * d, W2, f, d * f, dH, f, Cp * f, nullptr, H, rb, re, 0, (int)f, (int)d, c.act, (int)C};
  p1.part = (float*)ws;
  p1.ksplit = c.ksplit;
  bool tb = ptimer_begin(kProdDA, s);
  run_expert<false, false, EPI_DACT, true>(c, p1, C, (int)f, s);
  ptimer_end(tb, s);
  // dXe = dH W1_e  (B(k=i, n=j) = W1[e][i][j])
  GemmParams p2{dH, f, Cp * f, W1, d, f * d, dXe, d, Cp * d, nullptr, nullptr, rb, re, 0, (int)d, (int)f, c.act, (int)C};
  p2.part = (float*)ws;
  p2.ksplit = c.ksplit;
  tb = ptimer_begin(kProdDXe, s);
  run_expert<false, false, EPI_STORE, false>(c, p2, C, (int)d, s);   // dXe row-major
  ptimer_end(tb, s);
}

void launch_expert_bwd_dw(const moe_cfg& c, const void* X, const void* A, const void* dO, const void* dH,
                          const int32_t* rb, const int32_t* re, void* dW1, void* dW2, hipStream_t s) {
  const int64_t d = c.d_model, f = c.d_ff, C = c.C, Cp = rows_alloc(c);
  // dW2_e [d][f] = dO_e^T A_e : A-operand(m, k) = dO[e][k][m], B(k, n) = A[e][k][n]
  // (wpacked: written in the blocked layout of the packed weights)
  GemmParams p2{dO, d, Cp * d, A, f, Cp * f, dW2, f, d * f, nullptr, nullptr, rb, re, (int)d, (int)f, 0, c.act, (int)C};
  // dW1_e [f][d] = dH_e^T X_e
  GemmParams p1{dH, f, Cp * f, X, d, Cp * d, dW1, d, f * d, nullptr, nullptr, rb, re, (int)f, (int)d, 0, c.act, (int)C};
  const bool blk = c.wpacked && c.dtype == MOE_BF16;
  bool tb = ptimer_begin(kProdDW2, s);
  if (blk) run_expert<false, true, EPI_STORE, true>(c, p2, d, (int)f, s);
  else run_expert<false, true, EPI_STORE, false>(c, p2, d, (int)f, s);
  ptimer_end(tb, s);
  tb = ptimer_begin(kProdDW1, s);
  if (blk) run_expert<false, true, EPI_STORE, true>(c, p1, f, (int)d, s);
  else run_expert<false, true, EPI_STORE, false>(c, p1, f, (int)d, s);
  ptimer_end(tb, s);
}

// Sum of the S float partials of a K-split weight gradient, in group order,
// rounded once to bf16: 8 consecutive elements per thread.
__global__ __launch_bounds__(256) void gemm_wgrad_reduce_kernel(const float* __restrict__ part, int S, int64_t MN,
                                                                 uint16_t* __restrict__ C) {
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 8;
  if (i >= MN) return;
  f32x4 a0 = *reinterpret_cast<const f32x4*>(part + i), a1 = *reinterpret_cast<const f32x4*>(part + i + 4);
  for (int g = 1; g < S; ++g) {
    a0 += *reinterpret_cast<const f32x4*>(part + (int64_t)g * MN + i);
    a1 += *reinterpret_cast<const f32x4*>(part + (int64_t)g * MN + i + 4);
  }
  const float v0[4] = {a0[0], a0[1], a0[2], a0[3]}, v1[4] = {a1[0], a1[1], a1[2], a1[3]};
  const u32x2 lo = pack4_bf16(v0), hi = pack4_bf16(v1);
  *reinterpret_cast<u32x4*>(C + i) = u32x4{lo[0], lo[1], hi[0], hi[1]};
}

// Token ranges of the dense weight gradients: the block's 2048 x 2048 and
// 6144 x 2048 products have 64 and 192 tiles of 256 x 256, so four ranges give
// every CU work (256 and 768 tile-ranges).
constexpr int kWgradSplit = 4;
size_t wgrad_ws_bytes(int M, int N) { return (size_t)kWgradSplit * M * N * sizeof(float); }

// Weight gradient C[M][N] = A^T B of the block's dense projections, A [K][M]
// and B [K][N] row-major bf16 (K = tokens), C bf16: the wide kernel's ragged-K
// product with K split into wgrad_ksplit(M, N) token ranges of equal length
// (multiples of 32), one float partial per range in `part`
// (wgrad_ws_bytes(M, N) bytes), then their sum in range order.
void launch_dense_wgrad(int M, int N, int64_t K, const void* A, const void* B, void* C, void* part, hipStream_t s) {
  if (M <= 0 || N <= 0) return;
  const int S = kWgradSplit;
  const int64_t MN = (int64_t)M * N;
  GemmParams p{A, M, 0, B, N, 0, part, N, MN, nullptr, nullptr, nullptr, nullptr, M, N, 0, 0, (int)K};
  p.kchunk = (int)(((K + S - 1) / S + 31) / 32 * 32);
  launch_wide<false, true, EPI_WGF32, MOE_ACT_IDENTITY, false>(S, p, (M + kWB - 1) / kWB, (N + kWB - 1) / kWB, s);
  hipLaunchKernelGGL(gemm_wgrad_reduce_kernel, dim3((unsigned)((MN / 8 + 255) / 256)), dim3(256), 0, s,
                     (const float*)part, S, MN, (uint16_t*)C);
}

// Row-major [M][K] bf16 -> the blocked layout with pad16(M) rows (rows past M
// zero).  One wave per 16 x 32 block: each lane reads 16 bytes of one row and
// the wave writes the block's 1 KiB as one contiguous run.
__global__ __launch_bounds__(256) void pack_rows_kernel(const uint16_t* __restrict__ src, uint16_t* __restrict__ dst,
                                                        int64_t M, int K) {
  const int64_t b = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int lane = threadIdx.x & 63;
  const int kb = K >> 5;
  const int64_t rb = b / kb;
  if (rb * 16 >= pad16(M)) return;
  const int cb = (int)(b - rb * kb);
  const int64_t row = rb * 16 + (lane >> 2);
  const int col = cb * 32 + (lane & 3) * 8;
  u32x4 v = u32x4{0u, 0u, 0u, 0u};
  if (row < M) v = *reinterpret_cast<const u32x4*>(src + row * K + col);
  *reinterpret_cast<u32x4*>(dst + b * 512 + lane * 8) = v;
}

void launch_pack_rows(const void* src, void* dst, int64_t M, int K, hipStream_t s) {
  if (M <= 0 || K <= 0) return;
  const int64_t blocks = pad16(M) / 16 * (K / 32);
  hipLaunchKernelGGL(pack_rows_kernel, dim3((unsigned)((blocks * 64 + 255) / 256)), dim3(256), 0, s,
                     (const uint16_t*)src, (uint16_t*)dst, M, K);
}

// Dense products on the wide MFMA kernel: one group of M rows, both operands
// blocked (A [pad16(M)][K]; B [N][K] if b_nk else [K][N]), output row-major,
// + resid (row-major like C) if given.  Every output element is one in-order
// K sum (no K-split), so a product over a batch partition's rows gives the
// same bits as over the whole batch.
void launch_dense_wide(int64_t M, int N, int K, const void* A, const void* B, bool b_nk, void* C, int64_t ldc,
                       const void* resid, hipStream_t s) {
  if (M <= 0 || N <= 0 || K <= 0) return;
  GemmParams p{A, K, pad16(M) * K, B, b_nk ? K : N, (int64_t)N * K, C, ldc, M * ldc, nullptr, resid, nullptr, nullptr,
               0, N, K, 0, (int)M};
  p.ksplit = 0;
  const int tm = (int)((M + 15 + kWB - 1) / kWB), tn = (N + kWB - 1) / kWB;
  if (b_nk) {
    if (resid) launch_wide<true, false, EPI_RES, MOE_ACT_IDENTITY, false>(1, p, tm, tn, s);
    else launch_wide<true, false, EPI_STORE, MOE_ACT_IDENTITY, false>(1, p, tm, tn, s);
  } else {
    if (resid) launch_wide<false, false, EPI_RES, MOE_ACT_IDENTITY, false>(1, p, tm, tn, s);
    else launch_wide<false, false, EPI_STORE, MOE_ACT_IDENTITY, false>(1, p, tm, tn, s);
  }
}

}  // namespace lmoe
