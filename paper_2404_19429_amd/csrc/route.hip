// Capacity-bounded slot assignment, dispatch (scatter), combine (weighted
// gather) and their backward counterparts, plus the gate's weight gradient.
//
// Slot assignment walks assignments token by token, rank by rank; the row an
// assignment receives is carry_e plus the number of earlier assignments to
// the same expert.  It is computed without order-defining atomics in three
// launches: in-chunk ranks and per-chunk expert histograms (wavefront
// ballots), a per-expert exclusive scan over chunks (starting at carry, which
// makes batch partitions exact), and a final pass that adds the chunk base to
// each rank, applies the capacity and copies the kept rows with 16-byte
// vector accesses, one thread per (token, 16-byte column chunk).
#include <mutex>
#include <type_traits>

#include "internal.h"

namespace lmoe {

// Element offset of (expert e, row s, column col) in an [E][C][d] buffer that
// the expert products read (send_buf, dO): blocked for bf16 (rows padded to
// 16), row-major for float.
template <typename T>
__device__ __forceinline__ int64_t eoff(int e, int s, int col, int d, int C) {
  const int64_t rows = sizeof(T) == 2 ? pad16(C) : C;
  return (int64_t)e * rows * d + ebuf_off<T>(s, col, d);
}
// The same for the row-major product outputs (expert_out, dXe).
template <typename T>
__device__ __forceinline__ int64_t erow(int e, int s, int col, int d, int C) {
  const int64_t rows = sizeof(T) == 2 ? pad16(C) : C;
  return ((int64_t)e * rows + s) * d + col;
}

// ------------------------------------------------------------ slot assignment
// For every assignment (t, r) of a chunk: rank[t][r] = assignments to the same
// expert earlier in (token, rank) order inside the chunk; counts[chunk][e] =
// the chunk's assignments to e.  Lanes holding the same expert are found with
// one ballot per expert-index bit.
// perm (nullable): position j of the walk holds token perm[j] (batch-prioritized
// order); NULL = token order.  rank_out and the chunks are indexed by position.
__global__ __launch_bounds__(kRouteChunk) void route_rank_kernel(const int32_t* __restrict__ idx,
                                                                 const int32_t* __restrict__ perm,
                                                                 int32_t* __restrict__ counts,
                                                                 int32_t* __restrict__ rank_out,
                                                                 int64_t T_tokens, int E, int k) {
  constexpr int NW = kRouteChunk / kWave;
  __shared__ int32_t wcnt[NW][kMaxE];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  for (int i = threadIdx.x; i < NW * kMaxE; i += blockDim.x) (&wcnt[0][0])[i] = 0;
  __syncthreads();

  const int64_t t = (int64_t)blockIdx.x * kRouteChunk + threadIdx.x;
  const bool active = t < T_tokens;
  int64_t tok = t;
  if (active && perm) {
    tok = perm[t];
    if (tok < 0 || tok >= T_tokens) tok = t;   // (a valid order is a permutation of 0 .. T-1)
  }
  int my[kMaxK], rank[kMaxK];
#pragma unroll
  for (int r = 0; r < kMaxK; ++r) {
    const int e = (active && r < k) ? idx[tok * k + r] : -1;
    my[r] = (e >= 0 && e < E) ? e : -1;  // an out-of-range expert is treated as dropped
    rank[r] = 0;
  }
  // Earlier choices of the same token (only if a row repeats an expert).
#pragma unroll
  for (int r = 1; r < kMaxK; ++r)
#pragma unroll
    for (int q = 0; q < r; ++q) rank[r] += (my[r] >= 0 && my[q] == my[r]) ? 1 : 0;

  // Round rp: the bit masks of every lane's rp-th choice let each lane count,
  // for each of its own choices, the lower lanes whose rp-th choice matches.
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
  for (int rp = 0; rp < kMaxK; ++rp) {
    if (rp >= k) break;
    const int v = my[rp];
    const uint64_t valid = __ballot(v >= 0);
    uint64_t mb[6];
#pragma unroll
    for (int b = 0; b < 6; ++b) mb[b] = __ballot(v >= 0 && ((v >> b) & 1));
    auto holders = [&](int e) __attribute__((always_inline)) {   // lanes whose rp-th choice is e
      uint64_t m = valid;
#pragma unroll
      for (int b = 0; b < 6; ++b) m &= ((e >> b) & 1) ? mb[b] : ~mb[b];
      return m;
    };
#pragma unroll
    for (int r = 0; r < kMaxK; ++r)
      if (r < k && my[r] >= 0) rank[r] += __popcll(holders(my[r]) & lt);
    if (v >= 0) {
      const uint64_t peers = holders(v);
      if ((peers & lt) == 0) wcnt[wave][v] += __popcll(peers);  // one leader per expert
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < E; e += blockDim.x) {
    int n = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) n += wcnt[w][e];
    counts[(int64_t)blockIdx.x * E + e] = n;
  }
  if (!active) return;
#pragma unroll
  for (int r = 0; r < kMaxK; ++r) {
    if (r < k) {
      const int e = my[r];
      int s = -1;
      if (e >= 0) {
        s = rank[r];
        for (int w = 0; w < wave; ++w) s += wcnt[w][e];
      }
      rank_out[t * k + r] = s;
    }
  }
}

// base[chunk][e] = carry_e + assignments to e in earlier chunks; fill_e = min(C, carry_e + all).
// One wave per expert (grid = E).
__global__ __launch_bounds__(64) void route_scan_kernel(const int32_t* __restrict__ counts,
                                                        int32_t* __restrict__ base,
                                                        const int32_t* __restrict__ carry,
                                                        int32_t* __restrict__ fill, int nchunks, int E, int C) {
  const int lane = threadIdx.x;
  const int e = blockIdx.x;
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

// Row kernels (dispatch copy, combine, dispatch backward) give each thread one
// 16-byte column chunk of U tokens and issue every load of those tokens
// before any store, so a thread keeps U * k row loads in flight.  KT is the
// top-k as a constant (0: a runtime k up to kMaxK, with U = 1).

// slot[t][r] = base[chunk][e] + rank (or -1 past the capacity), and
// send_buf[e][slot][:] = x[t][:] for every kept (t, r).
// perm as in route_rank_kernel: the thread's positions j hold tokens perm[j].
// nfused > 0 (wave-uniform tokens, at most 64 chunks): the chunk bases are
// not read from `base` but summed here from the chunk counts (one wave
// reduction per token and choice; the scan launch is skipped), and the first
// wave of block b writes fill[e] = min(C, carry_e + all counts of e) for
// e = b, b + gridDim.x, ...
template <typename T, int KT, int U, bool UNI>
__global__ __launch_bounds__(256) void dispatch_copy_kernel(const T* __restrict__ x, const int32_t* __restrict__ idx,
                                                            const int32_t* __restrict__ perm,
                                                            const int32_t* __restrict__ rank,
                                                            const int32_t* __restrict__ base,
                                                            int32_t* __restrict__ slot, T* __restrict__ send,
                                                            int64_t T_tokens, int d, int E, int kr, int C,
                                                            const int32_t* __restrict__ counts,
                                                            const int32_t* __restrict__ carry,
                                                            int32_t* __restrict__ fill, int nfused) {
  constexpr int V = Vec<T>::N;
  constexpr int KK = KT > 0 ? KT : kMaxK;
  const int k = KT > 0 ? KT : kr;
  const int nc = d / V;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t g = UNI ? (int64_t)__builtin_amdgcn_readfirstlane((int)(gid / nc)) : gid / nc;
  const int c = (int)(gid - g * nc);
  const int64_t t0 = g * U;
  const int lane = threadIdx.x & 63;
  // Sum over the first n chunks of expert e's counts (wave-uniform n and e, n <= 64).
  auto counts_before = [&](int n, int e) __attribute__((always_inline)) {
    int v = lane < n ? counts[(int64_t)lane * E + e] : 0;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
  };
  if (nfused > 0 && threadIdx.x < kWave) {
    for (int e = blockIdx.x; e < E; e += gridDim.x) {
      const int tot = (carry ? carry[e] : 0) + counts_before(nfused, e);
      if (lane == 0) fill[e] = tot < C ? tot : C;
    }
  }
  if (t0 >= T_tokens) return;
  u32x4 v[U];
  int er[U][KK], sr[U][KK];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t j = t0 + u;                 // position of the walk
    const bool tok = j < T_tokens;
    int64_t t = j;
    if (tok && perm) {
      t = perm[j];
      if (t < 0 || t >= T_tokens) t = j;       // (a valid order is a permutation of 0 .. T-1)
    }
    v[u] = tok ? *reinterpret_cast<const u32x4*>(x + t * d + (int64_t)c * V) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int r = 0; r < KK; ++r) {
      er[u][r] = -1;
      sr[u][r] = -1;
      if (tok && r < k) {
        const int e = idx[t * k + r];
        const int rk = rank[j * k + r];
        if (rk >= 0 && e >= 0 && e < E) {
          const int sl = (UNI && nfused > 0 ? (carry ? carry[e] : 0) + counts_before((int)(j / kRouteChunk), e)
                                            : base[(j / kRouteChunk) * E + e]) + rk;
          if (sl < C) {
            er[u][r] = e;
            sr[u][r] = sl;
          }
        }
        if (c == 0) slot[t * k + r] = sr[u][r];
      }
    }
  }
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int r = 0; r < KK; ++r)
      if (sr[u][r] >= 0) *reinterpret_cast<u32x4*>(send + eoff<T>(er[u][r], sr[u][r], c * V, d, C)) = v[u];
}

// Launch a row kernel F::kernel<T, KT, U> over T tokens: one thread per
// (group of U tokens, 16-byte chunk).
// U1 / U2: tokens per thread for top-1 / top-2.  When a row is a multiple of
// 64 chunks, every lane of a wave works on the same tokens: the token index
// is made wave-uniform (UNI), so the tokens' idx / slot / w come through
// scalar loads.
template <template <typename, int, int, bool> class F, typename T, int U1, int U2, typename... Args>
static void row_launch(const moe_cfg& c, hipStream_t s, Args... args) {
  const int nc = c.d_model / Vec<T>::N;
  auto go = [&](auto kern, int U) {
    const int64_t n = (c.T + U - 1) / U * nc;
    hipLaunchKernelGGL(kern, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, args...);
  };
  const bool uni = nc % kWave == 0 && c.T < ((int64_t)1 << 30);
  auto pick = [&](auto ucst) {
    constexpr bool UNI = decltype(ucst)::value;
    if (c.k == 1) go(F<T, 1, U1, UNI>::kernel(), U1);
    else if (c.k == 2) go(F<T, 2, U2, UNI>::kernel(), U2);
    else go(F<T, 0, 1, UNI>::kernel(), 1);
  };
  if (uni) pick(std::true_type{});
  else pick(std::false_type{});
}
template <typename T, int KT, int U, bool UNI> struct DispatchCopy {
  static constexpr auto kernel() { return dispatch_copy_kernel<T, KT, U, UNI>; }
};

size_t dispatch_ws_bytes(const moe_cfg& c) {
  const int64_t nch = (c.T + kRouteChunk - 1) / kRouteChunk;
  return (size_t)(2 * nch * c.E + c.T * c.k) * sizeof(int32_t);
}

// Slot assignment and copy over the walk order perm (NULL = token order).
static void dispatch_walk(const moe_cfg& c, const void* x, const int32_t* idx, const int32_t* perm,
                          const int32_t* carry, int32_t* fill, int32_t* slot, void* send_buf, void* ws, hipStream_t s) {
  const int64_t nch = (c.T + kRouteChunk - 1) / kRouteChunk;
  int32_t* counts = (int32_t*)ws;
  int32_t* base = counts + nch * c.E;
  int32_t* rank = base + nch * c.E;
  // The copy launch sums the chunk bases itself when its waves are token-uniform
  // (as row_launch decides) and there are at most 64 chunks (one count per
  // lane); else a scan launch (with 128 chunks the in-copy sums cost more than
  // the launch they save).
  const int V = c.dtype == MOE_BF16 ? 8 : 4;
  const bool fused = nch > 0 && nch <= kWave && (c.d_model / V) % kWave == 0 && c.T < ((int64_t)1 << 30);
  const int nfused = fused ? (int)nch : 0;
  if (nch > 0)
    hipLaunchKernelGGL(route_rank_kernel, dim3((unsigned)nch), dim3(kRouteChunk), 0, s, idx, perm, counts, rank, c.T,
                       c.E, c.k);
  if (c.E > 0 && !fused)
    hipLaunchKernelGGL(route_scan_kernel, dim3((unsigned)c.E), dim3(64), 0, s, counts, base, carry, fill, (int)nch, c.E,
                       c.C);
  if (nch == 0) return;
  if (c.dtype == MOE_BF16)
    row_launch<DispatchCopy, uint16_t, 4, 2>(c, s, (const uint16_t*)x, idx, perm, rank, (const int32_t*)base, slot,
                                       (uint16_t*)send_buf, c.T, c.d_model, c.E, c.k, c.C, (const int32_t*)counts,
                                       carry, fill, nfused);
  else
    row_launch<DispatchCopy, float, 4, 2>(c, s, (const float*)x, idx, perm, rank, (const int32_t*)base, slot,
                                    (float*)send_buf, c.T, c.d_model, c.E, c.k, c.C, (const int32_t*)counts, carry,
                                    fill, nfused);
}

void launch_dispatch(const moe_cfg& c, const void* x, const int32_t* idx, const int32_t* carry, int32_t* fill,
                     int32_t* slot, void* send_buf, void* ws, hipStream_t s) {
  dispatch_walk(c, x, idx, nullptr, carry, fill, slot, send_buf, ws, s);
}

// ------------------------------------------- dispatch without caller workspace
// The workspace of moe_dispatch_noalloc: one file-scope device array, which
// every GPU the library runs on holds for the life of the process.  Host code
// never passes the array's name to a kernel (on the host it only stands in
// for the symbol); it takes the array's device address on each device once,
// with that device current, and uses that address from then on.
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_ptr[64];   // device address of `scratch` on device i (null until first use)
}  // namespace

hipError_t noalloc_scratch(void** out) {
  *out = nullptr;
  const int dev = current_device();
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

// ------------------------------------------------------ batch-prioritized routing
// The tokens are visited by importance (the sum of the selected experts'
// softmax probabilities) descending, equal importance in token order; the
// capacity rule then runs over that walk exactly as over token order.

// elem[t] = (key << 32) | t, key = ~bits of the float importance (ascending
// key = descending importance; importance >= 0), so the 64-bit elements are
// distinct and their ascending order is the visiting order: importance
// descending, then token ascending.  One wave per token, lane e for
// expert e: the softmax over all E experts in double, then the selected
// experts' probabilities summed in rank order, rounded once to float; the
// ordering decision is taken on the float values.
__global__ __launch_bounds__(256) void bpr_key_kernel(const float* __restrict__ logits, const int32_t* __restrict__ idx,
                                                      uint64_t* __restrict__ elem, int64_t T_tokens, int E, int k) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x >> 6);
  if (t >= T_tokens) return;
  const bool has = lane < E;
  const float l = has ? logits[t * E + lane] : -INFINITY;
  float mf = l;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mf = fmaxf(mf, __shfl_xor(mf, o, kWave));
  const double ex = has ? exp((double)l - (double)mf) : 0.0;
  double z = ex;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) z += __shfl_xor(z, o, kWave);
  const double p = ex / z;
  double imp = 0.0;
  for (int r = 0; r < k; ++r) {
    const int e = idx[t * k + r];
    const double pe = __shfl(p, (e >= 0 && e < E) ? e : 0, kWave);
    if (e >= 0 && e < E) imp += pe;
  }
  if (lane == 0) elem[t] = ((uint64_t)~__float_as_uint((float)imp) << 32) | (uint64_t)t;
}

constexpr int kSortThreads = 1024;
constexpr int kSortWaves = kSortThreads / kWave;
constexpr int kDigitBits = 8;
constexpr int kRadix = 1 << kDigitBits;
constexpr int kSortPasses = 4;             // the key's low 30 bits: digits of 8, 8, 8, 6 bits
constexpr int kCntStride = kSortWaves + 1; // counters of one digit (one per wave), padded
constexpr int kSortTile = 4096;            // elements per sorted tile: 16 waves x 4 rounds of 64
constexpr int kWaveSpan = kSortTile / kSortWaves;
constexpr size_t kTileSortLds = 2 * kSortTile * sizeof(uint64_t) + kSortWaves * kRadix * sizeof(uint64_t) +
                                (kRadix * kCntStride + kSortWaves) * sizeof(int32_t);
static_assert(kRadix * kSortWaves == 4 * kSortThreads, "scan layout");

// Sorts one tile of up to kSortTile elements in LDS by the key's low 30 bits
// (importance keys: ~bits of a float in [0, 1], whose two top bits are
// constant), stably: an LSD radix sort of four passes.  Wave w owns elements
// [w kWaveSpan, (w + 1) kWaveSpan) of the tile and takes them in rounds of
// 64 in order; cnt[digit][w] counts the digit in w's range, and its
// exclusive prefix in (digit, wave) order is where w's next element with
// that digit goes.  In a round, each lane ORs its lane bit into the wave's
// table entry of its digit and reads the entry back: the lanes sharing its
// digit.  They are ranked by lane, and the lowest of them claims their
// positions with one returning LDS add and clears the entry (a wave's LDS
// operations complete in order, so the rounds claim in order).  Equal keys
// keep their input order, which within a tile is token order: the sorted
// tile is in ascending order of the 64-bit elements.
// Lanes of a round by digit when the round holds at most two digits: m0 =
// the active lanes with the first active lane's digit (returned), m1 = the
// other active lanes if they all share one digit, rest = any active lanes
// left (nonzero: more than two digits; m1 then means nothing).
__device__ __forceinline__ int few_digits(int dg, bool ok, uint64_t& m0, uint64_t& m1, uint64_t& rest) {
  const uint64_t act = __ballot(ok);
  if (act == 0) {
    m0 = m1 = rest = 0ull;
    return 0;
  }
  const int d0 = __builtin_amdgcn_readlane(dg, (int)__builtin_ctzll(act));
  m0 = __ballot(ok && dg == d0);
  const uint64_t r = act & ~m0;
  if (r == 0) {
    m1 = rest = 0ull;
    return d0;
  }
  const int d1 = __builtin_amdgcn_readlane(dg, (int)__builtin_ctzll(r));
  m1 = __ballot(ok && dg == d1);
  rest = r & ~m1;
  return d0;
}

constexpr int kSplStep = 64;                          // a splitter every 64 sorted elements
constexpr int kSplPerTile = kSortTile / kSplStep;
__global__ __launch_bounds__(kSortThreads) void bpr_tile_sort_kernel(const uint64_t* __restrict__ in,
                                                                     uint64_t* __restrict__ out,
                                                                     uint64_t* __restrict__ spl, int64_t n) {
  extern __shared__ __attribute__((aligned(16))) unsigned char bpr_lds[];
  uint64_t* buf0 = reinterpret_cast<uint64_t*>(bpr_lds);
  uint64_t* buf1 = buf0 + kSortTile;
  uint64_t* table = buf1 + kSortTile;                                  // [kSortWaves][kRadix]
  int32_t* cnt = reinterpret_cast<int32_t*>(table + kSortWaves * kRadix);   // [kRadix][kCntStride]
  int32_t* wsum = cnt + kRadix * kCntStride;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t t0 = (int64_t)blockIdx.x * kSortTile;
  const int m = (int)min((int64_t)kSortTile, n - t0);
  for (int i = tid; i < m; i += kSortThreads) buf0[i] = in[t0 + i];
  for (int i = lane; i < kRadix; i += kWave) table[wave * kRadix + i] = 0ull;
  const int lo = min(m, wave * kWaveSpan), hi = min(m, lo + kWaveSpan);
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int pass = 0; pass < kSortPasses; ++pass) {
    const int sh = 32 + kDigitBits * pass;
    const uint32_t dmask = pass == kSortPasses - 1 ? 0x3fu : 0xffu;
    const uint64_t* src = (pass & 1) ? buf1 : buf0;   // 0 -> 1 -> 0 -> 1 -> 0
    uint64_t* dst = (pass & 1) ? buf0 : buf1;
    for (int i = tid; i < kRadix * kCntStride; i += kSortThreads) cnt[i] = 0;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kWaveSpan / kWave; ++j) {
      const int i = lo + kWave * j + lane;
      const bool ok = i < hi;
      const int dg = ok ? (int)((src[i] >> sh) & dmask) : 0;
      // A round with at most two digits (the high digits of nearby importances)
      // is counted by one lane per digit; otherwise one LDS add per lane.
      uint64_t m0, m1, rest;
      const int d0 = few_digits(dg, ok, m0, m1, rest);
      if (rest == 0) {
        if (m0 != 0 && lane == (int)__builtin_ctzll(m0)) atomicAdd(&cnt[d0 * kCntStride + wave], __popcll(m0));
        if (m1 != 0 && lane == (int)__builtin_ctzll(m1)) atomicAdd(&cnt[dg * kCntStride + wave], __popcll(m1));
      } else if (ok) {
        atomicAdd(&cnt[dg * kCntStride + wave], 1);
      }
    }
    __syncthreads();
    // Exclusive scan of the counters in (digit, wave) order; thread tid owns
    // digit tid / 4, waves 4 (tid % 4) .. + 3.
    const int d0 = tid >> 2, w0 = (tid & 3) * 4;
    int v[4];
    int sum = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      v[q] = cnt[d0 * kCntStride + w0 + q];
      sum += v[q];
    }
    int incl = sum;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int u = __shfl_up(incl, o, kWave);
      if (lane >= o) incl += u;
    }
    if (lane == kWave - 1) wsum[wave] = incl;
    __syncthreads();
    int ex = incl - sum;
    for (int w = 0; w < wave; ++w) ex += wsum[w];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      cnt[d0 * kCntStride + w0 + q] = ex;
      ex += v[q];
    }
    __syncthreads();
    constexpr int NR = kWaveSpan / kWave;
    uint64_t el[NR];
#pragma unroll
    for (int j = 0; j < NR; ++j) {   // the wave's elements of the pass, read up front
      const int i = lo + kWave * j + lane;
      el[j] = i < hi ? src[i] : 0ull;
    }
#pragma unroll
    for (int j = 0; j < NR; ++j) {
      // One LDS round trip per round: OR the lane bit into the digit's table
      // entry, then read the entry (the lanes sharing the digit) and the
      // digit's running position together; the lowest of those lanes then
      // advances the position and clears the entry.  A wave's LDS operations
      // complete in order, so every lane's reads precede the leader's writes.
      const bool ok = lo + kWave * j + lane < hi;
      const uint64_t e = el[j];
      const int dg = (int)((e >> sh) & dmask);
      uint64_t m0, m1, rest;
      few_digits(dg, ok, m0, m1, rest);
      uint64_t peers = 0ull;
      int base = 0;
      if (rest == 0) {   // at most two digits: the lanes sharing a digit are a ballot
        peers = ok ? (((m0 >> lane) & 1) ? m0 : m1) : 0ull;
        if (ok) base = cnt[dg * kCntStride + wave];
      } else if (ok) {
        atomicOr((unsigned long long*)&table[wave * kRadix + dg], (unsigned long long)(1ull << lane));
        peers = table[wave * kRadix + dg];
        base = cnt[dg * kCntStride + wave];
      }
      const int pos = base + __popcll(peers & lt);
      if (ok && (peers & lt) == 0) {
        cnt[dg * kCntStride + wave] = base + __popcll(peers);
        if (rest != 0) table[wave * kRadix + dg] = 0ull;
      }
      if (ok && pos >= 0 && pos < m) dst[pos] = e;   // always true for a consistent count; keeps stores in bounds
    }
    __syncthreads();
  }
  for (int i = tid; i < m; i += kSortThreads) out[t0 + i] = buf0[i];
  for (int i = tid; i * kSplStep < m; i += kSortThreads) spl[(int64_t)blockIdx.x * kSplPerTile + i] = buf0[i * kSplStep];
}

// Merges the sorted tiles: element i of tile a goes to its rank in the tile
// plus, for every other tile, the number of its elements below it, and
// perm[pos] = its token (the elements are distinct, so the positions are a
// permutation; every position is checked below n).  The count in tile b: the
// splitters of b (every 64th element, in LDS) bound it to a window of at most
// 63 elements, searched in device memory.
constexpr int kMergeTiles = 16;   // tiles whose splitters are in LDS at a time
__global__ __launch_bounds__(256) void bpr_merge_kernel(const uint64_t* __restrict__ sorted,
                                                        const uint64_t* __restrict__ spl, int32_t* __restrict__ perm,
                                                        int64_t n) {
  __shared__ uint64_t sp[kMergeTiles * kSplPerTile];
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool act = i < n;
  const uint64_t v = act ? sorted[i] : 0ull;
  const int64_t a = act ? i / kSortTile : -1;
  const int64_t ntiles = (n + kSortTile - 1) / kSortTile;
  int64_t pos = act ? i - a * kSortTile : 0;
  for (int64_t g0 = 0; g0 < ntiles; g0 += kMergeTiles) {
    const int ng = (int)min((int64_t)kMergeTiles, ntiles - g0);
    __syncthreads();
    for (int q = threadIdx.x; q < ng * kSplPerTile; q += blockDim.x) {
      const int64_t b = g0 + q / kSplPerTile;
      const int s = q % kSplPerTile;
      const int64_t len = min((int64_t)kSortTile, n - b * kSortTile);
      sp[q] = (int64_t)s * kSplStep < len ? spl[b * kSplPerTile + s] : ~0ull;   // past the tile: above every element
    }
    __syncthreads();
    if (!act) continue;
    int64_t wb[kMergeTiles];
    int wl[kMergeTiles];
#pragma unroll
    for (int q = 0; q < kMergeTiles; ++q) {
      const int64_t b = g0 + q;
      wb[q] = b * kSortTile;
      wl[q] = 0;
      if (q < ng && b != a) {
        // splitters below v (they are sorted): a binary search in LDS
        int lo = 0, cnt = kSplPerTile;
        while (cnt > 0) {
          const int half = cnt >> 1;
          if (sp[q * kSplPerTile + lo + half] < v) {
            lo += half + 1;
            cnt -= half + 1;
          } else {
            cnt = half;
          }
        }
        // the lower bound lies in (64 (lo - 1), 64 lo]: a window of at most 63
        if (lo > 0) {
          const int64_t len = min((int64_t)kSortTile, n - b * kSortTile);
          wb[q] = b * kSortTile + (int64_t)(lo - 1) * kSplStep + 1;
          wl[q] = (int)(min((int64_t)lo * kSplStep, len) - ((int64_t)(lo - 1) * kSplStep + 1));
        }
      }
    }
    for (int it = 0; it < 7; ++it) {   // lower bound in every window, the probes of all tiles in flight together
#pragma unroll
      for (int q = 0; q < kMergeTiles; ++q) {
        if (wl[q] > 0) {
          const int half = wl[q] >> 1;
          if (sorted[wb[q] + half] < v) {
            wb[q] += half + 1;
            wl[q] -= half + 1;
          } else {
            wl[q] = half;
          }
        }
      }
    }
#pragma unroll
    for (int q = 0; q < kMergeTiles; ++q) {
      const int64_t b = g0 + q;
      if (q < ng && b != a) pos += wb[q] - b * kSortTile;
    }
  }
  if (act && pos >= 0 && pos < n) perm[pos] = (int32_t)(v & 0xffffffffu);
}

static size_t bpr_spl_bytes(const moe_cfg& c) {
  const int64_t ntiles = (c.T + kSortTile - 1) / kSortTile;
  return ((size_t)ntiles * kSplPerTile * sizeof(uint64_t) + 255) / 256 * 256;
}
size_t dispatch_bpr_ws_bytes(const moe_cfg& c) {
  const size_t a = (dispatch_ws_bytes(c) + 255) / 256 * 256;
  const size_t eb = ((size_t)c.T * sizeof(uint64_t) + 255) / 256 * 256;
  const size_t tb = ((size_t)c.T * sizeof(int32_t) + 255) / 256 * 256;
  return a + 2 * eb + tb + bpr_spl_bytes(c);
}

void launch_dispatch_bpr(const moe_cfg& c, const void* x, const float* logits, const int32_t* idx, int32_t* fill,
                         int32_t* slot, void* send_buf, int32_t* order, void* ws, hipStream_t s) {
  const size_t a = (dispatch_ws_bytes(c) + 255) / 256 * 256;
  const size_t eb = ((size_t)c.T * sizeof(uint64_t) + 255) / 256 * 256;
  char* w = (char*)ws + a;
  uint64_t* e0 = (uint64_t*)w;
  uint64_t* e1 = (uint64_t*)(w + eb);
  const size_t tb = ((size_t)c.T * sizeof(int32_t) + 255) / 256 * 256;
  int32_t* perm = order ? order : (int32_t*)(w + 2 * eb);
  uint64_t* spl = (uint64_t*)(w + 2 * eb + tb);
  if (c.T > 0) {
    static std::atomic<uint64_t> lds_ok{0};
    allow_dyn_lds((const void*)bpr_tile_sort_kernel, (int)kTileSortLds, lds_ok);
    const int64_t ntiles = (c.T + kSortTile - 1) / kSortTile;
    hipLaunchKernelGGL(bpr_key_kernel, dim3((unsigned)((c.T + 3) / 4)), dim3(256), 0, s, logits, idx, e0, c.T, c.E,
                       c.k);
    hipLaunchKernelGGL(bpr_tile_sort_kernel, dim3((unsigned)ntiles), dim3(kSortThreads), kTileSortLds, s, e0, e1, spl,
                       c.T);
    hipLaunchKernelGGL(bpr_merge_kernel, dim3((unsigned)((c.T + 255) / 256)), dim3(256), 0, s, e1, spl, perm, c.T);
  }
  dispatch_walk(c, x, idx, perm, nullptr, fill, slot, send_buf, ws, s);
}

// -------------------------------------------------------------------- combine
// y[t][:] = resid[t][:] + sum_r kept w[t][r] * O[e][s][:], in rank order, float
// accumulation (resid NULL = 0; the block passes its residual stream).
template <typename T, int KT, int U, bool UNI>
__global__ __launch_bounds__(256) void combine_kernel(const T* __restrict__ O, const int32_t* __restrict__ idx,
                                                      const int32_t* __restrict__ slot, const float* __restrict__ w,
                                                      const T* __restrict__ resid, T* __restrict__ y, int64_t T_tokens,
                                                      int d, int E, int kr, int C) {
  constexpr int V = Vec<T>::N;
  constexpr int KK = KT > 0 ? KT : kMaxK;
  const int k = KT > 0 ? KT : kr;
  const int nc = d / V;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t g = UNI ? (int64_t)__builtin_amdgcn_readfirstlane((int)(gid / nc)) : gid / nc;
  const int c = (int)(gid - g * nc);
  const int64_t t0 = g * U;
  if (t0 >= T_tokens) return;
  int64_t off[U][KK];
  float wr[U][KK];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t t = t0 + u;
#pragma unroll
    for (int r = 0; r < KK; ++r) {
      off[u][r] = -1;
      wr[u][r] = 0.f;
      if (t < T_tokens && r < k) {
        const int sl = slot[t * k + r];
        const int e = idx[t * k + r];
        if (sl >= 0 && sl < C && e >= 0 && e < E) {
          off[u][r] = erow<T>(e, sl, c * V, d, C);
          wr[u][r] = w[t * k + r];
        }
      }
    }
  }
  float acc[U][V], v[U][KK][V];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t t = t0 + u;
    if (resid && t < T_tokens) {
      Vec<T>::load(resid + t * d + (int64_t)c * V, acc[u]);
    } else {
#pragma unroll
      for (int i = 0; i < V; ++i) acc[u][i] = 0.f;
    }
#pragma unroll
    for (int r = 0; r < KK; ++r)
      if (off[u][r] >= 0) Vec<T>::load(O + off[u][r], v[u][r]);
  }
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t t = t0 + u;
    if (t >= T_tokens) break;
#pragma unroll
    for (int r = 0; r < KK; ++r)
      if (off[u][r] >= 0)
#pragma unroll
        for (int i = 0; i < V; ++i) acc[u][i] = fmaf(wr[u][r], v[u][r][i], acc[u][i]);
    Vec<T>::store(y + t * d + (int64_t)c * V, acc[u]);
  }
}
template <typename T, int KT, int U, bool UNI> struct Combine {
  static constexpr auto kernel() { return combine_kernel<T, KT, U, UNI>; }
};

void launch_combine(const moe_cfg& c, const void* O, const int32_t* idx, const int32_t* slot, const float* w,
                    void* y, hipStream_t s, const void* resid) {
  if (c.T == 0) return;
  if (c.dtype == MOE_BF16)
    row_launch<Combine, uint16_t, 4, 2>(c, s, (const uint16_t*)O, idx, slot, w, (const uint16_t*)resid, (uint16_t*)y, c.T,
                                  c.d_model, c.E, c.k, c.C);
  else
    row_launch<Combine, float, 4, 2>(c, s, (const float*)O, idx, slot, w, (const float*)resid, (float*)y, c.T, c.d_model,
                               c.E, c.k, c.C);
}

// ------------------------------------------------------ combine + gate backward
// One wavefront per token: dO[e][s] = w dy, g_r = <dy, O[e][s]>, then dlogits.
template <typename T, int KT>
__global__ __launch_bounds__(256) void combine_bwd_kernel(const float* __restrict__ logits,
                                                          const int32_t* __restrict__ idx,
                                                          const float* __restrict__ w,
                                                          const int32_t* __restrict__ slot,
                                                          const T* __restrict__ O, const T* __restrict__ dy,
                                                          T* __restrict__ dO, float* __restrict__ dlogits,
                                                          int64_t T_tokens, int d, int E, int kr, int C, int renorm) {
  constexpr int V = Vec<T>::N;
  constexpr int KK = KT > 0 ? KT : kMaxK;
  const int k = KT > 0 ? KT : kr;
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
  if (t >= T_tokens) return;
  int er[KK], sr[KK];
  float wr[KK], gp[KK];
#pragma unroll
  for (int r = 0; r < KK; ++r) {
    er[r] = r < k ? idx[t * k + r] : 0;
    sr[r] = r < k ? slot[t * k + r] : -1;
    if (er[r] < 0 || er[r] >= E || sr[r] >= C) { er[r] = 0; sr[r] = -1; }
    wr[r] = r < k ? w[t * k + r] : 0.f;
    gp[r] = 0.f;
  }
  // Two 16-byte chunks per lane per round: every dy and O load of the round
  // is issued before the first product and store.
  const int nc = d / V;
  for (int c0 = lane; c0 < nc; c0 += 2 * kWave) {
    u32x4 gv[2], ov[2][KK];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int c = c0 + h * kWave;
      const bool ok = c < nc;
      gv[h] = ok ? *reinterpret_cast<const u32x4*>(dy + t * d + (int64_t)c * V) : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int r = 0; r < KK; ++r)
        ov[h][r] = (ok && sr[r] >= 0) ? *reinterpret_cast<const u32x4*>(O + erow<T>(er[r], sr[r], c * V, d, C))
                                      : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int c = c0 + h * kWave;
      if (c >= nc) continue;
      float g[V];
      Vec<T>::load(&gv[h], g);
#pragma unroll
      for (int r = 0; r < KK; ++r) {
        if (sr[r] < 0) continue;
        float o[V], out[V];
        Vec<T>::load(&ov[h][r], o);
#pragma unroll
        for (int i = 0; i < V; ++i) {
          gp[r] = fmaf(g[i], o[i], gp[r]);
          out[i] = wr[r] * g[i];
        }
        Vec<T>::store(dO + eoff<T>(er[r], sr[r], c * V, d, C), out);
      }
    }
  }
  float gsum = 0.f;  // sum_r w_r g_r
#pragma unroll
  for (int r = 0; r < KK; ++r) {
    gp[r] = wave_sum(gp[r]);
    gsum = fmaf(wr[r], gp[r], gsum);
  }
  // dlogits: lane j handles expert j (E <= 64).
  const int j = lane;
  float dl = 0.f;
  if (renorm) {
#pragma unroll
    for (int r = 0; r < KK; ++r)
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
    for (int r = 0; r < KK; ++r)
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
  auto go = [&](auto kern, auto tag) {
    using T = decltype(tag);
    hipLaunchKernelGGL(kern, dim3(blocks), dim3(256), 0, s, logits, idx, w, slot, (const T*)O, (const T*)dy,
                       (T*)dO, dlogits, c.T, c.d_model, c.E, c.k, c.C, c.renorm);
  };
  if (c.dtype == MOE_BF16) {
    if (c.k == 1) go(combine_bwd_kernel<uint16_t, 1>, uint16_t{});
    else if (c.k == 2) go(combine_bwd_kernel<uint16_t, 2>, uint16_t{});
    else go(combine_bwd_kernel<uint16_t, 0>, uint16_t{});
  } else {
    if (c.k == 1) go(combine_bwd_kernel<float, 1>, float{});
    else if (c.k == 2) go(combine_bwd_kernel<float, 2>, float{});
    else go(combine_bwd_kernel<float, 0>, float{});
  }
}

// ----------------------------------------------------------- dispatch backward
// dx[t] = sum_r kept dXe[e][s] + sum_j dlogits[t][j] Wg[j]  (renorm: only the k selected j are nonzero).
template <typename T, int KT, int U, bool UNI>
__global__ __launch_bounds__(256) void dispatch_bwd_kernel(const T* __restrict__ Wg, const float* __restrict__ dl,
                                                           const int32_t* __restrict__ idx,
                                                           const int32_t* __restrict__ slot,
                                                           const T* __restrict__ dXe, T* __restrict__ dx,
                                                           int64_t T_tokens, int d, int E, int kr, int C, int renorm) {
  constexpr int V = Vec<T>::N;
  constexpr int KK = KT > 0 ? KT : kMaxK;
  const int k = KT > 0 ? KT : kr;
  const int nc = d / V;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t g = UNI ? (int64_t)__builtin_amdgcn_readfirstlane((int)(gid / nc)) : gid / nc;
  const int c = (int)(gid - g * nc);
  const int64_t t0 = g * U;
  if (t0 >= T_tokens) return;
  int64_t off[U][KK];
  int ej[U][KK];      // renorm: the selected experts whose Wg rows enter dx
  float aj[U][KK];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t t = t0 + u;
#pragma unroll
    for (int r = 0; r < KK; ++r) {
      off[u][r] = -1;
      ej[u][r] = -1;
      aj[u][r] = 0.f;
      if (t < T_tokens && r < k) {
        const int sl = slot[t * k + r];
        const int e = idx[t * k + r];
        const bool ev = e >= 0 && e < E;
        if (sl >= 0 && sl < C && ev) off[u][r] = erow<T>(e, sl, c * V, d, C);
        if (renorm && ev) {
          ej[u][r] = e;
          aj[u][r] = dl[t * E + e];
        }
      }
    }
  }
  float v[U][KK][V], gw[U][KK][V];
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int r = 0; r < KK; ++r) {
      if (off[u][r] >= 0) Vec<T>::load(dXe + off[u][r], v[u][r]);
      if (ej[u][r] >= 0) Vec<T>::load(Wg + (int64_t)ej[u][r] * d + (int64_t)c * V, gw[u][r]);
    }
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t t = t0 + u;
    if (t >= T_tokens) break;
    float acc[V];
#pragma unroll
    for (int i = 0; i < V; ++i) acc[i] = 0.f;
#pragma unroll
    for (int r = 0; r < KK; ++r)
      if (off[u][r] >= 0)
#pragma unroll
        for (int i = 0; i < V; ++i) acc[i] += v[u][r][i];
#pragma unroll
    for (int r = 0; r < KK; ++r)
      if (ej[u][r] >= 0)
#pragma unroll
        for (int i = 0; i < V; ++i) acc[i] = fmaf(aj[u][r], gw[u][r][i], acc[i]);
    if (!renorm) {
      for (int j = 0; j < E; ++j) {
        const float a = dl[t * E + j];
        float gv[V];
        Vec<T>::load(Wg + (int64_t)j * d + (int64_t)c * V, gv);
#pragma unroll
        for (int i = 0; i < V; ++i) acc[i] = fmaf(a, gv[i], acc[i]);
      }
    }
    Vec<T>::store(dx + t * d + (int64_t)c * V, acc);
  }
}
template <typename T, int KT, int U, bool UNI> struct DispatchBwd {
  static constexpr auto kernel() { return dispatch_bwd_kernel<T, KT, U, UNI>; }
};

void launch_dispatch_bwd(const moe_cfg& c, const void* Wg, const float* dlogits, const int32_t* idx,
                         const int32_t* slot, const void* dXe, void* dx, hipStream_t s) {
  if (c.T == 0) return;
  if (c.dtype == MOE_BF16)
    row_launch<DispatchBwd, uint16_t, 2, 1>(c, s, (const uint16_t*)Wg, dlogits, idx, slot, (const uint16_t*)dXe,
                                      (uint16_t*)dx, c.T, c.d_model, c.E, c.k, c.C, c.renorm);
  else
    row_launch<DispatchBwd, float, 2, 1>(c, s, (const float*)Wg, dlogits, idx, slot, (const float*)dXe, (float*)dx, c.T,
                                   c.d_model, c.E, c.k, c.C, c.renorm);
}

// -------------------------------------------------------------------- dWg
// dWg[e][:] = sum_t dlogits[t][e] x[t][:].  Stage 1: a block owns a slab of
// 256 columns (each lane 4 consecutive columns), a chunk of tokens and a
// group of 8, 16 or 32 experts; its eight waves take every eighth token of
// the chunk, and their sums meet in LDS in wave order.  A dlogits entry that
// is zero (every unselected expert under renormalised top-k) skips its
// products: the branch is uniform, since a wave works on one token at a time.
// Stage 2 adds the chunk partials in a fixed order.  Deterministic.
constexpr int kDwgCPL = 4;                 // columns per lane
constexpr int kDwgSlab = 64 * kDwgCPL;     // columns per block
constexpr int kDwgWaves = 8;
constexpr int kDwgRound = 4;               // experts per LDS reduction round

struct DwgPlan {
  int64_t tch, nch;
  int slabs, egroups, eg;
};
static DwgPlan dwg_plan(const moe_cfg& c) {
  DwgPlan q;
  q.eg = c.E <= 8 ? 8 : (c.E <= 16 ? 16 : 32);
  q.slabs = (c.d_model + kDwgSlab - 1) / kDwgSlab;
  q.egroups = (c.E + q.eg - 1) / q.eg;
  // About 512 blocks over the chunks (a wave's few tokens per chunk are
  // latency-bound, so more blocks in flight read x faster), at least 64
  // tokens per chunk, at most 16 MiB of partials.
  int64_t want = 512 / (q.slabs * q.egroups);
  const int64_t cap = ((int64_t)16 << 20) / ((int64_t)c.E * c.d_model * 4);
  if (want > cap) want = cap;
  if (want < 1) want = 1;
  int64_t tch = (c.T + want - 1) / want;
  if (tch < 64) tch = 64;
  q.tch = tch;
  q.nch = (c.T + tch - 1) / tch;
  return q;
}

template <typename T> __device__ __forceinline__ void load4(const T* p, float (&v)[4]);
template <> __device__ __forceinline__ void load4<uint16_t>(const uint16_t* p, float (&v)[4]) {
  const u32x2 r = *reinterpret_cast<const u32x2*>(p);
  v[0] = __uint_as_float(r[0] << 16);
  v[1] = __uint_as_float(r[0] & 0xffff0000u);
  v[2] = __uint_as_float(r[1] << 16);
  v[3] = __uint_as_float(r[1] & 0xffff0000u);
}
template <> __device__ __forceinline__ void load4<float>(const float* p, float (&v)[4]) { Vec<float>::load(p, v); }

// SPARSE: a wave reads each token's dlogits row with one vector load (lane j
// holds expert j), and visits only the nonzero entries of its group (under
// renormalised top-k, the k selected experts).  Otherwise every expert of the
// group, with a uniform skip of zero entries.  Both orders are the same: per
// expert, the wave's tokens in sequence.
template <typename T, int EG, bool SPARSE>
__global__ __launch_bounds__(64 * kDwgWaves) void dwg_partial_kernel(const T* __restrict__ x,
                                                                     const float* __restrict__ dl,
                                                                     float* __restrict__ part, int64_t T_tokens,
                                                                     int d, int E, int64_t tch) {
  constexpr int NW = kDwgWaves, CPL = kDwgCPL;
  __shared__ float red[NW - 1][kDwgRound][kDwgSlab];
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int col = blockIdx.x * kDwgSlab + CPL * lane;
  const int e0 = blockIdx.z * EG;
  const int64_t ch = blockIdx.y;
  const int64_t t_begin = ch * tch;
  const int64_t t_end = min(t_begin + tch, T_tokens);
  float acc[EG][CPL];
#pragma unroll
  for (int e = 0; e < EG; ++e)
#pragma unroll
    for (int j = 0; j < CPL; ++j) acc[e][j] = 0.f;
  const bool colok = col < d;
  const bool full = (E % 4 == 0) && (e0 + EG <= E);   // whole group inside each dlogits row
  const bool mine = lane >= e0 && lane < e0 + EG && lane < E;
  constexpr int U = SPARSE ? 8 : 4;   // tokens in flight per wave
  for (int64_t t0 = t_begin + wid; t0 < t_end; t0 += NW * U) {
    float xv[U][CPL];
    float gl[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {   // unconditional loads (clamped), so all U are in flight together
      int64_t t = t0 + NW * u;
      if (t >= t_end) t = t_end - 1;
      load4<T>(x + t * d + (colok ? col : 0), xv[u]);
      if constexpr (SPARSE) gl[u] = dl[t * E + (mine ? lane : 0)];
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t t = t0 + NW * u;
      if (t >= t_end) break;
      if constexpr (SPARSE) {
        uint64_t m = __ballot(mine && gl[u] != 0.f);
        while (m) {
          const int e = __ffsll((unsigned long long)m) - 1;
          m &= m - 1;
          const float g = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, gl[u]), e));
          const int rel = e - e0;
#pragma unroll
          for (int R = 0; R < EG; ++R) {   // uniform compare chain: acc indices stay static
            if (rel == R) {
#pragma unroll
              for (int j = 0; j < CPL; ++j) acc[R][j] = fmaf(g, xv[u][j], acc[R][j]);
            }
          }
        }
      } else {
        const float* dr = dl + t * E + e0;
        float g[EG];
        if (full) {   // the group's dlogits as 16-byte (scalar-cache) loads
#pragma unroll
          for (int q = 0; q < EG / 4; ++q) {
            const f32x4 v = *reinterpret_cast<const f32x4*>(dr + 4 * q);
#pragma unroll
            for (int i = 0; i < 4; ++i) g[4 * q + i] = v[i];
          }
        } else {
#pragma unroll
          for (int e = 0; e < EG; ++e) g[e] = (e0 + e < E) ? dr[e] : 0.f;
        }
#pragma unroll
        for (int e = 0; e < EG; ++e) {
          if (g[e] != 0.f) {
#pragma unroll
            for (int j = 0; j < CPL; ++j) acc[e][j] = fmaf(g[e], xv[u][j], acc[e][j]);
          }
        }
      }
    }
  }
  // Block sum in wave order, kDwgRound experts per round through LDS.
  float* out = part + (ch * E + e0) * (int64_t)d + col;
#pragma unroll
  for (int r0 = 0; r0 < EG; r0 += kDwgRound) {
    if (wid > 0) {
#pragma unroll
      for (int i = 0; i < kDwgRound; ++i)
#pragma unroll
        for (int j = 0; j < CPL; ++j) red[wid - 1][i][CPL * lane + j] = acc[r0 + i][j];
    }
    __syncthreads();
    if (wid == 0 && colok) {
#pragma unroll
      for (int i = 0; i < kDwgRound; ++i) {
        if (e0 + r0 + i >= E) continue;
        float v[CPL];
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
          v[j] = acc[r0 + i][j];
#pragma unroll
          for (int w = 0; w < NW - 1; ++w) v[j] += red[w][i][CPL * lane + j];
        }
        Vec<float>::store(out + (int64_t)(r0 + i) * d, v);
      }
    }
    __syncthreads();
  }
}

// dWg[i] = sum over chunks of part[c][i]: the chunks fall into kDwgRuns
// contiguous runs, each summed in chunk order by its own thread, and the run
// sums are added in run order.  A block covers 32 x 4 consecutive outputs.
constexpr int kDwgRuns = 8;
__global__ __launch_bounds__(32 * kDwgRuns) void dwg_reduce_kernel(const float* __restrict__ part,
                                                                   float* __restrict__ dWg, int nch, int64_t ed) {
  __shared__ float red[kDwgRuns][32][4];
  const int q = threadIdx.x & 31, g = threadIdx.x >> 5;
  const int64_t i = ((int64_t)blockIdx.x * 32 + q) * 4;
  const int per = (nch + kDwgRuns - 1) / kDwgRuns;
  const int c_begin = min(nch, g * per), c_end = min(nch, c_begin + per);
  float s[4] = {0.f, 0.f, 0.f, 0.f};
  int c = c_begin;
  if (i >= ed) c = c_end;
  for (; c + 4 <= c_end; c += 4) {
    float v[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u) Vec<float>::load(part + (int64_t)(c + u) * ed + i, v[u]);
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int j = 0; j < 4; ++j) s[j] += v[u][j];
  }
  for (; c < c_end; ++c) {
    float v[4];
    Vec<float>::load(part + (int64_t)c * ed + i, v);
#pragma unroll
    for (int j = 0; j < 4; ++j) s[j] += v[j];
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) red[g][q][j] = s[j];
  __syncthreads();
  if (g == 0 && i < ed) {
#pragma unroll
    for (int r = 1; r < kDwgRuns; ++r)
#pragma unroll
      for (int j = 0; j < 4; ++j) s[j] += red[r][q][j];
    Vec<float>::store(dWg + i, s);
  }
}

size_t bwd_dw_ws_bytes(const moe_cfg& c) {
  const DwgPlan q = dwg_plan(c);
  return (size_t)(q.nch * c.E * (int64_t)c.d_model) * sizeof(float);
}

template <typename T, int EG>
static void launch_dwg_eg(const moe_cfg& c, const void* x, const float* dl, float* part, const DwgPlan& q,
                          hipStream_t s) {
  dim3 grid((unsigned)q.slabs, (unsigned)q.nch, (unsigned)q.egroups);
  if (c.renorm)
    hipLaunchKernelGGL((dwg_partial_kernel<T, EG, true>), grid, dim3(64 * kDwgWaves), 0, s, (const T*)x, dl, part,
                       c.T, c.d_model, c.E, q.tch);
  else
    hipLaunchKernelGGL((dwg_partial_kernel<T, EG, false>), grid, dim3(64 * kDwgWaves), 0, s, (const T*)x, dl, part,
                       c.T, c.d_model, c.E, q.tch);
}
template <typename T>
static void launch_dwg_t(const moe_cfg& c, const void* x, const float* dl, float* part, const DwgPlan& q,
                         hipStream_t s) {
  if (q.eg == 8) launch_dwg_eg<T, 8>(c, x, dl, part, q, s);
  else if (q.eg == 16) launch_dwg_eg<T, 16>(c, x, dl, part, q, s);
  else launch_dwg_eg<T, 32>(c, x, dl, part, q, s);
}

void launch_dwg(const moe_cfg& c, const void* x, const float* dlogits, float* dWg, void* ws, hipStream_t s) {
  const int64_t ed = (int64_t)c.E * c.d_model;   // a multiple of 8
  const DwgPlan q = dwg_plan(c);                 // nch = 0 when T == 0: the reduce then writes zeros
  float* part = (float*)ws;
  if (q.nch > 0) {
    if (c.dtype == MOE_BF16) launch_dwg_t<uint16_t>(c, x, dlogits, part, q, s);
    else launch_dwg_t<float>(c, x, dlogits, part, q, s);
  }
  hipLaunchKernelGGL(dwg_reduce_kernel, dim3((unsigned)((ed / 4 + 31) / 32)), dim3(32 * kDwgRuns), 0, s, part,
                     dWg, (int)q.nch, ed);
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
