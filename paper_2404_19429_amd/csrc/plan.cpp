// Host-side planners, plain C++ with no device code:
// * the weight-gradient computation schedule pass (Sec. 4: labelling by
//   dependency paths, Sec. 4.1; the greedy best-fit assignment of
//   weight-gradient operations to all-to-alls, Sec. 4.2 and Alg. 1; and the
//   reordering that places each assigned operation right after its
//   all-to-all) -- C ABI moe_dw_schedule;
// * the operator-partition pass's pipeline cost and range choice (Sec. 5.1's
//   dynamic program over Sec. 5.3's timeline simulation) -- C ABI
//   moe_pipeline_plan.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <iterator>
#include <string>
#include <vector>

#include "internal.h"

namespace lmoe {

namespace {

constexpr int kOther = 0, kA2A = 1, kDW = 2;

struct Reorder {
  const std::vector<std::vector<int>>& pred;   // ascending
  const std::vector<int32_t>& asg;             // DW -> all-to-all, or -1
  std::vector<char> emitted;
  std::vector<int32_t> out;

  // Emits i after the not-yet-emitted assigned operations it consumes.
  void pull(int i) {
    for (int p : pred[i])
      if (!emitted[p]) pull(p);
    if (!emitted[i]) {
      emitted[i] = 1;
      out.push_back(i);
    }
  }
  // Emits, in index order and until nothing changes, every assigned operation
  // whose all-to-all and predecessors are out.  Only the operations whose
  // all-to-all is already out (`active`, ascending) can qualify; all-to-alls
  // are emitted only outside this loop.
  void flush(std::vector<int>& active) {
    for (bool changed = true; changed;) {
      changed = false;
      for (int j : active) {
        if (emitted[j]) continue;
        bool ready = true;
        for (int p : pred[j]) ready = ready && emitted[p];
        if (ready) {
          emitted[j] = 1;
          out.push_back(j);
          changed = true;
        }
      }
    }
    active.erase(std::remove_if(active.begin(), active.end(), [&](int j) { return emitted[j] != 0; }), active.end());
  }
};

}  // namespace

std::string dw_schedule(int n, const int32_t* kind, const double* time, int n_edges, const int32_t* src,
                        const int32_t* dst, int32_t* assign, int32_t* order, double* overlap) {
  if (n < 0 || n > kMaxPlanInstr) return "n outside 0.." + std::to_string(kMaxPlanInstr);
  if (n_edges < 0) return "n_edges < 0";
  for (int i = 0; i < n; ++i) {
    if (kind[i] != kOther && kind[i] != kA2A && kind[i] != kDW) return "kind[" + std::to_string(i) + "] unknown";
    if (!std::isfinite(time[i]) || time[i] < 0) return "time[" + std::to_string(i) + "] not a finite value >= 0";
  }
  std::vector<std::vector<int>> succ(n), pred(n);
  for (int e = 0; e < n_edges; ++e) {
    if (src[e] < 0 || dst[e] >= n || src[e] >= dst[e])
      return "edge " + std::to_string(e) + " is not src < dst within 0..n-1 (the sequence must be an execution order)";
    succ[src[e]].push_back(dst[e]);
    pred[dst[e]].push_back(src[e]);
  }
  for (auto& p : pred) std::sort(p.begin(), p.end()), p.erase(std::unique(p.begin(), p.end()), p.end());

  // Labelling: reach[i] = the operations with a path from i, as bit rows,
  // built from the end of the sequence (every edge points forward).
  const int words = (n + 63) / 64;
  std::vector<uint64_t> reach((size_t)n * words, 0ull);
  for (int i = n - 1; i >= 0; --i) {
    uint64_t* ri = &reach[(size_t)i * words];
    for (int j : succ[i]) {
      const uint64_t* rj = &reach[(size_t)j * words];
      for (int w = 0; w < words; ++w) ri[w] |= rj[w];
      ri[j >> 6] |= 1ull << (j & 63);
    }
  }
  auto path = [&](int a, int b) { return (reach[(size_t)a * words + (b >> 6)] >> (b & 63)) & 1ull; };

  // Greedy assignment, all-to-alls in sequence order.
  std::vector<int32_t> asg(n, -1);
  std::vector<char> used(n, 0);
  std::vector<int> cand;
  std::vector<double> assigned_time(n, 0.0);
  for (int a = 0; a < n; ++a) {
    if (kind[a] != kA2A) continue;
    cand.clear();
    for (int j = 0; j < n; ++j)
      if (j != a && kind[j] == kDW && !path(a, j) && !path(j, a)) cand.push_back(j);
    double t_u = time[a];
    while (t_u > 0) {
      int best = -1;
      double bd = 0.0;
      for (int j : cand) {
        if (used[j]) continue;
        const double dj = std::fabs(t_u - time[j]);
        if (best < 0 || dj < bd) {   // ties keep the lower index
          best = j;
          bd = dj;
        }
      }
      if (best < 0) break;
      t_u -= time[best];
      used[best] = 1;
      asg[best] = a;
      assigned_time[a] += time[best];
    }
  }
  double ov = 0.0;
  for (int a = 0; a < n; ++a)
    if (kind[a] == kA2A) ov += std::min(time[a], assigned_time[a]);

  // Reordering.
  std::vector<int> assigned;
  std::vector<std::vector<int>> of_a2a(n);   // the operations assigned to each all-to-all, ascending
  for (int j = 0; j < n; ++j)
    if (asg[j] >= 0) {
      assigned.push_back(j);
      of_a2a[asg[j]].push_back(j);
    }
  Reorder R{pred, asg, std::vector<char>(n, 0), {}};
  R.out.reserve(n);
  std::vector<int> active;
  for (int i = 0; i < n; ++i) {
    if (asg[i] >= 0 || R.emitted[i]) continue;
    R.pull(i);
    if (kind[i] == kA2A && !of_a2a[i].empty()) {
      std::vector<int> merged;
      std::merge(active.begin(), active.end(), of_a2a[i].begin(), of_a2a[i].end(), std::back_inserter(merged));
      active.swap(merged);
    }
    R.flush(active);
  }
  for (int j : assigned)
    if (!R.emitted[j]) R.pull(j);

  for (int i = 0; i < n; ++i) {
    assign[i] = asg[i];
    order[i] = R.out[i];
  }
  *overlap = ov;
  return "";
}

// ------------------------------------------------- the block backward's schedule
// The block backward as the paper's expert-parallel step runs it, in the
// order reverse-mode differentiation emits it (the instance is spelled out
// with moe_block_dw_schedule in lancet_moe.h): the chain, each weight
// gradient where the backward of its layer produces it, and the two
// all-to-alls of the MoE layer around its experts.
std::string block_dw_schedule(const double* op_ms, double a2a_ms, int32_t* dw_order, int32_t* assign,
                              double* overlap) {
  if (!std::isfinite(a2a_ms) || a2a_ms < 0) return "a2a_ms not a finite value >= 0";
  constexpr int A2A = -1;   // stand-in for an all-to-all in the op list below
  static const int ops[16] = {MOE_BOP_COMBINE_BWD, A2A,           MOE_BOP_EXPERT_DX, MOE_BOP_DW_EXPERT,
                              A2A,                 MOE_BOP_DISPATCH_BWD, MOE_BOP_DWG,   MOE_BOP_LN2_BWD,
                              MOE_BOP_DLN2,        MOE_BOP_DWO,   MOE_BOP_DATTN,     MOE_BOP_ATTN_BWD,
                              MOE_BOP_DWQKV,       MOE_BOP_DA,    MOE_BOP_LN1_BWD,   MOE_BOP_DLN1};
  static const int32_t src[] = {0, 1, 1, 2, 2, 4, 0, 0, 5, 7, 7, 7, 10, 11, 11, 13, 14};
  static const int32_t dst[] = {1, 2, 3, 3, 4, 5, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15};
  int32_t kind[16];
  double time[16];
  for (int i = 0; i < 16; ++i) {
    const int op = ops[i];
    if (op == A2A) {
      kind[i] = kA2A;
      time[i] = a2a_ms;
    } else {
      kind[i] = op >= MOE_BOP_DW_EXPERT ? kDW : kOther;
      time[i] = op_ms[op];
    }
  }
  int32_t asg[16], ord[16];
  const std::string err = dw_schedule(16, kind, time, (int)(sizeof src / sizeof src[0]), src, dst, asg, ord, overlap);
  if (!err.empty()) return err;
  int q = 0;
  for (int i = 0; i < 16; ++i)
    if (kind[ord[i]] == kDW) dw_order[q++] = ops[ord[i]];
  if (assign)
    for (int i = 0; i < 16; ++i) assign[i] = asg[i];
  return "";
}

// ----------------------------------------------------------- partition ranges

namespace {

// End time of k partitions of the stages (kind, one partition's time): a
// partition's stage starts after its previous stage and after the previous
// instruction of its kind in the order stage by stage, partition by
// partition.
double simulate_stages(const std::vector<std::pair<int, double>>& st, int k, std::vector<double>& prev) {
  prev.assign(k, 0.0);
  double free_[2] = {0.0, 0.0};
  double last = 0.0;
  for (const auto& sd : st) {
    for (int p = 0; p < k; ++p) {
      const double s = std::max(prev[p], free_[sd.first]);
      const double e = s + sd.second;
      prev[p] = e;
      free_[sd.first] = e;
      last = std::max(last, e);
    }
  }
  return last;
}

}  // namespace

double pipeline_range_cost(int N, int K, const int32_t* kind, const double* times, const double* join, int i, int n,
                           int k) {
  (void)N;
  std::vector<std::pair<int, double>> st;
  double sum = 0.0;
  for (int j = i - 1; j < n; ++j) {
    const double t = times[(size_t)j * K + (k - 1)];
    if (std::isinf(t)) return INFINITY;
    sum += t;
    if (!st.empty() && st.back().first == kind[j]) st.back().second += t;
    else st.emplace_back(kind[j], t);
  }
  if (k == 1) return sum;
  std::vector<double> prev;
  return simulate_stages(st, k, prev) + join[k - 1];
}

std::string pipeline_plan(int N, int K, const int32_t* kind, const double* times, const double* join, int G,
                          int32_t* seg_begin, int32_t* seg_end, int32_t* seg_k, int32_t* n_seg, double* total) {
  if (N < 0 || N > kMaxPlanInstr) return "N outside 0.." + std::to_string(kMaxPlanInstr);
  if (K < 1 || K > 64) return "K outside 1..64";
  for (int j = 0; j < N; ++j) {
    if (kind[j] != 0 && kind[j] != 1) return "kind[" + std::to_string(j) + "] is neither 0 nor 1";
    for (int k = 0; k < K; ++k) {
      const double t = times[(size_t)j * K + k];
      if (std::isnan(t) || t < 0 || (k == 0 && std::isinf(t)))
        return "times[" + std::to_string(j) + "][" + std::to_string(k) + "] invalid (unsplit times must be finite)";
    }
  }
  for (int k = 0; k < K; ++k)
    if (!std::isfinite(join[k]) || join[k] < 0) return "join[" + std::to_string(k) + "] not a finite value >= 0";
  if (G <= 0 || G > N) G = N;
  std::vector<double> T(N + 1, INFINITY);
  std::vector<int> ai(N + 1, 0), ak(N + 1, 0);
  T[0] = 0.0;
  for (int n = 1; n <= N; ++n) {
    for (int i = std::max(1, n - G + 1); i <= n; ++i) {
      for (int k = 1; k <= K; ++k) {
        const double c = T[i - 1] + pipeline_range_cost(N, K, kind, times, join, i, n, k);
        if (c < T[n]) {
          T[n] = c;
          ai[n] = i;
          ak[n] = k;
        }
      }
    }
  }
  int cnt = 0;
  for (int n = N; n > 0; n = ai[n] - 1) ++cnt;
  int q = cnt;
  for (int n = N; n > 0; n = ai[n] - 1) {
    --q;
    seg_begin[q] = ai[n];
    seg_end[q] = n;
    seg_k[q] = ak[n];
  }
  *n_seg = cnt;
  *total = T[N];
  return "";
}

}  // namespace lmoe
