// Optimal token slicing (Sec. 3.3): the t_max enumeration of Eq. 6-7 over the
// distinct table values, each solved with the recurrence of Eq. 8 /
// Algorithm 1, the early stop and the eps windows of the "Optimization"
// paragraph.  Host code.
//
// The thresholds are independent subproblems, so they are solved in parallel
// batches; results are then scanned in ascending order with exactly the
// sequential stop and tie rules, so the answer does not depend on the thread
// count.  Inside one threshold the recurrence reads a transposed copy of the
// table in which all slices ending at one position are contiguous.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <thread>
#include <vector>

#include "../../include/terapipe.h"

namespace {

constexpr int64_t INF = INT64_MAX;

struct Solve {
  int64_t S = INF;  // S*(U; t_max)
  std::vector<int> lens;
};

// by_end[i][k-1] = t(k units, i-k units of context): every slice that ends at i.
struct Table {
  int U;
  std::vector<int64_t> by_end;
};

void solve_one(const Table& T, int64_t tmax, std::vector<int64_t>& S, std::vector<int>& q,
               Solve* out) {
  const int U = T.U;
  S[0] = 0;
  for (int i = 1; i <= U; ++i) {
    int64_t best = INF;
    int bk = 0;
    const int64_t* row = &T.by_end[(size_t)i * U];
    for (int k = 1; k <= i; ++k) {
      const int64_t c = row[k - 1];
      if (c > tmax) continue;
      const int64_t prev = S[i - k];
      if (prev == INF) continue;
      const int64_t v = prev + c;
      if (v < best) {
        best = v;
        bk = k;
      }
    }
    S[i] = best;
    q[i] = bk;
  }
  out->S = S[U];
  out->lens.clear();
  if (S[U] == INF) return;
  for (int i = U; i > 0; i -= q[i]) out->lens.push_back(q[i]);
  std::reverse(out->lens.begin(), out->lens.end());
}

}  // namespace

extern "C" tp_status tp_dp_optimal_slicing(const int64_t* cost, int L_units, int unit, int K,
                                           int64_t eps_ns, int* out_lens, int* out_M,
                                           int64_t* out_T) {
  if (!cost || !out_lens || !out_M || !out_T || L_units < 1 || unit < 1 || K < 1 || eps_ns < 0)
    return TP_ERR_INVALID;
  const int U = L_units;
  Table T;
  T.U = U;
  T.by_end.assign((size_t)(U + 1) * U, INF);
  std::vector<int64_t> vals;
  vals.reserve((size_t)U * (U + 1) / 2);
  for (int k = 1; k <= U; ++k)
    for (int j = 0; j + k <= U; ++j) {
      const int64_t c = cost[(size_t)(k - 1) * U + j];
      if (c < 0) return TP_ERR_INVALID;
      vals.push_back(c);
      T.by_end[(size_t)(j + k) * U + (k - 1)] = c;
    }
  std::sort(vals.begin(), vals.end());
  vals.erase(std::unique(vals.begin(), vals.end()), vals.end());

  // window representatives: from each not-yet-covered value v, the largest value <= v + eps
  std::vector<int64_t> starts, reps;
  for (size_t i = 0; i < vals.size();) {
    size_t j = i;
    while (j + 1 < vals.size() && vals[j + 1] <= vals[i] + eps_ns) ++j;
    starts.push_back(vals[i]);
    reps.push_back(vals[j]);
    i = j + 1;
  }

  unsigned hw = std::thread::hardware_concurrency();
  const int nthreads = (int)std::max(1u, std::min(hw ? hw : 1u, 16u));
  const size_t batch = (size_t)nthreads * 4;
  int64_t best = INF;
  std::vector<int> best_lens;
  std::vector<Solve> res;
  bool stop = false;
  for (size_t b0 = 0; b0 < reps.size() && !stop; b0 += batch) {
    const size_t b1 = std::min(reps.size(), b0 + batch);
    // thresholds whose window start already fails the stop test need no solve
    size_t bend = b0;
    while (bend < b1 && !(best != INF && (double)K * (double)starts[bend] > (double)best)) ++bend;
    res.assign(bend - b0, Solve());
    auto work = [&](int tid) {
      std::vector<int64_t> S(U + 1);
      std::vector<int> q(U + 1);
      for (size_t w = b0 + tid; w < bend; w += nthreads) solve_one(T, reps[w], S, q, &res[w - b0]);
    };
    if (bend - b0 > 1 && nthreads > 1) {
      std::vector<std::thread> th;
      const int used = (int)std::min<size_t>(nthreads, bend - b0);
      for (int t = 1; t < used; ++t) th.emplace_back(work, t);
      work(0);  // thread 0's share runs here
      for (auto& t : th) t.join();
    } else {
      work(0);
    }
    for (size_t w = b0; w < b1; ++w) {
      if (best != INF && (double)K * (double)starts[w] > (double)best) {
        stop = true;
        break;
      }
      const Solve& r = res[w - b0];
      if (r.S == INF) continue;
      const int64_t score = r.S + (int64_t)(K - 1) * reps[w];
      if (score < best) {
        best = score;
        best_lens = r.lens;
      }
    }
  }
  if (best == INF) return TP_ERR_INVALID;
  int64_t sum = 0, mx = 0;
  int ctx = 0;
  for (size_t i = 0; i < best_lens.size(); ++i) {
    const int64_t c = cost[(size_t)(best_lens[i] - 1) * U + ctx];
    sum += c;
    mx = std::max(mx, c);
    ctx += best_lens[i];
    out_lens[i] = best_lens[i] * unit;
  }
  *out_M = (int)best_lens.size();
  *out_T = sum + (int64_t)(K - 1) * mx;
  return TP_OK;
}

// Batch splitting (Sec. 3.4, combining token slicing with batch slicing): a
// batch of B sequences is cut into groups of b_1 + ... + b_D = B sequences
// that go through the pipeline one group after another, each with its own
// optimal token slicing; the group sizes minimise T_{b_1} + ... + T_{b_D}, a
// one-dimensional knapsack over the per-size latencies T_b.
//
// best[x] = the smallest total over groups that sum to x sequences:
// best[0] = 0, best[x] = min over b = 1..x (T_b >= 0) of best[x - b] + T_b,
// b scanned ascending and replaced only on a strictly smaller total (the last
// group is the smallest one that attains the minimum).  The groups are then
// reported largest first.
tp_status tp_dp_batch_split(const int64_t* T_b, int B, int* out_sizes, int* out_D,
                            int64_t* out_total) {
  if (!T_b || !out_sizes || !out_D || !out_total || B < 1) return TP_ERR_INVALID;
  std::vector<int64_t> best(B + 1, INF);
  std::vector<int> last(B + 1, 0);
  best[0] = 0;
  for (int x = 1; x <= B; ++x)
    for (int b = 1; b <= x; ++b) {
      const int64_t t = T_b[b - 1];
      if (t < 0 || best[x - b] == INF) continue;
      if (best[x - b] > INF - t) return TP_ERR_INVALID;  // overflow
      const int64_t v = best[x - b] + t;
      if (v < best[x]) {
        best[x] = v;
        last[x] = b;
      }
    }
  if (best[B] == INF) return TP_ERR_INVALID;
  std::vector<int> sizes;
  for (int x = B; x > 0; x -= last[x]) sizes.push_back(last[x]);
  std::sort(sizes.begin(), sizes.end(), [](int a, int b) { return a > b; });
  for (size_t i = 0; i < sizes.size(); ++i) out_sizes[i] = sizes[i];
  *out_D = (int)sizes.size();
  *out_total = best[B];
  return TP_OK;
}

// Joint batch x token plan (Sec. 3.4): the token DP of Sec. 3.3 for every
// group size b = 1..B on that size's cost table, then the batch split over the
// resulting T_b.
tp_status tp_dp_joint_slicing(const int64_t* costs, int B, int L_units, int unit, int K,
                              int64_t eps_ns, int* out_sizes, int* out_D, int* out_lens,
                              int* out_M, int64_t* out_T_b, int64_t* out_total) {
  if (!costs || !out_sizes || !out_D || !out_lens || !out_M || !out_T_b || !out_total || B < 1 ||
      L_units < 1)
    return TP_ERR_INVALID;
  const size_t plane = (size_t)L_units * L_units;
  std::vector<std::vector<int>> lens(B, std::vector<int>(L_units));
  std::vector<int> M(B, 0);
  for (int b = 1; b <= B; ++b) {
    const tp_status s = tp_dp_optimal_slicing(costs + (b - 1) * plane, L_units, unit, K, eps_ns,
                                              lens[b - 1].data(), &M[b - 1], &out_T_b[b - 1]);
    if (s != TP_OK) return s;
  }
  const tp_status s = tp_dp_batch_split(out_T_b, B, out_sizes, out_D, out_total);
  if (s != TP_OK) return s;
  for (int g = 0; g < *out_D; ++g) {
    const int b = out_sizes[g];
    out_M[g] = M[b - 1];
    std::copy(lens[b - 1].begin(), lens[b - 1].begin() + M[b - 1], out_lens + (size_t)g * L_units);
  }
  return TP_OK;
}
