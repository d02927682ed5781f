// CPU-only driver run under AddressSanitizer and UndefinedBehaviorSanitizer
// (tests/test_sanitizers.py builds it): the host planner (Sec. 3.3 DP,
// Algorithm 1; Sec. 3.4 batch split and joint plan), the Eq. 9 cost model and
// the C oracle of the stage, exercised on seeded inputs including the error
// paths.  Every check that fails prints a line and makes the exit status
// nonzero; a sanitizer report aborts the run.
//
// Test infrastructure: it links the oracle next to the product's host code
// only to compare them; neither uses the other.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "../../include/terapipe.h"

extern "C" {
// the oracle's C interface (oracle/tp_oracle.c)
typedef struct {
  const double *ln1_g, *ln1_b, *w_qkv, *b_qkv, *w_o, *b_o;
  const double *ln2_g, *ln2_b, *w1, *b1, *w2, *b2;
} or_params;
typedef struct {
  double *ln1_g, *ln1_b, *w_qkv, *b_qkv, *w_o, *b_o;
  double *ln2_g, *ln2_b, *w1, *b1, *w2, *b2;
} or_grads;
struct or_stage;
or_stage* or_stage_create(int n_layers, int H, int heads, int Lmax, double eps,
                          const or_params* p, or_grads* g);
void or_stage_destroy(or_stage* S);
void or_reset(or_stage* S);
int or_forward(or_stage* S, int l, int r, const double* x, double* y);
int or_backward(or_stage* S, int l, int r, const double* dy, double* dx);
int or_dp_optimal_slicing(const int64_t* cost, int U, int K, int64_t eps, int* out_units,
                          int* out_M, int64_t* out_T, int64_t* out_tmax, int* out_evaluated);
}

// Stand-in for the device profiler (the stage library's tp_profile_slice_cost
// is not linked into this CPU build): t_fwd = 1000 + 40 len + 2 ctx + len ctx / 8
// and t_bwd twice that, -1 past max_seq, so tp_profile_cost_model's
// orchestration runs here; its fit must then recover the overhead exactly.
static const int kFakeMaxSeq = 256;
extern "C" tp_status tp_profile_slice_cost(tp_stage* stage, const int* lens, int n_lens,
                                           const int* ctxs, int n_ctxs, int warmup, int reps,
                                           int64_t* t_fwd_ns, int64_t* t_bwd_ns) {
  if (!stage || !lens || !ctxs || !t_fwd_ns || !t_bwd_ns || n_lens < 1 || n_ctxs < 1 ||
      warmup < 0 || reps < 1)
    return TP_ERR_INVALID;
  for (int a = 0; a < n_lens; ++a)
    for (int b = 0; b < n_ctxs; ++b) {
      const int64_t n = lens[a], c = ctxs[b];
      const size_t i = (size_t)a * n_ctxs + b;
      if (n + c > kFakeMaxSeq) {
        t_fwd_ns[i] = t_bwd_ns[i] = -1;
      } else {
        t_fwd_ns[i] = 1000 + 40 * n + 2 * c + n * c / 8;
        t_bwd_ns[i] = 2 * t_fwd_ns[i];
      }
    }
  return TP_OK;
}

static int failures = 0;
#define CHECK(cond, ...)                     \
  do {                                       \
    if (!(cond)) {                           \
      ++failures;                            \
      std::printf("FAIL %s:%d: ", __FILE__, __LINE__); \
      std::printf(__VA_ARGS__);              \
      std::printf("\n");                     \
    }                                        \
  } while (0)

// SplitMix64: seeded, portable
struct Rng {
  uint64_t s;
  explicit Rng(uint64_t seed) : s(seed) {}
  uint64_t next() {
    uint64_t z = (s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  double uniform() { return (double)(next() >> 11) * (1.0 / 9007199254740992.0); }
  int below(int n) { return (int)(next() % (uint64_t)n); }
};

// cost tables of several shapes: random, tie-heavy, Eq. 9-like (linear in
// length and context), with -1 in the entries past the sequence end
static std::vector<int64_t> table(int U, int family, Rng& g) {
  std::vector<int64_t> c((size_t)U * U, -1);
  for (int k = 1; k <= U; ++k)
    for (int j = 0; j + k <= U; ++j) {
      int64_t v;
      if (family == 0) v = 1 + g.below(1000);
      else if (family == 1) v = 10 * (1 + g.below(4));
      else v = 500 + 97 * k + 3 * j + k * j + g.below(5);
      c[(size_t)(k - 1) * U + j] = v;
    }
  return c;
}

static void dp_against_oracle() {
  Rng g(7);
  int cases = 0;
  for (int U : {1, 2, 3, 5, 8, 13, 24, 40, 64})
    for (int family = 0; family < 3; ++family)
      for (int K : {1, 2, 3, 8, 48})
        for (int64_t eps : {0, 5, 50}) {
          const std::vector<int64_t> c = table(U, family, g);
          std::vector<int> lens(U), units(U);
          int M = -1, Mo = -1;
          int64_t T = -1, To = -1;
          const tp_status st = tp_dp_optimal_slicing(c.data(), U, 16, K, eps, lens.data(), &M, &T);
          const int ro = or_dp_optimal_slicing(c.data(), U, K, eps, units.data(), &Mo, &To,
                                               nullptr, nullptr);
          CHECK(st == TP_OK && ro == 0, "dp status %d / %d (U %d K %d)", st, ro, U, K);
          CHECK(M == Mo && T == To, "dp M %d/%d T %lld/%lld (U %d fam %d K %d eps %lld)", M, Mo,
                (long long)T, (long long)To, U, family, K, (long long)eps);
          int sum = 0;
          for (int i = 0; i < M && i < U; ++i) {
            CHECK(lens[i] == 16 * units[i], "dp slice %d: %d vs %d units", i, lens[i], units[i]);
            sum += lens[i];
          }
          CHECK(sum == 16 * U, "dp slices sum to %d, not %d", sum, 16 * U);
          ++cases;
        }
  std::printf("dp: %d tables\n", cases);
}

static void dp_errors() {
  const int U = 4;
  std::vector<int64_t> c((size_t)U * U, 5);
  std::vector<int> lens(U);
  int M = 0;
  int64_t T = 0;
  CHECK(tp_dp_optimal_slicing(nullptr, U, 1, 2, 0, lens.data(), &M, &T) == TP_ERR_INVALID, "null");
  CHECK(tp_dp_optimal_slicing(c.data(), 0, 1, 2, 0, lens.data(), &M, &T) == TP_ERR_INVALID, "U 0");
  CHECK(tp_dp_optimal_slicing(c.data(), U, 0, 2, 0, lens.data(), &M, &T) == TP_ERR_INVALID, "unit 0");
  CHECK(tp_dp_optimal_slicing(c.data(), U, 1, 0, 0, lens.data(), &M, &T) == TP_ERR_INVALID, "K 0");
  CHECK(tp_dp_optimal_slicing(c.data(), U, 1, 2, -1, lens.data(), &M, &T) == TP_ERR_INVALID, "eps");
  c[2] = -3;  // a used entry (k = 1, j = 2)
  CHECK(tp_dp_optimal_slicing(c.data(), U, 1, 2, 0, lens.data(), &M, &T) == TP_ERR_INVALID, "neg");
}

static void batch_and_joint() {
  Rng g(11);
  for (int B = 1; B <= 12; ++B) {
    std::vector<int64_t> Tb(B);
    for (int b = 0; b < B; ++b) Tb[b] = 100 + 60 * (b + 1) + g.below(50);
    if (B > 3) Tb[2] = -1;  // an unusable size
    std::vector<int> sizes(B);
    int D = 0;
    int64_t tot = 0;
    const tp_status st = tp_dp_batch_split(Tb.data(), B, sizes.data(), &D, &tot);
    CHECK(st == TP_OK, "batch split status %d (B %d)", st, B);
    int n = 0;
    int64_t s = 0;
    for (int i = 0; i < D; ++i) {
      CHECK(sizes[i] >= 1 && sizes[i] <= B && Tb[sizes[i] - 1] >= 0, "group size %d", sizes[i]);
      if (i) CHECK(sizes[i] <= sizes[i - 1], "groups not largest first");
      n += sizes[i];
      s += Tb[sizes[i] - 1];
    }
    CHECK(n == B && s == tot, "batch split covers %d of %d, sum %lld vs %lld", n, B,
          (long long)s, (long long)tot);
  }
  // joint plan over B tables
  const int B = 3, U = 12;
  std::vector<int64_t> costs;
  for (int b = 0; b < B; ++b) {
    std::vector<int64_t> c = table(U, 2, g);
    for (auto& v : c)
      if (v >= 0) v = v * (b + 2) / 2;
    costs.insert(costs.end(), c.begin(), c.end());
  }
  std::vector<int> sizes(B), M(B), lens(B * U);
  std::vector<int64_t> Tb(B);
  int D = 0;
  int64_t tot = 0;
  const tp_status st = tp_dp_joint_slicing(costs.data(), B, U, 16, 8, 0, sizes.data(), &D,
                                           lens.data(), M.data(), Tb.data(), &tot);
  CHECK(st == TP_OK, "joint status %d", st);
  for (int gi = 0; gi < D; ++gi) {
    int sum = 0;
    for (int i = 0; i < M[gi]; ++i) sum += lens[gi * U + i];
    CHECK(sum == 16 * U, "joint group %d covers %d tokens", gi, sum);
  }
  std::vector<int> sz1(1);
  int64_t bad = -1;
  CHECK(tp_dp_batch_split(&bad, 1, sz1.data(), &D, &tot) == TP_ERR_INVALID, "no usable size");
}

static void cost_model() {
  // exactly linear overheads are recovered: a0 + a1 i + a2 j + a3 i j
  const int U = 16, unit = 16;
  const double a[4] = {1500.0, 3.0, 7.0, 0.25};
  std::vector<int64_t> t0(U);
  for (int k = 1; k <= U; ++k) t0[k - 1] = 10000 + 900 * k;
  std::vector<int> sl, sc;
  std::vector<int64_t> stt;
  for (int k : {1, 2, 4, 8})
    for (int j : {1, 2, 4, 8}) {
      if (k + j > U) continue;
      const double i = k * unit, c = j * unit;
      sl.push_back(k * unit);
      sc.push_back(j * unit);
      stt.push_back(t0[k - 1] + (int64_t)(a[0] + a[1] * i + a[2] * c + a[3] * i * c));
    }
  double coef[4];
  CHECK(tp_fit_ctx_model(t0.data(), U, unit, sl.data(), sc.data(), stt.data(), (int)sl.size(),
                         coef) == TP_OK, "fit status");
  for (int q = 0; q < 4; ++q)
    CHECK(std::abs(coef[q] - a[q]) <= 1e-6 * (1 + std::abs(a[q])), "coef %d %.9g vs %.9g", q,
          coef[q], a[q]);
  std::vector<int64_t> cost((size_t)U * U);
  CHECK(tp_cost_table_from_model(t0.data(), U, unit, coef, cost.data()) == TP_OK, "table");
  for (int k = 1; k <= U; ++k)
    for (int j = 0; j < U; ++j) {
      const int64_t v = cost[(size_t)(k - 1) * U + j];
      if (k + j > U) CHECK(v == -1, "past-end entry %lld", (long long)v);
      else if (j == 0) CHECK(v == t0[k - 1], "j = 0 entry");
      else CHECK(v > t0[k - 1], "overhead entry");
    }
  // too few samples, one context only
  CHECK(tp_fit_ctx_model(t0.data(), U, unit, sl.data(), sc.data(), stt.data(), 3, coef) ==
            TP_ERR_INVALID, "3 samples");
  std::vector<int> one_ctx(sl.size(), 16);
  CHECK(tp_fit_ctx_model(t0.data(), U, unit, sl.data(), one_ctx.data(), stt.data(),
                         (int)sl.size(), coef) == TP_ERR_INVALID, "single context");
}

static void profile_model_orchestration() {
  // overhead of t_fwd + t_bwd: 3 (2 c + n c / 8) = 6 c + 0.375 n c, exactly
  // representable when n c / 8 is an integer (n a multiple of 16)
  const int U = 16, unit = 16;
  const int sub_lens[] = {16, 32, 64, 128}, sub_ctxs[] = {16, 64, 128};
  std::vector<int64_t> cost((size_t)U * U);
  double coef[4];
  int dummy = 0;
  tp_stage* fake = reinterpret_cast<tp_stage*>(&dummy);  // opaque, never dereferenced here
  const tp_status st = tp_profile_cost_model(fake, U, unit, sub_lens, 4, sub_ctxs, 3, 1, 3,
                                             cost.data(), coef);
  CHECK(st == TP_OK, "profile_cost_model status %d", st);
  const double want[4] = {0.0, 0.0, 6.0, 0.375};
  for (int q = 0; q < 4; ++q)
    CHECK(std::abs(coef[q] - want[q]) < 1e-6, "profiled coef %d %.9g vs %.9g", q, coef[q], want[q]);
  for (int k = 1; k <= U; ++k)
    for (int j = 0; k + j <= U; ++j) {
      const int64_t n = k * unit, c = j * unit;
      const int64_t exact = 3 * (1000 + 40 * n + 2 * c + n * c / 8);
      CHECK(cost[(size_t)(k - 1) * U + j] == exact, "model table (%d, %d): %lld vs %lld", k, j,
            (long long)cost[(size_t)(k - 1) * U + j], (long long)exact);
    }
  // arguments the profiler cannot take are rejected before any measurement
  const int bad_len[] = {24};
  CHECK(tp_profile_cost_model(fake, U, unit, bad_len, 1, sub_ctxs, 3, 1, 3, cost.data(), coef) ==
            TP_ERR_INVALID, "length off the unit grid accepted");
  CHECK(tp_profile_cost_model(nullptr, U, unit, sub_lens, 4, sub_ctxs, 3, 1, 3, cost.data(),
                              coef) == TP_ERR_INVALID, "null stage accepted");
}

static void oracle_stage() {
  // tiny stage: 2 layers, H = 16, 4 heads, L = 12; whole vs sliced bitwise
  const int NL = 2, H = 16, heads = 4, L = 12;
  Rng g(3);
  std::vector<std::vector<double>> P(NL * 12), G1(NL * 12), G2(NL * 12);
  const size_t sizes[12] = {(size_t)H, (size_t)H, (size_t)3 * H * H, (size_t)3 * H,
                            (size_t)H * H, (size_t)H, (size_t)H, (size_t)H,
                            (size_t)4 * H * H, (size_t)4 * H, (size_t)4 * H * H, (size_t)H};
  std::vector<or_params> op(NL);
  std::vector<or_grads> og1(NL), og2(NL);
  for (int li = 0; li < NL; ++li) {
    for (int k = 0; k < 12; ++k) {
      auto& v = P[li * 12 + k];
      v.resize(sizes[k]);
      for (auto& e : v) e = (k == 0 || k == 6 ? 1.0 : 0.0) + 0.1 * (g.uniform() - 0.5);
      G1[li * 12 + k].assign(sizes[k], 0.0);
      G2[li * 12 + k].assign(sizes[k], 0.0);
    }
    const double** pp = (const double**)&op[li];
    double** g1 = (double**)&og1[li];
    double** g2 = (double**)&og2[li];
    for (int k = 0; k < 12; ++k) {
      pp[k] = P[li * 12 + k].data();
      g1[k] = G1[li * 12 + k].data();
      g2[k] = G2[li * 12 + k].data();
    }
  }
  std::vector<double> x((size_t)L * H), dy((size_t)L * H);
  for (auto& e : x) e = g.uniform() - 0.5;
  for (auto& e : dy) e = g.uniform() - 0.5;
  auto run = [&](or_grads* gr, const std::vector<int>& fwd, const std::vector<int>& bwd,
                 std::vector<double>& y, std::vector<double>& dx) {
    or_stage* S = or_stage_create(NL, H, heads, L, 1e-5, op.data(), gr);
    CHECK(S != nullptr, "or_stage_create");
    if (!S) return;
    or_reset(S);
    y.assign((size_t)L * H, 0.0);
    dx.assign((size_t)L * H, 0.0);
    int l = 0;
    for (int n : fwd) {
      CHECK(or_forward(S, l, l + n, x.data() + (size_t)l * H, y.data() + (size_t)l * H) == 0,
            "or_forward");
      l += n;
    }
    // out of order: must be rejected
    CHECK(or_forward(S, 0, 1, x.data(), y.data()) != 0, "forward out of order accepted");
    int r = L;
    for (int n : bwd) {
      CHECK(or_backward(S, r - n, r, dy.data() + (size_t)(r - n) * H,
                        dx.data() + (size_t)(r - n) * H) == 0, "or_backward");
      r -= n;
    }
    or_stage_destroy(S);
  };
  std::vector<double> y1, dx1, y2, dx2;
  run(og1.data(), {12}, {12}, y1, dx1);
  run(og2.data(), {3, 4, 5}, {2, 7, 3}, y2, dx2);
  CHECK(std::memcmp(y1.data(), y2.data(), y1.size() * 8) == 0, "oracle y not slicing-invariant");
  CHECK(std::memcmp(dx1.data(), dx2.data(), dx1.size() * 8) == 0, "oracle dx not invariant");
  for (size_t k = 0; k < G1.size(); ++k)
    CHECK(std::memcmp(G1[k].data(), G2[k].data(), G1[k].size() * 8) == 0,
          "oracle gradient %zu not invariant", k);
}

int main() {
  dp_against_oracle();
  dp_errors();
  batch_and_joint();
  cost_model();
  profile_model_orchestration();
  oracle_stage();
  std::printf("%s (%d failures)\n", failures ? "FAILED" : "OK", failures);
  return failures ? 1 : 0;
}
