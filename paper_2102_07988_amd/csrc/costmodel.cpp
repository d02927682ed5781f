// Cost estimate of Sec. 3.3 ("Estimating t_fwd", Eq. 9): the cost of a slice
// of i tokens after j tokens of context is t(i, 0), measured for every length,
// plus a context overhead t_ctx(i, j) = a0 + a1 i + a2 j + a3 i j fitted by
// least squares to a subset of measured (i, j > 0) points.  Host code.
//
// The fit solves the 4-column least-squares problem by Householder QR on the
// design with i and j divided by the sequence length (so the four columns have
// comparable norms), then scales the coefficients back to tokens.
#include <cmath>
#include <cstdint>
#include <vector>

#include "../../include/terapipe.h"

namespace {

// Least squares min |A b - y| for an n x 4 row-major A (n >= 4) by Householder
// QR.  Returns false if a column is (numerically) dependent on the others.
bool lsq4(std::vector<double>& A, std::vector<double>& y, int n, double b[4]) {
  double col_norm[4];
  for (int c = 0; c < 4; ++c) {
    double s = 0;
    for (int r = 0; r < n; ++r) s += A[r * 4 + c] * A[r * 4 + c];
    col_norm[c] = std::sqrt(s);
    if (col_norm[c] == 0) return false;
  }
  std::vector<double> v(n);
  for (int k = 0; k < 4; ++k) {
    double s = 0;
    for (int r = k; r < n; ++r) s += A[r * 4 + k] * A[r * 4 + k];
    const double norm = std::sqrt(s);
    if (norm <= 1e-10 * col_norm[k]) return false;
    const double alpha = A[k * 4 + k] > 0 ? -norm : norm;
    double vv = 0;
    for (int r = k; r < n; ++r) {
      v[r] = A[r * 4 + k] - (r == k ? alpha : 0.0);
      vv += v[r] * v[r];
    }
    if (vv == 0) continue;
    for (int c = k; c < 4; ++c) {
      double d = 0;
      for (int r = k; r < n; ++r) d += v[r] * A[r * 4 + c];
      const double f = 2 * d / vv;
      for (int r = k; r < n; ++r) A[r * 4 + c] -= f * v[r];
    }
    double d = 0;
    for (int r = k; r < n; ++r) d += v[r] * y[r];
    const double f = 2 * d / vv;
    for (int r = k; r < n; ++r) y[r] -= f * v[r];
  }
  for (int k = 3; k >= 0; --k) {
    double s = y[k];
    for (int c = k + 1; c < 4; ++c) s -= A[k * 4 + c] * b[c];
    b[k] = s / A[k * 4 + k];
  }
  return true;
}

}  // namespace

extern "C" {

tp_status tp_fit_ctx_model(const int64_t* t0_ns, int L_units, int unit, const int* s_len,
                           const int* s_ctx, const int64_t* s_t_ns, int n_samples,
                           double* coef) {
  if (!t0_ns || !s_len || !s_ctx || !s_t_ns || !coef || L_units < 1 || unit < 1 ||
      n_samples < 4)
    return TP_ERR_INVALID;
  const long L = (long)L_units * unit;
  const double scale = (double)L;
  std::vector<double> A((size_t)n_samples * 4), y(n_samples);
  for (int s = 0; s < n_samples; ++s) {
    const int i = s_len[s], j = s_ctx[s];
    if (i < 1 || i % unit || j < 1 || (long)i + j > L || s_t_ns[s] < 0) return TP_ERR_INVALID;
    const int64_t base = t0_ns[i / unit - 1];
    if (base < 0) return TP_ERR_INVALID;
    const double x = i / scale, z = j / scale;
    A[s * 4 + 0] = 1.0;
    A[s * 4 + 1] = x;
    A[s * 4 + 2] = z;
    A[s * 4 + 3] = x * z;
    y[s] = (double)(s_t_ns[s] - base);
  }
  double b[4];
  if (!lsq4(A, y, n_samples, b)) return TP_ERR_INVALID;
  coef[0] = b[0];
  coef[1] = b[1] / scale;
  coef[2] = b[2] / scale;
  coef[3] = b[3] / (scale * scale);
  return TP_OK;
}

tp_status tp_cost_table_from_model(const int64_t* t0_ns, int L_units, int unit, const double* coef,
                                   int64_t* cost) {
  if (!t0_ns || !coef || !cost || L_units < 1 || unit < 1) return TP_ERR_INVALID;
  for (int k = 0; k < L_units; ++k)
    if (t0_ns[k] < 0) return TP_ERR_INVALID;
  for (int k = 1; k <= L_units; ++k)
    for (int j = 0; j < L_units; ++j) {
      int64_t& out = cost[(size_t)(k - 1) * L_units + j];
      if (k + j > L_units) {
        out = -1;
      } else if (j == 0) {
        out = t0_ns[k - 1];
      } else {
        const double i = (double)k * unit, c = (double)j * unit;
        const double pred = coef[0] + coef[1] * i + coef[2] * c + coef[3] * i * c;
        const int64_t v = t0_ns[k - 1] + (int64_t)std::llround(pred);
        out = v < 0 ? 0 : v;
      }
    }
  return TP_OK;
}

tp_status tp_profile_cost_model(tp_stage* stage, int L_units, int unit, const int* sub_lens,
                                int n_sub_lens, const int* sub_ctxs, int n_sub_ctxs, int warmup,
                                int reps, int64_t* cost, double* coef) {
  if (!stage || !sub_lens || !sub_ctxs || !cost || !coef || L_units < 1 || unit < 1 ||
      n_sub_lens < 1 || n_sub_ctxs < 1)
    return TP_ERR_INVALID;
  const long L = (long)L_units * unit;
  for (int a = 0; a < n_sub_lens; ++a)
    if (sub_lens[a] < 1 || sub_lens[a] % unit || sub_lens[a] > L) return TP_ERR_INVALID;
  for (int b = 0; b < n_sub_ctxs; ++b)
    if (sub_ctxs[b] < 1 || sub_ctxs[b] >= L) return TP_ERR_INVALID;
  // t(i, 0) for every length
  std::vector<int> lens(L_units), zero(1, 0);
  for (int k = 0; k < L_units; ++k) lens[k] = (k + 1) * unit;
  std::vector<int64_t> f0(L_units), b0(L_units), t0(L_units);
  tp_status st = tp_profile_slice_cost(stage, lens.data(), L_units, zero.data(), 1, warmup, reps,
                                       f0.data(), b0.data());
  if (st != TP_OK) return st;
  for (int k = 0; k < L_units; ++k) {
    if (f0[k] < 0) return TP_ERR_INVALID;  // the stage holds fewer than L tokens
    t0[k] = f0[k] + b0[k];
  }
  // the subset
  const size_t n = (size_t)n_sub_lens * n_sub_ctxs;
  std::vector<int64_t> fs(n), bs(n);
  st = tp_profile_slice_cost(stage, sub_lens, n_sub_lens, sub_ctxs, n_sub_ctxs, warmup, reps,
                             fs.data(), bs.data());
  if (st != TP_OK) return st;
  std::vector<int> si, sj;
  std::vector<int64_t> stv;
  for (int a = 0; a < n_sub_lens; ++a)
    for (int b = 0; b < n_sub_ctxs; ++b) {
      if ((long)sub_lens[a] + sub_ctxs[b] > L) continue;
      const size_t idx = (size_t)a * n_sub_ctxs + b;
      si.push_back(sub_lens[a]);
      sj.push_back(sub_ctxs[b]);
      stv.push_back(fs[idx] + bs[idx]);
    }
  if (si.size() < 4) return TP_ERR_INVALID;
  st = tp_fit_ctx_model(t0.data(), L_units, unit, si.data(), sj.data(), stv.data(),
                        (int)si.size(), coef);
  if (st != TP_OK) return st;
  return tp_cost_table_from_model(t0.data(), L_units, unit, coef, cost);
}

}  // extern "C"
