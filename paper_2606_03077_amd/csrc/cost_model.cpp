// Cost evaluator polynomials and the rollout partition DP (Sec. 4.2, Sec. 4.5, Alg. 1,
// App. B.1).  Host arithmetic only.
#include <algorithm>
#include <cmath>
#include <limits>
#include <new>
#include <numeric>
#include <vector>

#include "internal.h"

namespace libra {
namespace {

constexpr int64_t kMaxLen = int64_t(1) << 24;

bool finite_nonneg(double x) { return std::isfinite(x) && x >= 0.0; }

double poly_eval(const libra_ce_poly& p, double L) { return (p.gamma * L + p.eta) * L + p.theta; }

// sum_{l=a}^{b} T(l) written over the count m = b - a + 1 so that no large terms cancel:
// sum l = m a + m(m-1)/2, sum l^2 = m a^2 + a m(m-1) + (m-1) m (2m-1) / 6.
double poly_sum(const libra_ce_poly& p, int64_t a, int64_t b) {
  if (b < a) return 0.0;
  const long double A = a, m = (long double)(b - a + 1);
  const long double s1 = m * A + m * (m - 1) / 2;
  const long double s2 = m * A * A + A * m * (m - 1) + (m - 1) * m * (2 * m - 1) / 6;
  return double((long double)p.gamma * s2 + (long double)p.eta * s1 + (long double)p.theta * m);
}

int tp_slot(int tp) {
  switch (tp) {
    case 1: return 0;
    case 2: return 1;
    case 4: return 2;
    case 8: return 3;
    default: return -1;
  }
}

libra_status rollout_dp(const int64_t* lengths, int32_t n_req, int32_t n_gpus,
                        const int32_t* tp_set, int32_t n_tp, const int* slot,
                        const libra_rollout_model& m, bool exact, double* makespan,
                        int32_t* order, int32_t* instances, int32_t* n_instances) {
  const libra_rollout_model* model = &m;
  // Sort requests by (length, index); per-request trajectory attention A(len).
  std::vector<int32_t> ord(n_req);
  std::iota(ord.begin(), ord.end(), 0);
  std::stable_sort(ord.begin(), ord.end(),
                   [&](int32_t x, int32_t y) { return lengths[x] < lengths[y]; });
  std::vector<double> len(n_req), prefix(size_t(n_req) + 1, 0.0);
  for (int32_t j = 0; j < n_req; ++j) {
    len[j] = double(lengths[ord[j]]);
    const double A = poly_sum(model->attn_step, 1, lengths[ord[j]]);
    if (!finite_nonneg(A)) return set_error(LIBRA_E_INVAL, "attention model gives a negative time");
    prefix[j + 1] = prefix[j] + A;
  }
  // Cost of an instance of TP slot s over sorted positions [i - x, i) (0-based).
  auto cost = [&](int s, int32_t i, int32_t x) -> double {
    if (x == 0) return 0.0;
    return model->linear_step[s] * len[i - 1] + model->attn_scale[s] * (prefix[i] - prefix[i - x]);
  };

  const double inf = std::numeric_limits<double>::infinity();
  const size_t W = size_t(n_req) + 1;
  std::vector<double> dp(size_t(n_gpus + 1) * W, inf);
  std::vector<int32_t> pick_t(size_t(n_gpus + 1) * W, -1), pick_x(size_t(n_gpus + 1) * W, -1);
  dp[0] = 0.0;
  for (int32_t g = 1; g <= n_gpus; ++g) {
    for (int32_t i = 0; i <= n_req; ++i) {
      double best = inf;
      int32_t bt = -1, bx = -1;
      for (int t = 0; t < n_tp; ++t) {
        const int tp = tp_set[t];
        if (tp > g) continue;
        const double* prev = &dp[size_t(g - tp) * W];
        if (exact) {
          for (int32_t x = 0; x <= i; ++x) {
            const double c = std::max(prev[i - x], cost(slot[t], i, x));
            if (c < best) { best = c; bt = t; bx = x; }
          }
        } else {
          // prev[i - x] does not increase with x, cost does not decrease: the max is
          // smallest where they cross.  Find the first x with cost >= prev[i - x].
          int32_t lo = 0, hi = i + 1;
          while (lo < hi) {
            const int32_t mid = lo + (hi - lo) / 2;
            if (cost(slot[t], i, mid) >= prev[i - mid]) hi = mid; else lo = mid + 1;
          }
          for (int32_t x = std::max(0, lo - 1); x <= std::min(i, lo); ++x) {
            const double c = std::max(prev[i - x], cost(slot[t], i, x));
            if (c < best) { best = c; bt = t; bx = x; }
          }
        }
      }
      dp[size_t(g) * W + i] = best;
      pick_t[size_t(g) * W + i] = bt;
      pick_x[size_t(g) * W + i] = bx;
    }
  }
  for (int32_t j = 0; j < n_req; ++j) order[j] = ord[j];
  *makespan = dp[size_t(n_gpus) * W + n_req];
  int32_t k = 0;
  if (std::isfinite(*makespan)) {
    int32_t g = n_gpus, i = n_req;
    while (g > 0) {
      const int32_t t = pick_t[size_t(g) * W + i], x = pick_x[size_t(g) * W + i];
      instances[3 * k + 0] = tp_set[t];
      instances[3 * k + 1] = i - x;
      instances[3 * k + 2] = x;
      ++k;
      g -= tp_set[t];
      i -= x;
    }
  }
  *n_instances = k;
  return LIBRA_OK;
}

}  // namespace
}  // namespace libra

using namespace libra;

extern "C" {

libra_status libra_ce_fit(const double* lengths, const double* times, int32_t n,
                          libra_ce_poly* out) {
  if (!lengths || !times || !out) return set_error(LIBRA_E_INVAL, "NULL argument");
  if (n < 3) return set_error(LIBRA_E_INVAL, "need at least 3 points");
  double lmax = 0.0;
  for (int32_t i = 0; i < n; ++i) {
    if (!finite_nonneg(lengths[i])) return set_error(LIBRA_E_INVAL, "lengths must be finite, >= 0");
    if (!std::isfinite(times[i]) || times[i] <= 0.0)
      return set_error(LIBRA_E_INVAL, "times must be finite and > 0");
    lmax = std::max(lmax, lengths[i]);
  }
  std::vector<double> distinct(lengths, lengths + n);
  std::sort(distinct.begin(), distinct.end());
  if (std::unique(distinct.begin(), distinct.end()) - distinct.begin() < 3)
    return set_error(LIBRA_E_INVAL, "need at least 3 distinct lengths");
  // Weighted design: row i = (x_i^2, x_i, 1) / t_i with x = L / lmax, target 1, so the
  // residual of row i is the relative error of point i.  Solved by Householder QR.
  const double s = lmax;
  std::vector<double> a(size_t(n) * 3), r(n);
  for (int32_t i = 0; i < n; ++i) {
    const double x = lengths[i] / s, w = 1.0 / times[i];
    a[size_t(i) * 3 + 0] = w * x * x;
    a[size_t(i) * 3 + 1] = w * x;
    a[size_t(i) * 3 + 2] = w;
    r[i] = 1.0;
  }
  double diag[3];
  for (int c = 0; c < 3; ++c) {
    double norm = 0.0;
    for (int32_t i = c; i < n; ++i) norm += a[size_t(i) * 3 + c] * a[size_t(i) * 3 + c];
    norm = std::sqrt(norm);
    if (!(norm > 0.0)) return set_error(LIBRA_E_INVAL, "degenerate fit");
    const double alpha = a[size_t(c) * 3 + c] > 0 ? -norm : norm;
    // v = column c below the diagonal with v_c = a_cc - alpha; H = I - 2 v v^T / v^T v
    std::vector<double> v(size_t(n - c));
    for (int32_t i = c; i < n; ++i) v[i - c] = a[size_t(i) * 3 + c];
    v[0] -= alpha;
    double vv = 0.0;
    for (double e : v) vv += e * e;
    if (vv > 0.0) {
      for (int k = c; k < 3; ++k) {
        double d = 0.0;
        for (int32_t i = c; i < n; ++i) d += v[i - c] * a[size_t(i) * 3 + k];
        const double f = 2.0 * d / vv;
        for (int32_t i = c; i < n; ++i) a[size_t(i) * 3 + k] -= f * v[i - c];
      }
      double d = 0.0;
      for (int32_t i = c; i < n; ++i) d += v[i - c] * r[i];
      const double f = 2.0 * d / vv;
      for (int32_t i = c; i < n; ++i) r[i] -= f * v[i - c];
    }
    diag[c] = a[size_t(c) * 3 + c];
    if (std::fabs(diag[c]) <= 1e-14 * norm) return set_error(LIBRA_E_INVAL, "degenerate fit");
  }
  double c2 = r[2] / diag[2];
  double c1 = (r[1] - a[1 * 3 + 2] * c2) / diag[1];
  double c0 = (r[0] - a[0 * 3 + 1] * c1 - a[0 * 3 + 2] * c2) / diag[0];
  out->gamma = c0 / (s * s);
  out->eta = c1 / s;
  out->theta = c2;
  return LIBRA_OK;
}

libra_status libra_ce_mape(const libra_ce_poly* poly, const double* lengths, const double* times,
                           int32_t n, double* mape) {
  if (!poly || !lengths || !times || !mape) return set_error(LIBRA_E_INVAL, "NULL argument");
  if (n < 1) return set_error(LIBRA_E_INVAL, "need at least one point");
  double acc = 0.0;
  for (int32_t i = 0; i < n; ++i) {
    if (!std::isfinite(times[i]) || times[i] <= 0.0)
      return set_error(LIBRA_E_INVAL, "times must be finite and > 0");
    acc += std::fabs(poly_eval(*poly, lengths[i]) - times[i]) / times[i];
  }
  *mape = 100.0 * acc / n;
  return LIBRA_OK;
}

libra_status libra_ce_poly_sum(const libra_ce_poly* poly, int64_t a, int64_t b, double* out) {
  if (!poly || !out) return set_error(LIBRA_E_INVAL, "NULL argument");
  if (a < 0 || b < 0 || a > kMaxLen || b > kMaxLen)
    return set_error(LIBRA_E_INVAL, "a and b must be in [0, 2^24]");
  *out = poly_sum(*poly, a, b);
  return LIBRA_OK;
}

libra_status libra_rollout_dp(const int64_t* lengths, int32_t n_req, int32_t n_gpus,
                              const int32_t* tp_set, int32_t n_tp,
                              const libra_rollout_model* model, int32_t exact, double* makespan,
                              int32_t* order, int32_t* instances, int32_t* n_instances) {
  if (!model || !makespan || !n_instances || !tp_set || (n_req > 0 && (!lengths || !order)) ||
      (n_gpus > 0 && !instances))
    return set_error(LIBRA_E_INVAL, "NULL argument");
  if (n_req < 0 || n_req > 65536) return set_error(LIBRA_E_INVAL, "n_req must be in [0, 65536]");
  if (n_gpus < 0 || n_gpus > 4096) return set_error(LIBRA_E_INVAL, "n_gpus must be in [0, 4096]");
  if (n_tp < 1 || n_tp > 4) return set_error(LIBRA_E_INVAL, "n_tp must be in [1, 4]");
  int slot[4];
  for (int t = 0; t < n_tp; ++t) {
    slot[t] = tp_slot(tp_set[t]);
    if (slot[t] < 0) return set_error(LIBRA_E_INVAL, "TP degrees must come from {1, 2, 4, 8}");
    for (int u = 0; u < t; ++u)
      if (tp_set[u] == tp_set[t]) return set_error(LIBRA_E_INVAL, "TP degrees must be distinct");
    if (!finite_nonneg(model->linear_step[slot[t]]) || !finite_nonneg(model->attn_scale[slot[t]]))
      return set_error(LIBRA_E_INVAL, "model times must be finite and >= 0");
  }
  for (int32_t i = 0; i < n_req; ++i)
    if (lengths[i] < 0 || lengths[i] > kMaxLen)
      return set_error(LIBRA_E_INVAL, "lengths must be in [0, 2^24]");
  if (int64_t(n_gpus + 1) * (int64_t(n_req) + 1) > (int64_t(1) << 26))
    return set_error(LIBRA_E_INVAL, "(n_gpus + 1) * (n_req + 1) must be <= 2^26 states");
  try {
    return rollout_dp(lengths, n_req, n_gpus, tp_set, n_tp, slot, *model, exact != 0, makespan,
                      order, instances, n_instances);
  } catch (const std::bad_alloc&) {
    return set_error(LIBRA_E_NOMEM, "DP tables do not fit in host memory");
  }
}

}  // extern "C"

