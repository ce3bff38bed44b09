// Time-budget controller (host code): least-squares fit of the execution-time
// model, WCET, the closed-form eviction ratio alpha*, and the longest
// predictor input that finishes within the prefill phase.
//
// Model (TimeBill Sec. 4.2): prefill a N_x^2 + b N_x + c, decode step
// p N_kv + q with N_kv = (1 - alpha) N_x + i - 1 at step i (Eq. N_kv); the
// decode phase sums steps i = 1 .. N_hat_W - 1; WCET adds the prefill
// (Eq. wcet).  alpha* is the smallest alpha in [0, alpha_max] with
// t_predict + WCET(alpha) <= T (Sec. 5.1).  Solving that constraint gives
//   alpha* = 1 - (T - t_prefill - t_predict) / (p N_x (N_hat_W - 1))
//              + (N_hat_W - 2) / (2 N_x) + q / (p N_x),
// i.e. the paper's closed form with the second term divided by 2 N_x (the
// printed form also divides it by p, which is dimensionally inconsistent).
// The closed form needs p > 0; p = 0 (a step time that does not grow with the
// cache) makes WCET independent of alpha, and p < 0 is rejected.

#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <cmath>

#include "../../include/timebill.h"

namespace {

// Solve the (deg+1)x(deg+1) normal equations of a centred, scaled basis in
// long double, then map the coefficients back to powers of n.
int fit(const double* n, const double* t, int count, int deg, double* coef) {
  long double mean = 0, scale = 0;
  for (int i = 0; i < count; ++i) mean += n[i];
  mean /= count;
  for (int i = 0; i < count; ++i) scale = std::max(scale, fabsl(n[i] - mean));
  if (scale == 0) scale = 1;
  const int m = deg + 1;
  long double A[3][4] = {};
  for (int i = 0; i < count; ++i) {
    const long double x = (n[i] - mean) / scale;
    long double pw[3] = {1, x, x * x};
    for (int r = 0; r < m; ++r) {
      for (int c = 0; c < m; ++c) A[r][c] += pw[r] * pw[c];
      A[r][m] += pw[r] * t[i];
    }
  }
  for (int c = 0; c < m; ++c) {                      // Gauss-Jordan, partial pivoting
    int piv = c;
    for (int r = c + 1; r < m; ++r) if (fabsl(A[r][c]) > fabsl(A[piv][c])) piv = r;
    if (fabsl(A[piv][c]) < 1e-300L) return -1;
    for (int k = 0; k <= m; ++k) std::swap(A[c][k], A[piv][k]);
    for (int r = 0; r < m; ++r) {
      if (r == c) continue;
      const long double f = A[r][c] / A[c][c];
      for (int k = c; k <= m; ++k) A[r][k] -= f * A[c][k];
    }
  }
  long double u[3] = {0, 0, 0};                      // t = u0 + u1 x + u2 x^2, x = (n - mean)/scale
  for (int r = 0; r < m; ++r) u[r] = A[r][m] / A[r][r];
  const long double s = scale, mu = mean;
  if (deg == 1) {
    coef[0] = static_cast<double>(u[1] / s);
    coef[1] = static_cast<double>(u[0] - u[1] * mu / s);
  } else {
    coef[0] = static_cast<double>(u[2] / (s * s));
    coef[1] = static_cast<double>(u[1] / s - 2 * u[2] * mu / (s * s));
    coef[2] = static_cast<double>(u[0] - u[1] * mu / s + u[2] * mu * mu / (s * s));
  }
  return 0;
}

double prefill(const double* abc, double n_x) { return abc[0] * n_x * n_x + abc[1] * n_x + abc[2]; }

}  // namespace

extern "C" {

int32_t tb_ete_fit(const double* n, const double* t, int32_t count, int32_t degree,
                   double* coef) {
  if (!n || !t || !coef || (degree != 1 && degree != 2) || count < degree + 1) return -1;
  return fit(n, t, count, degree, coef);
}

double tb_wcet(const double* prefill_abc, const double* step_pq, double n_x, double alpha,
               int32_t n_hat_w) {
  if (!prefill_abc || !step_pq) return NAN;
  const double m = n_hat_w > 1 ? static_cast<double>(n_hat_w - 1) : 0.0;
  // sum_{i=1}^{M} p((1 - alpha) N_x + i - 1) + q
  const double dec = step_pq[0] * (m * (1.0 - alpha) * n_x + m * (m - 1.0) / 2.0) + m * step_pq[1];
  return prefill(prefill_abc, n_x) + dec;
}

double tb_alpha_star(const double* prefill_abc, const double* step_pq, double n_x,
                     int32_t n_hat_w, double budget, double t_predict, double alpha_max,
                     int32_t* feasible) {
  if (feasible) *feasible = 0;
  if (!prefill_abc || !step_pq || !(n_x > 0) || !(alpha_max >= 0 && alpha_max < 1)) return NAN;
  const double p = step_pq[0], q = step_pq[1];
  // A step time that falls as the cache grows is not a model of decoding
  // (Eq. decoding_step_time_raw is linear in N_kv with a non-negative slope).
  if (!(p >= 0) || !std::isfinite(p) || !std::isfinite(q) || std::isnan(budget) ||
      !std::isfinite(t_predict))
    return NAN;
  const double fixed = t_predict + prefill(prefill_abc, n_x);
  if (n_hat_w <= 1) {
    if (feasible) *feasible = fixed <= budget ? 1 : 0;
    return 0.0;
  }
  const double m = static_cast<double>(n_hat_w - 1);
  if (p == 0) {
    // WCET does not depend on alpha: the constraint of Eq. problem_converted
    // holds for every alpha or for none.  The closed form's limit p -> 0+ gives
    // 0 in the first case and alpha_max (clamped) in the second.
    const bool ok = fixed + m * q <= budget;
    if (feasible) *feasible = ok ? 1 : 0;
    return ok ? 0.0 : alpha_max;
  }
  const double raw = 1.0 - (budget - fixed) / (p * n_x * m) + (n_hat_w - 2) / (2.0 * n_x) +
                     q / (p * n_x);
  if (feasible) *feasible = raw <= alpha_max ? 1 : 0;
  return std::min(alpha_max, std::max(0.0, raw));
}

int32_t tb_response_length(int32_t n_hat, int32_t bucket, int32_t k, int32_t n_max,
                           int32_t* n_hat_len) {
  if (n_hat < 0 || bucket < 1 || k < 1 || n_max < 0) return -1;
  // N_hat = min(N_max, n_hat B) (Eq. predictor_inference); N_hat_W = min(k N_hat, N_max)
  const int64_t nh = std::min<int64_t>(n_max, static_cast<int64_t>(n_hat) * bucket);
  if (n_hat_len) *n_hat_len = static_cast<int32_t>(nh);
  return static_cast<int32_t>(std::min<int64_t>(static_cast<int64_t>(k) * nh, n_max));
}

int64_t tb_predictor_length(const double* prefill_abc, const double* predict_abc, double n_x,
                            int64_t max_len) {
  if (!prefill_abc || !predict_abc || max_len < 0 || !(n_x >= 0)) return -2;
  const double ap = predict_abc[0], bp = predict_abc[1], cp = predict_abc[2];
  if (!(ap >= 0) || !(bp >= 0)) return -2;           // the model must grow with length
  const double T = prefill(prefill_abc, n_x);
  auto f = [&](double x) { return (ap * x + bp) * x + cp; };
  if (!(cp <= T)) return -1;                         // not even an empty input fits
  if (f(static_cast<double>(max_len)) <= T) return max_len;
  // f is increasing on [0, inf): the answer is the floor of the positive root
  double r;
  if (ap > 0) {
    const double disc = bp * bp + 4.0 * ap * (T - cp);
    r = (2.0 * (T - cp)) / (bp + sqrt(disc));         // the same root, without cancellation
  } else {
    r = (T - cp) / bp;                               // bp > 0 here since f(max_len) > T >= cp
  }
  int64_t n = static_cast<int64_t>(std::min<double>(std::max(0.0, floor(r)), static_cast<double>(max_len)));
  while (n + 1 <= max_len && f(static_cast<double>(n + 1)) <= T) ++n;   // settle rounding
  while (n > 0 && f(static_cast<double>(n)) > T) --n;
  return n;
}

}  // extern "C"
