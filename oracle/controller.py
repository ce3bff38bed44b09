"""Float64 reference of TimeBill's time-budget controller.

TEST INFRASTRUCTURE ONLY (same rules as timebill_oracle: only tests, the smoke
check and the benchmark's CPU-baseline leg may use it).

What it computes (TimeBill, arXiv 2512.21859):

* Predicted response length N_hat = min(N_max, n_hat * B) from the predicted
  bucket index (Sec. 4.1, Eq. predictor_inference) and the pessimistic length
  N_hat_W = min(k * N_hat, N_max) (Sec. 4.2, before Eq. wcet).
* Execution-time model: prefill a N_x^2 + b N_x + c and decode step
  p N_kv + q (Sec. 4.2, Eq. exeuction_time_part), with coefficients fitted by
  least squares on profiled (N, t) pairs (Sec. 4.2, profiling-based fitting).
* Retained length at decode step i: (1 - alpha) N_x + i - 1 (Eq. N_kv); the
  decode phase sums the steps i = 1 .. N_hat - 1 (Eqs. decoding-step,
  decoding-phase); WCET = prefill + decode phase at N_hat_W (Eq. wcet).
* The predictor runs beside the prefill (Sec. 5.2): its input is compressed
  to the longest N_p whose own time a_p N_p^2 + b_p N_p + c_p stays within the
  prefill time a N_x^2 + b N_x + c.
* alpha* = the smallest alpha in [0, alpha_max] with
  t_predict + WCET(alpha) <= T (Sec. 5.1, Eq. problem_converted), in closed
  form (Eq. alpha_with_predictor).

Reading: substituting the equations gives a second term (N_hat_W - 2)/(2 N_x);
the printed formula divides it by p as well, which is dimensionally
inconsistent (1/time) and disagrees with solving the constraint, so the
derived form is used.  The paper gives no lower clamp; alpha* is clamped to
[0, alpha_max], and N_hat_W <= 1 (no decode step) gives alpha* = 0.  The
closed form needs a positive slope p; p = 0 and p < 0 are handled in
alpha_star (the constraint itself, Eq. problem_converted, is well defined at
p = 0).
"""
from __future__ import annotations

import numpy as np


def predicted_length(n_hat: int, bucket: int, n_max: int) -> int:
    """N_hat = min(N_max, n_hat * B) (Eq. predictor_inference)."""
    return min(n_max, n_hat * bucket)


def pessimistic_length(n_hat: int, k: int, n_max: int) -> int:
    """N_hat_W = min(k * N_hat, N_max)."""
    return min(k * n_hat, n_max)


def kv_length(n_x: float, alpha: float, i: int) -> float:
    """Retained KV length at decode step i (Eq. N_kv)."""
    return (1.0 - alpha) * n_x + i - 1


def t_prefill(abc, n_x: float) -> float:
    a, b, c = abc
    return a * n_x * n_x + b * n_x + c


def t_step(pq, n_kv: float) -> float:
    p, q = pq
    return p * n_kv + q


def t_decoding_phase(pq, n_x: float, alpha: float, n_hat: int) -> float:
    """Sum of the decode-step times for i = 1 .. n_hat - 1 (Eq. decoding-phase)."""
    return float(sum(t_step(pq, kv_length(n_x, alpha, i)) for i in range(1, n_hat)))


def t_wcet(abc, pq, n_x: float, alpha: float, n_hat_w: int) -> float:
    """Eq. wcet: prefill plus the decode phase at the pessimistic length."""
    return t_prefill(abc, n_x) + t_decoding_phase(pq, n_x, alpha, n_hat_w)


def alpha_star(abc, pq, n_x: float, n_hat_w: int, budget: float, t_predict: float,
               alpha_max: float):
    """Smallest feasible eviction ratio; returns (alpha, feasible).

    With M = n_hat_w - 1 decode steps the constraint is
    t_predict + t_prefill + M p (1 - alpha) N_x + p M (M - 1) / 2 + M q <= T.

    The closed form divides by p.  With p = 0 the left side does not depend on
    alpha: every alpha meets the constraint or none does, and the result is the
    closed form's limit as p -> 0 from above (0 when feasible, alpha_max
    otherwise).  A negative slope is not a decode-step model: (nan, False).
    """
    p, q = pq
    if not p >= 0:
        return float("nan"), False
    fixed = t_predict + t_prefill(abc, n_x)
    if n_hat_w <= 1:
        return 0.0, fixed <= budget
    m = n_hat_w - 1
    if p == 0:
        ok = fixed + m * q <= budget
        return (0.0 if ok else float(alpha_max)), bool(ok)
    raw = (1.0 - (budget - t_prefill(abc, n_x) - t_predict) / (p * n_x * m)
           + (n_hat_w - 2) / (2.0 * n_x) + q / (p * n_x))
    feasible = raw <= alpha_max
    return float(min(alpha_max, max(0.0, raw))), bool(feasible)


def fit_poly(n, t, degree: int):
    """Least-squares polynomial coefficients, highest power first."""
    n = np.asarray(n, dtype=np.float64)
    t = np.asarray(t, dtype=np.float64)
    V = np.vander(n, degree + 1)
    coef, *_ = np.linalg.lstsq(V, t, rcond=None)
    return coef


def predictor_length(prefill_abc, predict_abc, n_x: float, max_len: int) -> int:
    """Largest integer N_p in [0, max_len] with t_predict(N_p) <= t_prefill(N_x),
    by direct search over the integers; -1 when none fits."""
    budget = t_prefill(prefill_abc, n_x)
    a, b, c = predict_abc
    best = -1
    for n in range(max_len + 1):
        if a * n * n + b * n + c <= budget:
            best = n
    return best
