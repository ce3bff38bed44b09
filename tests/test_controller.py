"""Time-budget controller: the float64 reference pinned against the paper's
constraint (bisection), a hand-derived example and library least squares; the
C ABI host functions checked against the reference.  No GPU."""
import json
import math
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import controller as C
from paper_2512_21859_amd import _lib

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "controller_example.json")


def _ex():
    with open(GOLDEN) as f:
        return json.load(f)


def _bisect_alpha(abc, pq, n_x, n_hat_w, budget, t_pred, alpha_max):
    """Smallest alpha in [0, alpha_max] meeting t_pred + WCET <= budget, found by
    bisection on the explicit-loop WCET (independent of the closed form)."""
    f = lambda a: t_pred + C.t_wcet(abc, pq, n_x, a, n_hat_w) - budget
    if f(0.0) <= 0:
        return 0.0, True
    if f(alpha_max) > 0:
        return alpha_max, False
    lo, hi = 0.0, alpha_max
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        lo, hi = (lo, mid) if f(mid) <= 0 else (mid, hi)
    return hi, True


def test_hand_example():
    e = _ex()
    a, feas = C.alpha_star(e["prefill_abc"], e["step_pq"], e["n_x"], e["n_hat_w"], e["budget"],
                           e["t_predict"], e["alpha_max"])
    assert feas and abs(a - e["alpha_star"]) < 1e-12
    assert abs(C.t_wcet(e["prefill_abc"], e["step_pq"], e["n_x"], 0.0, e["n_hat_w"]) -
               e["wcet_at_alpha_0"]) < 1e-9
    assert abs(C.t_wcet(e["prefill_abc"], e["step_pq"], e["n_x"], e["alpha_star"], e["n_hat_w"]) -
               e["budget"]) < 1e-9
    L = e["lengths"]
    for c in L["cases"]:
        nh = C.predicted_length(c["n_hat"], L["bucket"], L["n_max"])
        assert nh == c["N_hat"]
        assert C.pessimistic_length(nh, L["k"], L["n_max"]) == c["N_hat_W"]


@settings(max_examples=200, deadline=None)
@given(st.floats(1e-9, 1e-6), st.floats(1e-6, 1e-3), st.floats(0.0, 1.0),
       st.one_of(st.just(0.0), st.floats(1e-6, 1e-3)), st.floats(1e-4, 0.1),
       st.integers(100, 32768),
       st.integers(1, 600), st.floats(0.5, 60.0), st.floats(0.0, 0.5), st.floats(0.5, 0.99))
def test_closed_form_equals_bisection(a, b, c, p, q, n_x, n_hat_w, budget, t_pred, amax):
    abc, pq = (a, b, c), (p, q)
    got, feas = C.alpha_star(abc, pq, n_x, n_hat_w, budget, t_pred, amax)
    ref, rfeas = _bisect_alpha(abc, pq, n_x, n_hat_w, budget, t_pred, amax)
    if n_hat_w <= 1:
        assert got == 0.0
        return
    assert feas == rfeas
    assert abs(got - ref) < 1e-9


def test_zero_slope_hand_case():
    """p = 0: the WCET does not depend on alpha (Eq. problem_converted).  With
    prefill c = 2 s, q = 1/128 s, N_hat_W = 129 (128 decode steps) and
    t_predict = 0.5 s the worst case is 0.5 + 2 + 128 / 128 = 3.5 s at every
    alpha (all exact in binary): a budget of 3.5 s is met with no eviction,
    3.49 s by none."""
    abc, pq = (0.0, 0.0, 2.0), (0.0, 1.0 / 128)
    for impl in (C.alpha_star, _lib.tb_alpha_star):
        assert impl(abc, pq, 1000.0, 129, 3.5, 0.5, 0.95) == (0.0, True)
        assert impl(abc, pq, 1000.0, 129, 3.49, 0.5, 0.95) == (0.95, False)
        assert impl(abc, pq, 1000.0, 129, float("inf"), 0.5, 0.95) == (0.0, True)
    for T in (3.5, 3.49):                       # the constraint by bisection agrees
        assert _bisect_alpha(abc, pq, 1000.0, 129, T, 0.5, 0.95) == C.alpha_star(
            abc, pq, 1000.0, 129, T, 0.5, 0.95)
    assert C.t_wcet(abc, pq, 1000.0, 0.0, 129) == 3.0
    assert C.t_wcet(abc, pq, 1000.0, 0.9, 129) == 3.0


def test_negative_slope_is_rejected():
    """A step time that falls as the cache grows is not a decode-step model:
    both implementations return (nan, infeasible), whatever the budget (the
    closed form would return alpha_max for a budget met at alpha = 0, and 0
    for one that no alpha meets)."""
    abc, pq = (0.0, 0.0, 2.0), (-1e-6, 0.01)
    for impl in (C.alpha_star, _lib.tb_alpha_star):
        for T in (12.0, 2.5):
            a, feas = impl(abc, pq, 1000.0, 100, T, 0.0, 0.95)
            assert math.isnan(a) and not feas


def test_response_length_matches_reference():
    e = _ex()
    L = e["lengths"]
    for c in L["cases"]:
        assert _lib.tb_response_length(c["n_hat"], L["bucket"], L["k"], L["n_max"]) == (
            c["N_hat"], c["N_hat_W"])
    rng = np.random.default_rng(11)
    for _ in range(500):
        nh, b, k, nmax = (int(rng.integers(0, 600)), int(rng.integers(1, 64)),
                          int(rng.integers(1, 9)), int(rng.integers(0, 40000)))
        want = C.predicted_length(nh, b, nmax)
        assert _lib.tb_response_length(nh, b, k, nmax) == (want, C.pessimistic_length(want, k, nmax))
    for bad in ((-1, 16, 5, 8192), (3, 0, 5, 8192), (3, 16, 0, 8192), (3, 16, 5, -1)):
        with pytest.raises(ValueError):
            _lib.tb_response_length(*bad)


def test_printed_second_term_disagrees():
    """The printed closed form divides (N_hat_W - 2)/2 by p N_x; it does not
    solve the constraint, the derived (N_hat_W - 2)/(2 N_x) does."""
    e = _ex()
    (a, b, c), (p, q) = e["prefill_abc"], e["step_pq"]
    n_x, nw, T = e["n_x"], e["n_hat_w"], e["budget"]
    pre = a * n_x ** 2 + b * n_x + c
    printed = 1 - (T - pre) / (p * n_x * (nw - 1)) + (nw - 2) / (2 * p * n_x) + q / (p * n_x)
    derived = 1 - (T - pre) / (p * n_x * (nw - 1)) + (nw - 2) / (2 * n_x) + q / (p * n_x)
    assert abs(derived - e["alpha_star"]) < 1e-12
    assert abs(printed - e["alpha_star"]) > 1.0


def test_prefill_and_step_time_hand_values():
    """The time model's terms at hand-computed points (the worked example
    above has a = b = 0, so the prefill's N^2 and N terms are pinned here):
    1e-8 * 10000^2 + 1e-4 * 10000 + 0.5 = 1 + 1 + 0.5 = 2.5 s;
    2e-9 * 30000^2 = 1.8 s; 1e-4 * 5000 + 0.01 = 0.51 s; the retained length at
    step i is (1 - alpha) N_x + i - 1: 7500 at i = 1 and 7502 at i = 3 for
    alpha = 0.25, N_x = 10000."""
    assert abs(C.t_prefill((1e-8, 1e-4, 0.5), 10000) - 2.5) < 1e-12
    assert abs(C.t_prefill((2e-9, 0.0, 0.0), 30000) - 1.8) < 1e-12
    assert abs(C.t_step((1e-4, 0.01), 5000) - 0.51) < 1e-12
    assert C.kv_length(10000, 0.25, 1) == 7500.0
    assert C.kv_length(10000, 0.25, 3) == 7502.0


def test_decoding_phase_explicit_sum():
    pq = (2e-5, 3e-3)
    for n_x, alpha, nh in [(1000, 0.0, 1), (1000, 0.3, 2), (4096, 0.5, 65), (32768, 0.95, 257)]:
        want = sum(pq[0] * ((1 - alpha) * n_x + i - 1) + pq[1] for i in range(1, nh))
        assert abs(C.t_decoding_phase(pq, n_x, alpha, nh) - want) < 1e-12


def test_fit_poly_recovers_exact_and_matches_polyfit():
    n = np.linspace(0, 32768, 41)
    t = 3e-9 * n ** 2 + 2e-5 * n + 0.04
    assert np.allclose(C.fit_poly(n, t, 2), [3e-9, 2e-5, 0.04], rtol=1e-8, atol=1e-12)
    rng = np.random.default_rng(5)
    tn = 7e-6 * n + 0.02 + rng.normal(0, 1e-4, n.size)
    assert np.allclose(C.fit_poly(n, tn, 1), np.polyfit(n, tn, 1), rtol=1e-9)


# ---------------------------------------------------------------- C ABI vs reference
@pytest.mark.parametrize("degree", [1, 2])
def test_abi_fit_matches_reference(degree):
    rng = np.random.default_rng(degree)
    for _ in range(20):
        n = np.sort(rng.uniform(0, 32768, rng.integers(degree + 1, 60)))
        t = rng.uniform(0, 1e-9) * n ** 2 * (degree == 2) + rng.uniform(0, 1e-4) * n + \
            rng.uniform(0, 0.1) + rng.normal(0, 1e-5, n.size)
        got = _lib.tb_ete_fit(n.tolist(), t.tolist(), degree)
        ref = C.fit_poly(n, t, degree)
        V = np.vander(n, degree + 1)                                # compare the fitted curves
        assert np.abs(V @ np.array(got) - V @ ref).max() <= 1e-9 * np.abs(t).max()
    with pytest.raises(ValueError):
        _lib.tb_ete_fit([1.0], [2.0], 1)
    with pytest.raises(ValueError):
        _lib.tb_ete_fit([3.0, 3.0, 3.0], [1.0, 2.0, 3.0], 1)


@settings(max_examples=200, deadline=None)
@given(st.floats(0.0, 1e-6), st.floats(0.0, 1e-3), st.floats(0.0, 1.0),
       st.one_of(st.just(0.0), st.floats(1e-6, 1e-3)), st.floats(1e-4, 0.1),
       st.integers(100, 32768),
       st.integers(0, 600), st.floats(0.1, 60.0), st.floats(0.0, 0.5), st.floats(0.5, 0.99),
       st.floats(0.0, 0.99))
def test_abi_wcet_and_alpha_match_reference(a, b, c, p, q, n_x, n_hat_w, budget, t_pred, amax,
                                            alpha):
    abc, pq = (a, b, c), (p, q)
    w_ref = C.t_wcet(abc, pq, n_x, alpha, n_hat_w)
    assert math.isclose(_lib.tb_wcet(abc, pq, n_x, alpha, n_hat_w), w_ref, rel_tol=1e-10,
                        abs_tol=1e-12)
    got, feas = _lib.tb_alpha_star(abc, pq, n_x, n_hat_w, budget, t_pred, amax)
    ref, rfeas = C.alpha_star(abc, pq, n_x, n_hat_w, budget, t_pred, amax)
    assert feas == rfeas
    assert math.isclose(got, ref, rel_tol=1e-12, abs_tol=1e-12)


def test_abi_alpha_edges():
    e = _ex()
    got, feas = _lib.tb_alpha_star(e["prefill_abc"], e["step_pq"], e["n_x"], e["n_hat_w"],
                                   e["budget"], e["t_predict"], e["alpha_max"])
    assert feas and abs(got - e["alpha_star"]) < 1e-12
    assert _lib.tb_alpha_star(e["prefill_abc"], e["step_pq"], e["n_x"], 101, 1e6, 0.0, 0.95) == (0.0, True)
    assert _lib.tb_alpha_star(e["prefill_abc"], e["step_pq"], e["n_x"], 101, 5.0, 0.0, 0.95) == (0.95, False)
    assert _lib.tb_alpha_star(e["prefill_abc"], e["step_pq"], e["n_x"], 1, 5.0, 0.0, 0.95) == (0.0, True)
    assert math.isnan(_lib.tb_alpha_star(e["prefill_abc"], e["step_pq"], 0.0, 101, 5.0, 0.0, 0.95)[0])


def test_choose_alpha_matches_reference():
    from paper_2512_21859_amd.pipeline import choose_alpha
    e = _ex()
    L = e["lengths"]
    for c in L["cases"]:
        for budget in (0.5, 2.0, 5.0, 50.0):
            got = choose_alpha(e["prefill_abc"], e["step_pq"], e["n_x"], c["n_hat"], L["bucket"],
                               L["k"], L["n_max"], budget, 0.1, 0.95)
            nw = C.pessimistic_length(C.predicted_length(c["n_hat"], L["bucket"], L["n_max"]),
                                      L["k"], L["n_max"])
            ref = C.alpha_star(e["prefill_abc"], e["step_pq"], e["n_x"], nw, budget, 0.1, 0.95)
            assert got[2] == nw == c["N_hat_W"]
            assert got[1] == ref[1] and abs(got[0] - ref[0]) < 1e-12


def test_predictor_length_golden_and_abi():
    """Hand-derived cases (tests/golden/controller_example.json) for the oracle's
    integer search and for tb_predictor_length."""
    ex = _ex()["predictor_length"]
    for cs in ex["cases"]:
        got_o = C.predictor_length(ex["prefill_abc"], cs["predict_abc"], ex["n_x"], cs["max_len"])
        got_c = _lib.tb_predictor_length(ex["prefill_abc"], cs["predict_abc"], ex["n_x"],
                                         cs["max_len"])
        assert got_o == cs["n_p"], cs
        assert got_c == cs["n_p"], cs


def test_predictor_length_random_against_search():
    rng = np.random.default_rng(17)
    for _ in range(300):
        pre = [rng.uniform(0, 2e-6), rng.uniform(0, 1e-3), rng.uniform(0, 0.05)]
        pred = [rng.choice([0.0, rng.uniform(0, 4e-6)]), rng.uniform(0, 2e-3),
                rng.uniform(0, 0.2)]
        n_x = float(rng.integers(1, 3000))
        max_len = int(rng.integers(0, 3000))
        assert (_lib.tb_predictor_length(pre, pred, n_x, max_len)
                == C.predictor_length(pre, pred, n_x, max_len))
    with pytest.raises(ValueError):
        _lib.tb_predictor_length([1, 0, 0], [0, -1.0, 0], 10.0, 10)
