"""Planted mistakes in the oracle must fail its pins.

Each mutant is the oracle with one plausible error: an index off by one, a
dropped scale or term, a wrong sign or axis, swapped operands, a wrong tie or
order rule, a wrong rounding.  The test swaps it into the oracle module (on
the CPU, for this test only) and runs the fixed-case pins that cover that
function; at least one of them must fail.  This is evidence that the pins,
not the oracle checking itself, fix what the oracle computes.
"""
import math

import numpy as np
import pytest

from oracle import controller as C
from oracle import scorers as S
from oracle import timebill_oracle as O
from tests import test_controller as PC
from tests import test_oracle_pins as P
from tests import test_oracle_pins_scorers as PS

_orig = {name: getattr(O, name) for name in (
    "window_logits", "window_probs", "window_scores", "max_pool", "select_keep",
    "decode_step", "merge_partials", "keep_count", "prefill_attention",
    "prefill_window_stats", "window_column_mass")}
_orig_s = {name: getattr(S, name) for name in ("knorm_scores", "avg_pool", "h2o_scores")}
_orig_c = {name: getattr(C, name) for name in (
    "kv_length", "t_prefill", "t_decoding_phase", "t_wcet", "alpha_star", "predicted_length",
    "pessimistic_length", "fit_poly", "predictor_length")}


# ---------------------------------------------------------------- mutants
def _logits(q_win, k, n_x, g, shift=0, scale=True, group=True):
    hq, w, d = q_win.shape
    G = hq // k.shape[0]
    heads = q_win[g * G:(g + 1) * G] if group else q_win[:G]
    q = np.asarray(heads, dtype=np.float64).reshape(G * w, d)
    s = q @ np.asarray(k[g, :n_x], dtype=np.float64).T
    if scale:
        s = s / math.sqrt(d)
    pos = n_x - w + np.tile(np.arange(w), G)
    s[np.arange(n_x)[None, :] > pos[:, None] + shift] = -np.inf
    return s


def logits_mask_late(q_win, k, n_x, g):
    return _logits(q_win, k, n_x, g, shift=1)


def logits_mask_early(q_win, k, n_x, g):
    return _logits(q_win, k, n_x, g, shift=-1)


def logits_no_scale(q_win, k, n_x, g):
    return _logits(q_win, k, n_x, g, scale=False)


def logits_group0(q_win, k, n_x, g):
    return _logits(q_win, k, n_x, g, group=False)


def probs_column_softmax(q_win, k, n_x, g):
    s = O.window_logits(q_win, k, n_x, g)
    s = np.where(np.isinf(s), -1e300, s)
    e = np.exp(s - s.max(axis=0, keepdims=True))
    return e / e.sum(axis=0, keepdims=True)


def scores_shifted(q_win, k, n_x, w):
    out = np.empty((k.shape[0], n_x - w))
    for g in range(k.shape[0]):
        out[g] = O.window_column_mass(q_win, k, n_x, g)[1:n_x - w + 1]
    return out


def pool_wide(a, pool):
    return _orig["max_pool"](a, pool + 2)


def pool_left_only(a, pool):
    r = pool // 2
    a = np.asarray(a, dtype=np.float64)
    padded = np.pad(a, [(0, 0)] * (a.ndim - 1) + [(2 * r, 0)], constant_values=-np.inf)
    return np.lib.stride_tricks.sliding_window_view(padded, pool, axis=-1).max(axis=-1)


def keep_high_ties(pooled, n_x, w, n_keep):
    pref = n_x - w
    idx = np.arange(pref)
    chosen = np.sort(np.lexsort((-idx, -pooled))[:n_keep - w])
    return np.concatenate([chosen, np.arange(pref, n_x)]).astype(np.int64)


def keep_window_first(pooled, n_x, w, n_keep):
    k = _orig["select_keep"](pooled, n_x, w, n_keep)
    return np.concatenate([k[n_keep - w:], k[:n_keep - w]])


def keep_smallest(pooled, n_x, w, n_keep):
    return _orig["select_keep"](-np.asarray(pooled), n_x, w, n_keep)


def decode_swapped(q, k_cache, v_cache):
    return _orig["decode_step"](q, v_cache, k_cache)


def decode_no_scale(q, k_cache, v_cache):
    return _orig["decode_step"](np.asarray(q) * math.sqrt(np.asarray(q).shape[-1]), k_cache,
                                v_cache)


def decode_drop_last(q, k_cache, v_cache):
    n = len(k_cache)
    return _orig["decode_step"](q, k_cache[:max(n - 1, 1)], v_cache[:max(n - 1, 1)])


def decode_negated(q, k_cache, v_cache):
    return _orig["decode_step"](-np.asarray(q), k_cache, v_cache)


def merge_no_rescale(parts):
    L = sum(p[1] for p in parts)
    return sum(p[2] for p in parts) / L[:, None]


def keep_count_ceil(n_x, alpha, w):
    if not (0 < w < n_x) or not (0.0 <= alpha < 1.0):
        raise ValueError("bad arguments")
    return max(w, n_x - math.ceil(alpha * n_x))


def keep_count_no_window_floor(n_x, alpha, w):
    if not (0 < w < n_x) or not (0.0 <= alpha < 1.0):
        raise ValueError("bad arguments")
    return n_x - math.floor(alpha * n_x)


def prefill_sees_next(q, k, v, n_x, rows=None):
    hq, hkv = q.shape[0], k.shape[0]
    G = hq // hkv
    rows = np.arange(n_x) if rows is None else np.asarray(rows)
    out = np.empty((hq, len(rows), q.shape[-1]))
    for h in range(hq):
        for r, i in enumerate(rows):
            j = min(i + 2, n_x)
            out[h, r] = O.decode_step(q[h:h + 1, i], k[h // G, :j], v[h // G, :j])[0]
    return out


def prefill_wrong_group(q, k, v, n_x, rows=None):
    hq, hkv = q.shape[0], k.shape[0]
    rows = np.arange(n_x) if rows is None else np.asarray(rows)
    out = np.empty((hq, len(rows), q.shape[-1]))
    for h in range(hq):
        for r, i in enumerate(rows):
            out[h, r] = O.decode_step(q[h:h + 1, i], k[h % hkv, :i + 1], v[h % hkv, :i + 1])[0]
    return out


def stats_no_scale(q, k, n_x, w):
    return _orig["prefill_window_stats"](np.asarray(q) * math.sqrt(q.shape[-1]), k, n_x, w)


def _fixed(test, cases):
    """A parametrized pin bound to its fixed cases, as one callable."""
    def run():
        for c in cases:
            test(*c)
    run.__name__ = test.__name__
    return run


_WINDOW_FIXED = _fixed(P.test_window_probs_match_torch_sdpa_fixed,
                       [(2, 3, 9, 8, 1), (4, 5, 20, 2, 7), (1, 1, 3, 8, 2)])
_MERGE_FIXED = _fixed(P.test_split_merge_equals_direct_fixed, [(50, 7, 3), (9, 3, 11), (80, 1, 5)])
# ---- scorer variants
def knorm_positive(k, n_x, w):
    return -_orig_s["knorm_scores"](k, n_x, w)


def knorm_squared(k, n_x, w):
    return -_orig_s["knorm_scores"](k, n_x, w) ** 2


def knorm_shifted(k, n_x, w):
    return _orig_s["knorm_scores"](np.asarray(k)[:, 1:], n_x - 1, w - 1)[:, :n_x - w]


def avg_pool_valid_divisor(a, pool):
    a = np.asarray(a, dtype=np.float64)
    ones = np.ones_like(a)
    return _orig_s["avg_pool"](a, pool) / _orig_s["avg_pool"](ones, pool)


def avg_pool_wrapping(a, pool):
    a = np.asarray(a, dtype=np.float64)
    h = pool // 2
    return sum(np.roll(a, s, axis=-1) for s in range(-h, h + 1)) / pool


def _h2o(q, k, n_x, diag=0, scale=True):
    hq, hkv = q.shape[0], k.shape[0]
    G, d = hq // hkv, q.shape[-1]
    out = np.zeros((hkv, n_x))
    allowed = np.tril(np.ones((n_x, n_x), dtype=bool), k=diag)
    for h in range(hq):
        s = np.asarray(q[h, :n_x], dtype=np.float64) @ np.asarray(k[h // G, :n_x], dtype=np.float64).T
        s = s / np.sqrt(d) if scale else s
        s = np.where(allowed, s, -np.inf)
        p = np.exp(s - s.max(axis=1, keepdims=True))
        out[h // G] += (p / p.sum(axis=1, keepdims=True)).sum(axis=0)
    return out


def h2o_sees_next(q, k, n_x):
    return _h2o(q, k, n_x, diag=1)


def h2o_no_scale(q, k, n_x):
    return _h2o(q, k, n_x, scale=False)


# ---- time-budget controller
def kv_length_no_minus_one(n_x, alpha, i):
    return (1.0 - alpha) * n_x + i


def decoding_phase_one_more(pq, n_x, alpha, n_hat):
    return _orig_c["t_decoding_phase"](pq, n_x, alpha, n_hat + 1)


def wcet_without_prefill(abc, pq, n_x, alpha, n_hat_w):
    return C.t_decoding_phase(pq, n_x, alpha, n_hat_w)


def prefill_linear_only(abc, n_x):
    return abc[1] * n_x + abc[2]


def alpha_star_printed(abc, pq, n_x, n_hat_w, budget, t_predict, alpha_max):
    if n_hat_w <= 1:
        return 0.0, t_predict + C.t_prefill(abc, n_x) <= budget
    p, q = pq
    m = n_hat_w - 1
    raw = (1.0 - (budget - C.t_prefill(abc, n_x) - t_predict) / (p * n_x * m)
           + (n_hat_w - 2) / (2.0 * p * n_x) + q / (p * n_x))
    return float(min(alpha_max, max(0.0, raw))), bool(raw <= alpha_max)


def predicted_no_cap(n_hat, bucket, n_max):
    return n_hat * bucket


def pessimistic_no_cap(n_hat, k, n_max):
    return k * n_hat


def fit_poly_reversed(n, t, degree):
    return _orig_c["fit_poly"](n, t, degree)[::-1]


def predictor_length_one_short(prefill_abc, predict_abc, n_x, max_len):
    return _orig_c["predictor_length"](prefill_abc, predict_abc, n_x, max(max_len - 1, 0))


_WINDOW_PINS = [P.test_hand_example_column_mass_and_mask, P.test_hand_example_scores_and_pool,
                _WINDOW_FIXED, P.test_rows_are_distributions_and_mass_is_Gw,
                P.test_window_probs_match_torch_sdpa, P.test_alpha_zero_is_identity_and_full_attention]
_POOL_PINS = [P.test_hand_example_scores_and_pool, P.test_max_pool_matches_torch]
_SELECT_PINS = [P.test_hand_example_keep, P.test_select_matches_brute_force]
_DECODE_PINS = [P.test_hand_example_decode, P.test_decode_matches_torch_sdpa,
                P.test_decode_special_cases, P.test_decode_append_order,
                P.test_alpha_zero_is_identity_and_full_attention]
_KEEP_PINS = [P.test_keep_count_table, P.test_keep_count_edges]
_KNORM_PINS = [PS.test_knorm_hand_example, PS.test_knorm_matches_torch_norm]
_AVG_PINS = [PS.test_avg_pool_hand_example, _fixed(PS.test_avg_pool_matches_torch,
                                                   [(1,), (3,), (5,), (7,), (9,)]),
             PS.test_avg_pool_constant_closed_form]
_H2O_PINS = [PS.test_h2o_hand_example, PS.test_h2o_total_mass_and_torch,
             PS.test_h2o_last_row_only_matches_window_mass]
_CTRL_PINS = [PC.test_hand_example, PC.test_prefill_and_step_time_hand_values,
              PC.test_decoding_phase_explicit_sum, PC.test_predictor_length_golden_and_abi,
              PC.test_closed_form_equals_bisection]

MUTANTS = {
    "causal mask one key late": ("window_logits", logits_mask_late, _WINDOW_PINS),
    "causal mask one key early": ("window_logits", logits_mask_early, _WINDOW_PINS),
    "1/sqrt(d) dropped from the window logits": ("window_logits", logits_no_scale, _WINDOW_PINS),
    "every group reads group 0's queries": ("window_logits", logits_group0, _WINDOW_PINS),
    "softmax over keys instead of rows": ("window_probs", probs_column_softmax, _WINDOW_PINS),
    "scores shifted by one position": ("window_scores", scores_shifted, _WINDOW_PINS),
    "pool two wider": ("max_pool", pool_wide, _POOL_PINS),
    "pool looks left only": ("max_pool", pool_left_only, _POOL_PINS),
    "ties kept at the higher position": ("select_keep", keep_high_ties, _SELECT_PINS),
    "window emitted first": ("select_keep", keep_window_first, _SELECT_PINS),
    "smallest scores kept": ("select_keep", keep_smallest, _SELECT_PINS),
    "K and V swapped in decode": ("decode_step", decode_swapped, _DECODE_PINS),
    "1/sqrt(d) dropped from decode": ("decode_step", decode_no_scale, _DECODE_PINS),
    "last cached row dropped": ("decode_step", decode_drop_last, _DECODE_PINS),
    "query sign flipped": ("decode_step", decode_negated, _DECODE_PINS),
    "partials merged without the max rescale": ("merge_partials", merge_no_rescale,
                                                [_MERGE_FIXED, P.test_split_merge_equals_direct]),
    "ratio rounded up": ("keep_count", keep_count_ceil, _KEEP_PINS),
    "window floor dropped": ("keep_count", keep_count_no_window_floor, _KEEP_PINS),
    "prefill row sees the next key": ("prefill_attention", prefill_sees_next,
                                      [P.test_prefill_attention_matches_torch_sdpa]),
    "prefill query head in the wrong group": ("prefill_attention", prefill_wrong_group,
                                              [P.test_prefill_attention_matches_torch_sdpa]),
    "window statistics without 1/sqrt(d)": ("prefill_window_stats", stats_no_scale,
                                            [P.test_prefill_attention_matches_torch_sdpa]),
}
MUTANTS = {k: (O,) + v for k, v in MUTANTS.items()}
MUTANTS.update({
    "KNorm keeps the largest norms": (S, "knorm_scores", knorm_positive, _KNORM_PINS),
    "KNorm without the square root": (S, "knorm_scores", knorm_squared, _KNORM_PINS),
    "KNorm one key off": (S, "knorm_scores", knorm_shifted, _KNORM_PINS),
    "mean pool divides by the in-range count": (S, "avg_pool", avg_pool_valid_divisor, _AVG_PINS),
    "mean pool wraps around": (S, "avg_pool", avg_pool_wrapping, _AVG_PINS),
    "H2O query sees the next key": (S, "h2o_scores", h2o_sees_next, _H2O_PINS),
    "H2O without 1/sqrt(d)": (S, "h2o_scores", h2o_no_scale, _H2O_PINS),
    "retained length without the -1": (C, "kv_length", kv_length_no_minus_one, _CTRL_PINS),
    "one decode step too many": (C, "t_decoding_phase", decoding_phase_one_more, _CTRL_PINS),
    "WCET without the prefill": (C, "t_wcet", wcet_without_prefill, _CTRL_PINS),
    "prefill time without the N^2 term": (C, "t_prefill", prefill_linear_only, _CTRL_PINS),
    "alpha* with the printed second term": (C, "alpha_star", alpha_star_printed, _CTRL_PINS),
    "predicted length not capped": (C, "predicted_length", predicted_no_cap, _CTRL_PINS),
    "pessimistic length not capped": (C, "pessimistic_length", pessimistic_no_cap, _CTRL_PINS),
    "fit coefficients in the wrong order": (C, "fit_poly", fit_poly_reversed,
                                            [PC.test_fit_poly_recovers_exact_and_matches_polyfit]),
    "predictor length search one short": (C, "predictor_length", predictor_length_one_short,
                                          [PC.test_predictor_length_golden_and_abi]),
})


# pins driven by hypothesis draw their cases at random; each mutant must also
# fail at least one pin that runs fixed cases, so the result does not depend
# on the draw
_RANDOM = {P.test_rows_are_distributions_and_mass_is_Gw, P.test_window_probs_match_torch_sdpa,
           P.test_max_pool_matches_torch, P.test_select_matches_brute_force,
           P.test_decode_matches_torch_sdpa, P.test_split_merge_equals_direct,
           PC.test_closed_form_equals_bisection}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, monkeypatch):
    module, attr, mutant, pins = MUTANTS[name]
    monkeypatch.setattr(module, attr, mutant)
    caught = []
    for pin in [p for p in pins if p not in _RANDOM]:
        try:
            pin()
        except (Exception, pytest.fail.Exception):   # an assertion, a failed
            caught.append(pin.__name__)              # pytest.raises, or an error it causes
    assert caught, f"no fixed-case pin fails when the oracle has: {name}"


def test_pins_pass_on_the_oracle():
    """The same pins, run the same way, pass on the unmodified oracle."""
    pins = {p for _, _, _, ps in MUTANTS.values() for p in ps if p not in _RANDOM}
    for pin in sorted(pins, key=lambda p: p.__name__):
        pin()
