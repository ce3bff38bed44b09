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

from oracle import timebill_oracle as O
from tests import test_oracle_pins as P

_orig = {name: getattr(O, name) for name in (
    "window_logits", "window_probs", "window_scores", "max_pool", "select_keep",
    "decode_step", "merge_partials", "keep_count", "prefill_attention",
    "prefill_window_stats", "window_column_mass")}


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
_WINDOW_PINS = [P.test_hand_example_column_mass_and_mask, P.test_hand_example_scores_and_pool,
                _WINDOW_FIXED, P.test_rows_are_distributions_and_mass_is_Gw,
                P.test_window_probs_match_torch_sdpa, P.test_alpha_zero_is_identity_and_full_attention]
_POOL_PINS = [P.test_hand_example_scores_and_pool, P.test_max_pool_matches_torch]
_SELECT_PINS = [P.test_hand_example_keep, P.test_select_matches_brute_force]
_DECODE_PINS = [P.test_hand_example_decode, P.test_decode_matches_torch_sdpa,
                P.test_decode_special_cases, P.test_decode_append_order,
                P.test_alpha_zero_is_identity_and_full_attention]
_KEEP_PINS = [P.test_keep_count_table, P.test_keep_count_edges]

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


# pins driven by hypothesis draw their cases at random; each mutant must also
# fail at least one pin that runs fixed cases, so the result does not depend
# on the draw
_RANDOM = {P.test_rows_are_distributions_and_mass_is_Gw, P.test_window_probs_match_torch_sdpa,
           P.test_max_pool_matches_torch, P.test_select_matches_brute_force,
           P.test_decode_matches_torch_sdpa, P.test_split_merge_equals_direct}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, monkeypatch):
    attr, mutant, pins = MUTANTS[name]
    monkeypatch.setattr(O, attr, mutant)
    caught = []
    for pin in [p for p in pins if p not in _RANDOM]:
        try:
            pin()
        except (Exception, pytest.fail.Exception):   # an assertion, a failed
            caught.append(pin.__name__)              # pytest.raises, or an error it causes
    assert caught, f"no fixed-case pin fails when the oracle has: {name}"


def test_pins_pass_on_the_oracle():
    """The same pins, run the same way, pass on the unmodified oracle."""
    pins = {p for _, _, ps in MUTANTS.values() for p in ps if p not in _RANDOM}
    for pin in sorted(pins, key=lambda p: p.__name__):
        pin()
