"""Pins of the float64 oracle against facts that do not come from the oracle.

Each test checks the oracle against a hand-derived worked example, a closed
form, an invariant, a library routine computing the same definition, or brute
force on tiny inputs.  None of them touches the GPU.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

from oracle import timebill_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _frac(pairs):
    return np.array([n / d for n, d in pairs], dtype=np.float64)


def _hand():
    with open(os.path.join(GOLDEN, "hand_example.json")) as f:
        return json.load(f)


def _hand_inputs(h):
    p = h["prompt"]
    c = np.array(p["c"], dtype=np.float64)
    k = np.log(c).reshape(1, p["n_x"], 1)                 # [Hkv, n_x, d]
    v = np.zeros_like(k)
    q = np.array(p["q_win"], dtype=np.float64).reshape(p["Hq"], p["w"], 1)
    return q, k, v, p


# ---------------------------------------------------------------- worked example
def test_hand_example_column_mass_and_mask():
    h = _hand()
    q, k, _, p = _hand_inputs(h)
    mass = O.window_column_mass(q, k, p["n_x"], 0)
    np.testing.assert_allclose(mass, _frac(h["column_mass"]), rtol=1e-14, atol=0)


def test_hand_example_scores_and_pool():
    h = _hand()
    q, k, _, p = _hand_inputs(h)
    raw = O.window_scores(q, k, p["n_x"], p["w"])
    np.testing.assert_allclose(raw[0], _frac(h["raw_scores"]), rtol=1e-14, atol=0)
    for P, vals in h["pooled"].items():
        pooled = O.max_pool(raw, int(P))
        np.testing.assert_allclose(pooled[0], _frac(vals), rtol=1e-14, atol=0)


def test_hand_example_keep():
    h = _hand()
    q, k, v, p = _hand_inputs(h)
    for case in h["keep"]:
        r = O.evict_sequence(q, k, v, p["n_x"], p["w"], case["pool"], case["alpha"])
        assert r["n_keep"] == case["n_keep"]
        assert r["keep"][0].tolist() == case["keep"]


def test_hand_example_decode():
    h = _hand()["decode"]
    kc = np.log(np.array(h["k_cache_c"], dtype=np.float64)).reshape(1, -1, 1)
    vc = np.array(h["v_cache"], dtype=np.float64).reshape(1, -1, 1)
    kn = np.log(np.array(h["k_new_c"], dtype=np.float64)).reshape(-1, 1, 1)
    vn = np.array(h["v_new"], dtype=np.float64).reshape(-1, 1, 1)
    q = np.array(h["q"], dtype=np.float64).reshape(2, 2, 1)      # [T, Hq, d]
    out = O.decode_sequence(q, kn, vn, kc, vc)
    for t in range(2):
        np.testing.assert_allclose(out[t][:, 0], _frac(h["out"][t]), rtol=1e-14)


# ---------------------------------------------------------------- n_keep
def test_keep_count_table():
    with open(os.path.join(GOLDEN, "n_keep_table.json")) as f:
        tab = json.load(f)
    for case in tab["cases"]:
        alphas = case.get("alphas") or [k / 20 for k in case["alphas_k_over_20"]]
        got = [O.keep_count(case["n_x"], a, case["w"]) for a in alphas]
        assert got == case["n_keep"]


def test_keep_count_edges():
    assert O.keep_count(100, 0.0, 4) == 100
    assert O.keep_count(100, 0.99, 4) == 4          # clamped to the window
    assert O.keep_count(10, 0.5, 9) == 9
    for bad in [(10, 1.0, 2), (10, -0.1, 2), (10, 0.5, 10), (10, 0.5, 0)]:
        with pytest.raises(ValueError):
            O.keep_count(*bad)


# ---------------------------------------------------------------- softmax pins
def _rand_prompt(rng, hq, hkv, w, n_x, d):
    q = rng.standard_normal((hq, w, d))
    k = rng.standard_normal((hkv, n_x, d))
    v = rng.standard_normal((hkv, n_x, d))
    return q, k, v


@settings(max_examples=40, deadline=None)
@given(st.integers(1, 3), st.sampled_from([1, 2, 4]), st.integers(1, 6),
       st.integers(2, 40), st.sampled_from([1, 3, 8]), st.integers(0, 10_000))
def test_rows_are_distributions_and_mass_is_Gw(hkv, G, w, extra, d, seed):
    rng = np.random.default_rng(seed)
    n_x = w + extra
    q, k, _ = _rand_prompt(rng, hkv * G, hkv, w, n_x, d)
    for g in range(hkv):
        p = O.window_probs(q, k, n_x, g)
        np.testing.assert_allclose(p.sum(axis=1), 1.0, atol=1e-12)
        assert abs(O.window_column_mass(q, k, n_x, g).sum() - G * w) < 1e-11


@settings(max_examples=30, deadline=None)
@given(st.sampled_from([1, 2, 4]), st.integers(1, 5), st.integers(1, 30),
       st.sampled_from([2, 8]), st.integers(0, 10_000))
def test_window_probs_match_torch_sdpa(G, w, extra, d, seed):
    """p @ V of the oracle equals torch's attention with an explicit causal mask."""
    _check_window_probs(G, w, extra, d, seed)


@pytest.mark.parametrize("G,w,extra,d,seed", [(2, 3, 9, 8, 1), (4, 5, 20, 2, 7), (1, 1, 3, 8, 2)])
def test_window_probs_match_torch_sdpa_fixed(G, w, extra, d, seed):
    """Fixed instances of the check above (two KV groups, d > 1)."""
    _check_window_probs(G, w, extra, d, seed)


def _check_window_probs(G, w, extra, d, seed):
    rng = np.random.default_rng(seed)
    n_x = w + extra
    hkv = 2
    q, k, v = _rand_prompt(rng, hkv * G, hkv, w, n_x, d)
    pos = n_x - w + np.arange(w)
    allowed = np.arange(n_x)[None, :] <= pos[:, None]              # [w, n_x]
    mask = torch.from_numpy(allowed)
    for g in range(hkv):
        p = O.window_probs(q, k, n_x, g)                             # [G*w, n_x]
        mine = (p @ v[g]).reshape(G, w, d)
        tq = torch.from_numpy(q[g * G:(g + 1) * G])                  # [G, w, d]
        tk = torch.from_numpy(k[g]).expand(G, n_x, d)
        tv = torch.from_numpy(v[g]).expand(G, n_x, d)
        ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask)
        np.testing.assert_allclose(mine, ref.numpy(), rtol=0, atol=1e-12)
        # and the softmax itself against torch.softmax on the masked logits
        s = torch.from_numpy(O.window_logits(q, k, n_x, g))
        np.testing.assert_allclose(p, torch.softmax(s, dim=1).numpy(), atol=1e-14)


# ---------------------------------------------------------------- pooling
@settings(max_examples=40, deadline=None)
@given(st.integers(1, 60), st.sampled_from([1, 3, 5, 7, 9]), st.integers(0, 10_000))
def test_max_pool_matches_torch(n, P, seed):
    rng = np.random.default_rng(seed)
    a = rng.random((3, n))
    mine = O.max_pool(a, P)
    ref = torch.nn.functional.max_pool1d(torch.from_numpy(a)[None], P, stride=1,
                                         padding=P // 2)[0].numpy()
    np.testing.assert_array_equal(mine, ref)
    np.testing.assert_array_equal(O.max_pool(a, 1), a)
    np.testing.assert_array_equal(O.max_pool(np.full((2, n), 0.25), P), np.full((2, n), 0.25))


def test_max_pool_rejects_even():
    with pytest.raises(ValueError):
        O.max_pool(np.zeros(5), 4)


# ---------------------------------------------------------------- selection
def _brute_force_keep(pooled, n_sel):
    """Max-sum subset of size n_sel; among equal sums the lexicographically
    smallest ascending index tuple (i.e. ties go to lower positions)."""
    best = None
    for sub in itertools.combinations(range(len(pooled)), n_sel):
        key = (-math.fsum(pooled[list(sub)]), sub)
        if best is None or key < best:
            best = key
    return list(best[1]) if best else []


@settings(max_examples=60, deadline=None)
@given(st.integers(2, 14), st.integers(1, 3), st.integers(0, 10_000),
       st.sampled_from([1, 3, 5]), st.booleans())
def test_select_matches_brute_force(n_x, w, seed, P, few_values):
    if w >= n_x:
        return
    rng = np.random.default_rng(seed)
    pref = n_x - w
    if few_values:   # many exact ties, as max-pool plateaus produce
        raw = rng.integers(0, 3, pref).astype(np.float64) / 4
    else:
        raw = rng.random(pref)
    pooled = O.max_pool(raw, P)
    for n_keep in range(w, n_x + 1):
        keep = O.select_keep(pooled, n_x, w, n_keep)
        expect = _brute_force_keep(pooled, n_keep - w) + list(range(pref, n_x))
        assert keep.tolist() == expect
        # rank formulation: j kept iff fewer than n_sel positions beat it
        n_sel = n_keep - w
        for j in range(pref):
            beats = sum(1 for i in range(pref)
                        if pooled[i] > pooled[j] or (pooled[i] == pooled[j] and i < j))
            assert (j in set(keep.tolist())) == (beats < n_sel)


# ---------------------------------------------------------------- alpha = 0 and decode
def test_alpha_zero_is_identity_and_full_attention():
    rng = np.random.default_rng(7)
    hq, hkv, w, n_x, d, T = 4, 2, 3, 23, 8, 4
    q, k, v = _rand_prompt(rng, hq, hkv, w, n_x, d)
    r = O.evict_sequence(q, k, v, n_x, w, 3, 0.0)
    assert r["n_keep"] == n_x
    for g in range(hkv):
        assert r["keep"][g].tolist() == list(range(n_x))
        assert np.array_equal(r["k_cache"][g], k[g]) and np.array_equal(r["v_cache"][g], v[g])
    qs = rng.standard_normal((T, hq, d))
    kn = rng.standard_normal((T, hkv, d))
    vn = rng.standard_normal((T, hkv, d))
    a = O.decode_sequence(qs, kn, vn, r["k_cache"], r["v_cache"])
    b = O.decode_sequence(qs, kn, vn, k, v)
    for t in range(T):
        assert np.array_equal(a[t], b[t])


@settings(max_examples=30, deadline=None)
@given(st.sampled_from([1, 2, 7]), st.integers(1, 50), st.sampled_from([4, 16]),
       st.integers(0, 10_000))
def test_decode_matches_torch_sdpa(G, N, d, seed):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((G, d))
    kc = rng.standard_normal((N, d))
    vc = rng.standard_normal((N, d))
    mine = O.decode_step(q, kc, vc)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[:, None], torch.from_numpy(kc).expand(G, N, d),
        torch.from_numpy(vc).expand(G, N, d))[:, 0].numpy()
    np.testing.assert_allclose(mine, ref, rtol=0, atol=1e-12)


def test_decode_special_cases():
    rng = np.random.default_rng(3)
    d = 8
    q = rng.standard_normal((3, d))
    v1 = rng.standard_normal((1, d))
    np.testing.assert_allclose(O.decode_step(q, rng.standard_normal((1, d)), v1),
                               np.repeat(v1, 3, 0), atol=1e-15)
    kc = np.repeat(rng.standard_normal((1, d)), 9, 0)
    vc = rng.standard_normal((9, d))
    np.testing.assert_allclose(O.decode_step(q, kc, vc), np.repeat(vc.mean(0, keepdims=True), 3, 0),
                               atol=1e-14)
    vconst = np.full((9, d), 0.375)
    np.testing.assert_allclose(O.decode_step(q, rng.standard_normal((9, d)), vconst), 0.375,
                               atol=1e-15)
    np.testing.assert_allclose(O.decode_step(np.zeros((2, d)), rng.standard_normal((9, d)), vc),
                               np.repeat(vc.mean(0, keepdims=True), 2, 0), atol=1e-14)


@settings(max_examples=30, deadline=None)
@given(st.integers(1, 80), st.integers(1, 9), st.integers(0, 10_000))
def test_split_merge_equals_direct(N, n_chunks, seed):
    _check_split_merge(N, n_chunks, seed)


@pytest.mark.parametrize("N,n_chunks,seed", [(50, 7, 3), (9, 3, 11), (80, 1, 5)])
def test_split_merge_equals_direct_fixed(N, n_chunks, seed):
    """Fixed instances of the check above."""
    _check_split_merge(N, n_chunks, seed)


def _check_split_merge(N, n_chunks, seed):
    rng = np.random.default_rng(seed)
    d, G = 16, 7
    q = rng.standard_normal((G, d)) * 2
    kc = rng.standard_normal((N, d))
    vc = rng.standard_normal((N, d))
    cuts = sorted(set([0, N] + rng.integers(1, max(N, 2), n_chunks).tolist()))
    cuts = [c for c in cuts if c <= N]
    parts = [O.decode_partial(q, kc[a:b], vc[a:b]) for a, b in zip(cuts[:-1], cuts[1:]) if b > a]
    np.testing.assert_allclose(O.merge_partials(parts), O.decode_step(q, kc, vc), atol=1e-12)


def test_decode_append_order():
    """Step t attends over the n_keep cached rows plus t + 1 appended rows."""
    rng = np.random.default_rng(11)
    G, d, n, T = 2, 4, 5, 3
    q = rng.standard_normal((T, G, d))
    kc, vc = rng.standard_normal((1, n, d)), rng.standard_normal((1, n, d))
    kn, vn = rng.standard_normal((T, 1, d)), rng.standard_normal((T, 1, d))
    out = O.decode_sequence(q, kn, vn, kc, vc)
    for t in range(T):
        # weights by hand: exp(q.k/sqrt d) over the n + t + 1 rows
        rows_k = np.concatenate([kc[0], kn[:t + 1, 0]])
        rows_v = np.concatenate([vc[0], vn[:t + 1, 0]])
        for h in range(G):
            wts = np.array([math.exp(float(q[t, h] @ r) / 2.0) for r in rows_k])
            np.testing.assert_allclose(out[t][h], (wts[:, None] * rows_v).sum(0) / wts.sum(),
                                       atol=1e-13)


def test_fraction_sanity_of_hand_example():
    """The hand fractions themselves: column sums total G*w."""
    h = _hand()
    total = sum(Fraction(n, d) for n, d in h["column_mass"])
    assert total == 4


def test_prefill_attention_matches_torch_sdpa():
    """Causal prefill attention and the window statistics against torch's float64
    scaled_dot_product_attention (KV heads repeated by G) and logsumexp."""
    rng = np.random.default_rng(41)
    hq, hkv, n, d, w = 6, 2, 77, 32, 5
    q = rng.standard_normal((hq, n, d))
    k = rng.standard_normal((hkv, n, d)) * 1.3
    v = rng.standard_normal((hkv, n, d))
    got = O.prefill_attention(q, k, v, n)
    qt = torch.from_numpy(q)[None]
    kt = torch.from_numpy(k).repeat_interleave(hq // hkv, dim=0)[None]
    vt = torch.from_numpy(v).repeat_interleave(hq // hkv, dim=0)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True)[0]
    np.testing.assert_allclose(got, ref.numpy(), rtol=1e-12, atol=1e-12)
    rows = [0, 1, 40, n - 1]
    np.testing.assert_allclose(O.prefill_attention(q, k, v, n, rows), got[:, rows], rtol=0, atol=0)
    st = O.prefill_window_stats(q, k, n, w)
    logits = (qt[0] @ kt[0].transpose(1, 2)) / math.sqrt(d)
    mask = torch.ones(n, n, dtype=torch.bool).tril()
    logits = logits.masked_fill(~mask, float("-inf"))[:, n - w:]
    lse = torch.logsumexp(logits, dim=-1).numpy()
    np.testing.assert_allclose(st[..., 0], logits.max(dim=-1).values.numpy(), rtol=0, atol=1e-13)
    np.testing.assert_allclose(st[..., 0] + np.log(st[..., 1]), lse, rtol=1e-13)
    # row 0 attends to key 0 only: its output is v[0]
    np.testing.assert_allclose(got[:, 0], np.repeat(v[:, 0], hq // hkv, axis=0), rtol=0, atol=0)
