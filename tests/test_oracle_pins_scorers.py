"""Pins of the alternative-scorer oracle (KNorm, average-pool SnapKV).

Hand-derived worked examples (tests/golden/scorers_example.json), closed forms,
the same definitions computed by library routines, and brute force on tiny
inputs.  None of them touches the GPU.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import scorers as S
from oracle import timebill_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _ex():
    with open(os.path.join(GOLDEN, "scorers_example.json")) as f:
        return json.load(f)


def _frac(pairs):
    return np.array([n / d for n, d in pairs], dtype=np.float64)


def test_knorm_hand_example():
    ex = _ex()["knorm"]
    k = np.array(ex["k"], dtype=np.float64)[None]          # [Hkv=1, n_x, d]
    sc = S.knorm_scores(k, ex["n_x"], ex["w"])[0]
    assert np.array_equal(sc, np.array(ex["scores"], dtype=np.float64))
    for case in ex["keep"]:
        n_keep = O.keep_count(ex["n_x"], case["alpha"], ex["w"])
        assert n_keep == case["n_keep"]
        keep = O.select_keep(sc, ex["n_x"], ex["w"], n_keep)
        assert keep.tolist() == case["keep"], case


def test_avg_pool_hand_example():
    ex = _ex()["avg_pool"]
    raw = _frac(ex["raw"])
    for p, want in ex["pooled"].items():
        np.testing.assert_allclose(S.avg_pool(raw, int(p)), _frac(want), rtol=0, atol=1e-15)
    for case in ex["keep"]:
        pooled = S.avg_pool(raw, case["pool"])
        n_keep = O.keep_count(ex["n_x"], case["alpha"], ex["w"])
        assert n_keep == case["n_keep"]
        assert O.select_keep(pooled, ex["n_x"], ex["w"], n_keep).tolist() == case["keep"], case


@pytest.mark.parametrize("pool", [1, 3, 5, 7, 9])
def test_avg_pool_matches_torch(pool):
    rng = np.random.default_rng(pool)
    a = rng.random((3, 101))
    ref = torch.nn.functional.avg_pool1d(torch.from_numpy(a)[:, None, :], pool, stride=1,
                                         padding=pool // 2, count_include_pad=True)[:, 0, :]
    np.testing.assert_allclose(S.avg_pool(a, pool), ref.numpy(), rtol=1e-15, atol=1e-16)


def test_avg_pool_constant_closed_form():
    c, n, p = 0.75, 20, 7
    out = S.avg_pool(np.full(n, c), p)
    h = p // 2
    for j in range(n):
        inside = min(j + h, n - 1) - max(j - h, 0) + 1
        assert math.isclose(out[j], c * inside / p, rel_tol=1e-15)


def test_knorm_matches_torch_norm():
    rng = np.random.default_rng(3)
    k = rng.standard_normal((2, 300, 128))
    got = S.knorm_scores(k, 300, 17)
    ref = -torch.linalg.vector_norm(torch.from_numpy(k[:, :283]), dim=-1).numpy()
    np.testing.assert_allclose(got, ref, rtol=1e-14)


def test_select_keep_signed_scores_bruteforce():
    """Top-k of negative and mixed-sign scores with ties, against all subsets."""
    rng = np.random.default_rng(11)
    for trial in range(60):
        n_x, w = int(rng.integers(5, 12)), int(rng.integers(1, 3))
        pref = n_x - w
        sc = rng.integers(-4, 3, pref).astype(np.float64) * 0.5
        if trial % 3 == 0:
            sc = -np.abs(sc) - 1.0                           # all negative
        for n_keep in range(w, n_x + 1):
            n_sel = n_keep - w
            best, best_sum = None, None
            for sub in itertools.combinations(range(pref), n_sel):
                s = math.fsum(sc[list(sub)])
                if best is None or s > best_sum:              # combinations() is lexicographic,
                    best, best_sum = sub, s                   # so the first maximum is the smallest set
            want = list(best) + list(range(pref, n_x))
            assert O.select_keep(sc, n_x, w, n_keep).tolist() == want


def test_h2o_hand_example():
    ex = _ex()["h2o"]
    c = np.array(ex["c"], dtype=np.float64)
    k = np.log(c).reshape(1, ex["n_x"], 1)
    q = np.array(ex["q"], dtype=np.float64).reshape(1, ex["n_x"], 1)
    sc = S.h2o_scores(q, k, ex["n_x"])[0]
    np.testing.assert_allclose(sc, _frac(ex["scores"]), rtol=1e-15)
    for case in ex["keep"]:
        n_keep = O.keep_count(ex["n_x"], case["alpha"], ex["w"])
        assert n_keep == case["n_keep"]
        keep = O.select_keep(sc[: ex["n_x"] - ex["w"]], ex["n_x"], ex["w"], n_keep)
        assert keep.tolist() == case["keep"], case


def test_h2o_total_mass_and_torch():
    """Every causal row sums to 1, so the scores of a KV head total G * N_x; the
    column sums equal those of torch's float64 softmax over a masked product."""
    rng = np.random.default_rng(5)
    hq, hkv, n, d = 6, 2, 97, 32
    q = rng.standard_normal((hq, n, d))
    k = rng.standard_normal((hkv, n, d)) * 1.5
    sc = S.h2o_scores(q, k, n)
    np.testing.assert_allclose(sc.sum(axis=1), np.full(hkv, (hq // hkv) * n), rtol=1e-13)
    qt = torch.from_numpy(q)
    kt = torch.from_numpy(k).repeat_interleave(hq // hkv, dim=0)
    mask = torch.ones(n, n, dtype=torch.bool).tril()
    logits = (qt @ kt.transpose(1, 2)) / math.sqrt(d)
    p = torch.softmax(logits.masked_fill(~mask, float("-inf")), dim=-1)
    ref = p.sum(dim=1).reshape(hkv, hq // hkv, n).sum(dim=1).numpy()
    np.testing.assert_allclose(sc, ref, rtol=1e-12)


def test_h2o_last_row_only_matches_window_mass():
    """The last query row's contribution equals the window column mass of a
    one-row window at the last position (both are one causal softmax row)."""
    rng = np.random.default_rng(8)
    hq, hkv, n, d = 2, 1, 40, 16
    q = rng.standard_normal((hq, n, d))
    k = rng.standard_normal((hkv, n, d))
    full = S.h2o_scores(q, k, n)
    head = S.h2o_scores(q[:, : n - 1], k, n - 1)                 # rows 0 .. n-2
    last = full[0].copy()
    last[: n - 1] -= head[0]
    mass = O.window_column_mass(q[:, n - 1:], k, n, 0)
    np.testing.assert_allclose(last, mass, rtol=1e-12, atol=1e-15)
