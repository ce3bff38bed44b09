"""Float64 CPU oracle for the TimeBill eviction + decode hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product package may import, call or
link this module; only the test suite, the smoke check and the benchmark's
CPU-baseline leg use it.  It shares no code with the HIP path.

What it computes (TimeBill, arXiv 2512.21859):

* Eviction happens once, after the prefill phase and before the decoding
  phase, and removes a fraction alpha of the prompt's KV cache, so that the
  retained length at decode step i is (1 - alpha) * N_x + i - 1
  (Sec. 4.2, "End-to-end Execution Time Prediction", Eq. N_kv).  The paper
  performs the eviction with SnapKV (Sec. 6.1, experimental setup).
* Attention is softmax(Q K^T / sqrt(d)) V under a causal mask
  (Sec. 4.2, "FLOPs-based Modeling").  In a decoding step Q has length 1 and
  K has length N_kv (same paragraph).

The paper does not spell out SnapKV's scoring, so the steps below follow the
observation-window recipe the method names (window queries against the prompt
keys, softmax, a sum over the window, a 1-D max-pool, a per-KV-head top-k),
with these readings where the paper is silent:

* the observation window is the last ``w`` prompt positions; window row i sits
  at absolute position N_x - w + i and sees keys j <= N_x - w + i;
* the logit scale is 1/sqrt(d_head) (the paper's "hidden size" is read as the
  head dimension);
* the mask is additive -inf (the paper's elementwise product with M is read as
  the usual causal mask);
* the softmax runs over the whole causal row; only prefix columns
  j < N_x - w are scored;
* the G = Hq/Hkv query heads of a KV head are summed (not averaged) together
  with the w window rows, then pooled once per KV head;
* the max-pool has odd kernel P, stride 1, "same" length, out-of-range
  neighbours ignored, and runs over the prefix only;
* n_keep = N_x - floor(alpha * N_x) in IEEE double, at least w; the w window
  positions are always kept and count toward n_keep;
* ties in the pooled score go to the lower position; kept positions are in
  ascending order with the window last;
* at decode step t the new key/value row is appended first, then the query
  attends over n_keep + t rows.

Everything is float64.  Inputs are the exact values the GPU receives (bf16 or
fp32), upcast exactly.
"""
from __future__ import annotations

import math

import numpy as np

__all__ = [
    "keep_count",
    "window_logits",
    "window_probs",
    "window_column_mass",
    "window_scores",
    "max_pool",
    "select_keep",
    "compact",
    "decode_step",
    "prefill_attention",
    "prefill_window_stats",
    "decode_partial",
    "merge_partials",
    "evict_sequence",
    "decode_sequence",
]


def keep_count(n_x: int, alpha: float, w: int) -> int:
    """Retained positions after evicting a fraction alpha of n_x (Eq. N_kv).

    The paper writes the retained length as the real number (1 - alpha) N_x.
    It is made an integer as n_x - floor(alpha * n_x), with the product taken
    in IEEE double, so alpha = 0 keeps every position.  The observation window
    is always kept, so the count is at least w.
    """
    if not (0 < w < n_x) or not (0.0 <= alpha < 1.0):
        raise ValueError("need 0 < w < n_x and 0 <= alpha < 1")
    n_keep = n_x - math.floor(float(alpha) * float(n_x))
    return max(n_keep, w)


def _group_of(h: int, hq: int, hkv: int) -> int:
    """Query head h reads KV head h // (Hq / Hkv) (grouped-query attention)."""
    return h // (hq // hkv)


def window_logits(q_win: np.ndarray, k: np.ndarray, n_x: int, g: int) -> np.ndarray:
    """Masked logits of the observation-window rows of KV group g.

    q_win: [Hq, w, d] window queries of one sequence.
    k:     [Hkv, >= n_x, d] prompt keys of that sequence.
    Returns [G*w, n_x] with row r = (h - g*G) * w + i and -inf above the
    causal diagonal (row i may see keys j <= n_x - w + i).
    """
    hq, w, d = q_win.shape
    hkv = k.shape[0]
    G = hq // hkv
    q = np.asarray(q_win[g * G:(g + 1) * G], dtype=np.float64).reshape(G * w, d)
    kk = np.asarray(k[g, :n_x], dtype=np.float64)
    s = (q @ kk.T) / math.sqrt(d)
    i = np.tile(np.arange(w), G)                     # window index of each row
    pos = n_x - w + i                                # absolute position of the row
    j = np.arange(n_x)
    s[j[None, :] > pos[:, None]] = -np.inf
    return s


def window_probs(q_win: np.ndarray, k: np.ndarray, n_x: int, g: int) -> np.ndarray:
    """Row softmax of the window logits, max-subtracted ([G*w, n_x])."""
    s = window_logits(q_win, k, n_x, g)
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=1, keepdims=True)


def window_column_mass(q_win: np.ndarray, k: np.ndarray, n_x: int, g: int) -> np.ndarray:
    """Sum of the window probabilities per key over ALL n_x columns.

    Each of the G*w rows is a distribution, so this vector sums to G*w.
    """
    return window_probs(q_win, k, n_x, g).sum(axis=0)


def window_scores(q_win: np.ndarray, k: np.ndarray, n_x: int, w: int) -> np.ndarray:
    """Raw score per KV head and prefix position: [Hkv, n_x - w].

    A[g, j] = sum over the G query heads of group g and the w window rows of
    the softmax probability that row gives key j, for j < n_x - w.
    """
    hq = q_win.shape[0]
    hkv = k.shape[0]
    assert q_win.shape[1] == w and hq % hkv == 0
    out = np.empty((hkv, n_x - w), dtype=np.float64)
    for g in range(hkv):
        out[g] = window_column_mass(q_win, k, n_x, g)[: n_x - w]
    return out


def max_pool(a: np.ndarray, pool: int) -> np.ndarray:
    """1-D max-pool along the last axis: odd kernel, stride 1, same length.

    Out-of-range neighbours are ignored (padding with -inf).
    """
    if pool < 1 or pool % 2 == 0:
        raise ValueError("pool must be odd and >= 1")
    r = pool // 2
    pad = [(0, 0)] * (a.ndim - 1) + [(r, r)]
    padded = np.pad(np.asarray(a, dtype=np.float64), pad, constant_values=-np.inf)
    windows = np.lib.stride_tricks.sliding_window_view(padded, pool, axis=-1)
    return windows.max(axis=-1)


def select_keep(pooled: np.ndarray, n_x: int, w: int, n_keep: int) -> np.ndarray:
    """Kept positions of one KV head, ascending, window last.

    pooled: [n_x - w] pooled prefix scores.  The n_keep - w prefix positions
    with the largest score are selected, a tie going to the lower position.
    """
    n_sel = n_keep - w
    pref = n_x - w
    assert pooled.shape == (pref,) and 0 <= n_sel <= pref
    idx = np.arange(pref)
    order = np.lexsort((idx, -pooled))               # by (-score, position)
    chosen = np.sort(order[:n_sel])
    return np.concatenate([chosen, np.arange(pref, n_x)]).astype(np.int64)


def compact(k: np.ndarray, v: np.ndarray, keep: np.ndarray):
    """Gather the kept rows of one KV head: K_c = K[keep], V_c = V[keep]."""
    return (np.asarray(k, dtype=np.float64)[keep],
            np.asarray(v, dtype=np.float64)[keep])


def decode_step(q: np.ndarray, k_cache: np.ndarray, v_cache: np.ndarray) -> np.ndarray:
    """Single-token attention of one KV group.

    q: [G, d] queries of the group's heads; k_cache, v_cache: [N, d].
    Returns [G, d] = softmax(q K^T / sqrt(d)) V.
    """
    q = np.asarray(q, dtype=np.float64)
    kc = np.asarray(k_cache, dtype=np.float64)
    vc = np.asarray(v_cache, dtype=np.float64)
    d = q.shape[-1]
    s = (q @ kc.T) / math.sqrt(d)
    m = s.max(axis=1, keepdims=True)
    p = np.exp(s - m)
    return (p @ vc) / p.sum(axis=1, keepdims=True)


def decode_partial(q: np.ndarray, k_chunk: np.ndarray, v_chunk: np.ndarray):
    """Unnormalised attention over one chunk of keys: (m, l, o).

    m = max logit, l = sum exp(s - m), o = sum exp(s - m) v.
    """
    q = np.asarray(q, dtype=np.float64)
    d = q.shape[-1]
    s = (q @ np.asarray(k_chunk, dtype=np.float64).T) / math.sqrt(d)
    m = s.max(axis=1)
    p = np.exp(s - m[:, None])
    return m, p.sum(axis=1), p @ np.asarray(v_chunk, dtype=np.float64)


def merge_partials(parts) -> np.ndarray:
    """Combine chunk partials (m, l, o) by log-sum-exp into the attention output."""
    ms = np.stack([p[0] for p in parts])             # [C, G]
    M = ms.max(axis=0)
    scale = np.exp(ms - M)                           # [C, G]
    L = sum(scale[c] * parts[c][1] for c in range(len(parts)))
    O = sum(scale[c][:, None] * parts[c][2] for c in range(len(parts)))
    return O / L[:, None]


def evict_sequence(q_win, k, v, n_x: int, w: int, pool: int, alpha: float):
    """Whole eviction of one sequence.

    q_win [Hq, w, d], k and v [Hkv, >= n_x, d].  Returns a dict with raw and
    pooled scores [Hkv, n_x - w], n_keep, keep [Hkv, n_keep] and the
    compacted caches [Hkv, n_keep, d].
    """
    hkv = k.shape[0]
    raw = window_scores(q_win, k, n_x, w)
    pooled = max_pool(raw, pool)
    n_keep = keep_count(n_x, alpha, w)
    keep = np.stack([select_keep(pooled[g], n_x, w, n_keep) for g in range(hkv)])
    kc = np.stack([compact(k[g], v[g], keep[g])[0] for g in range(hkv)])
    vc = np.stack([compact(k[g], v[g], keep[g])[1] for g in range(hkv)])
    return {"raw": raw, "pooled": pooled, "n_keep": n_keep, "keep": keep,
            "k_cache": kc, "v_cache": vc}


def decode_sequence(q_steps, k_new, v_new, k_cache, v_cache, steps=None):
    """Decode outputs of one sequence over its compacted cache.

    q_steps [T, Hq, d]; k_new, v_new [T, Hkv, d]; k_cache, v_cache
    [Hkv, n_keep, d].  Step t (0-based) appends rows 0..t of k_new/v_new and
    attends over n_keep + t + 1 rows.  ``steps`` limits the steps computed
    (each step is independent of the others' outputs).  Returns {t: [Hq, d]}.
    """
    T, hq, d = q_steps.shape
    hkv = k_cache.shape[0]
    G = hq // hkv
    kc = np.asarray(k_cache, dtype=np.float64)
    vc = np.asarray(v_cache, dtype=np.float64)
    kn = np.asarray(k_new, dtype=np.float64)
    vn = np.asarray(v_new, dtype=np.float64)
    out = {}
    for t in (range(T) if steps is None else steps):
        o = np.empty((hq, d), dtype=np.float64)
        for g in range(hkv):
            kk = np.concatenate([kc[g], kn[: t + 1, g]], axis=0)
            vv = np.concatenate([vc[g], vn[: t + 1, g]], axis=0)
            o[g * G:(g + 1) * G] = decode_step(q_steps[t, g * G:(g + 1) * G], kk, vv)
        out[t] = o
    return out


def prefill_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_x: int,
                      rows=None) -> np.ndarray:
    """Causal attention of the prompt (Sec. 4.2's attention with a causal mask):
    q [Hq, >= n_x, d], k/v [Hkv, >= n_x, d] -> [Hq, len(rows), d] for the query
    rows `rows` (default: all n_x), row i attending over keys 0..i."""
    hq, hkv = q.shape[0], k.shape[0]
    G = hq // hkv
    d = q.shape[-1]
    rows = np.arange(n_x) if rows is None else np.asarray(rows)
    out = np.empty((hq, len(rows), d), dtype=np.float64)
    for h in range(hq):
        g = h // G
        kk = np.asarray(k[g, :n_x], dtype=np.float64)
        vv = np.asarray(v[g, :n_x], dtype=np.float64)
        for r, i in enumerate(rows):
            out[h, r] = decode_step(np.asarray(q[h:h + 1, i], dtype=np.float64),
                                    kk[: i + 1], vv[: i + 1])[0]
    return out


def prefill_window_stats(q: np.ndarray, k: np.ndarray, n_x: int, w: int) -> np.ndarray:
    """For the last w query rows i = n_x - w + r: (M, Z) with M the row's largest
    logit q.k/sqrt(d) over keys 0..i and Z = sum_j exp(s_j - M).  [Hq, w, 2]."""
    hq, hkv = q.shape[0], k.shape[0]
    G = hq // hkv
    d = q.shape[-1]
    out = np.empty((hq, w, 2), dtype=np.float64)
    for h in range(hq):
        kk = np.asarray(k[h // G, :n_x], dtype=np.float64)
        for r in range(w):
            i = n_x - w + r
            s = kk[: i + 1] @ np.asarray(q[h, i], dtype=np.float64) / math.sqrt(d)
            m = s.max()
            out[h, r] = (m, np.exp(s - m).sum())
    return out
