"""Float64 reference of the alternative eviction scorers.

TEST INFRASTRUCTURE ONLY (same rules as timebill_oracle: only tests, the smoke
check and the benchmark's CPU-baseline leg may use it; no code is shared with
the HIP path).

TimeBill evicts with SnapKV (Sec. 6.1) and compares against fixed-ratio
eviction whose scorers it cites without defining them (Sec. 6.1, the
fixed-alpha baselines, citing KNorm and H2O).  Three variants are built on the
same select / compact / decode path:

* KNorm: a prefix key's score is the negated L2 norm of its (post-RoPE) key
  vector, so keeping the largest scores keeps the smallest norms (the cited
  norm-based strategy).  Reading: as for SnapKV, the last w positions are
  always kept and only the prefix j < N_x - w competes; ties go to the lower
  position.
* H2O: a key's score is the attention mass it receives from every prompt
  query under the causal softmax of Sec. 4.2, summed over the G query heads of
  its KV head (the accumulated-attention "heavy hitter" score).  Reading: the
  queries are the prefill's (post-RoPE) queries at all N_x positions; there is
  no pooling; the last w positions are kept as a recent window and count
  toward n_keep, the prefix j < N_x - w competes; ties go to the lower
  position.
* Average-pool SnapKV: the window scores of timebill_oracle.window_scores
  smoothed by a mean instead of a max.  Reading: odd kernel P, stride 1,
  "same" length, positions outside the prefix count as zeros and the divisor
  is always P (the convention of torch.nn.functional.avg_pool1d with
  count_include_pad=True).
"""
from __future__ import annotations

import numpy as np

__all__ = ["knorm_scores", "avg_pool", "h2o_scores"]


def knorm_scores(k: np.ndarray, n_x: int, w: int) -> np.ndarray:
    """k [Hkv, >= n_x, d] -> scores [Hkv, n_x - w]: -||k_j||_2 for j < n_x - w."""
    pref = n_x - w
    kk = np.asarray(k[:, :pref, :], dtype=np.float64)
    return -np.sqrt(np.sum(kk * kk, axis=-1))


def avg_pool(a: np.ndarray, pool: int) -> np.ndarray:
    """Mean over the odd window |i - j| <= pool // 2 along the last axis, with
    out-of-range positions counted as zeros and a fixed divisor pool."""
    if pool < 1 or pool % 2 == 0:
        raise ValueError("pool must be odd and >= 1")
    a = np.asarray(a, dtype=np.float64)
    h = pool // 2
    n = a.shape[-1]
    padded = np.concatenate([np.zeros(a.shape[:-1] + (h,)), a,
                             np.zeros(a.shape[:-1] + (h,))], axis=-1)
    out = np.zeros_like(a)
    for off in range(pool):             # sum of the pool shifted copies
        out += padded[..., off:off + n]
    return out / pool


def h2o_scores(q: np.ndarray, k: np.ndarray, n_x: int) -> np.ndarray:
    """q [Hq, >= n_x, d], k [Hkv, >= n_x, d] -> [Hkv, n_x]: for key j, the sum over
    the group's query heads h and query positions i >= j of
    softmax_{j' <= i}(q[h, i] . k[j'] / sqrt(d)) at j'."""
    hq, hkv = q.shape[0], k.shape[0]
    G = hq // hkv
    d = q.shape[-1]
    scale = 1.0 / np.sqrt(d)
    causal = np.tril(np.ones((n_x, n_x), dtype=bool))          # row i sees j <= i
    out = np.zeros((hkv, n_x), dtype=np.float64)
    for h in range(hq):
        g = h // G
        s = (np.asarray(q[h, :n_x], dtype=np.float64) @ np.asarray(k[g, :n_x], dtype=np.float64).T) * scale
        s = np.where(causal, s, -np.inf)
        s -= s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        out[g] += p.sum(axis=0)
    return out
