"""Comparison rules between the HIP path and the float64 oracle.

Selection acceptance: for each (sequence, layer, KV head) the GPU and the
oracle keep the same number of positions; every position in their symmetric
difference must have an oracle pooled score within REL_BAND (relative) of the
oracle's n_sel-th largest prefix score; window positions are never in the
difference; the GPU list is ascending in the prefix and ends with the window.

Decode outputs are checked against the oracle decode run on the GPU's own
kept set, so allowed selection differences never count as decode errors.
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import timebill_oracle as O

REL_BAND = 1e-6
DECODE_TOL = {torch.bfloat16: 2e-2, torch.float32: 1e-5}


def f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu").to(torch.float64).numpy()


def check_keep(gpu_keep: np.ndarray, pooled: np.ndarray, n_x: int, w: int, n_keep: int,
               where: str = "") -> int:
    """Apply the acceptance rule to one KV head; returns the excused-difference count."""
    pref = n_x - w
    gk = np.asarray(gpu_keep, dtype=np.int64)
    assert gk.shape == (n_keep,), f"{where}: GPU kept {gk.shape} positions, expected {n_keep}"
    assert np.array_equal(gk[n_keep - w:], np.arange(pref, n_x)), f"{where}: window not last"
    sel = gk[: n_keep - w]
    assert np.all(np.diff(sel) > 0), f"{where}: kept prefix positions not strictly ascending"
    assert sel.size == 0 or (sel[0] >= 0 and sel[-1] < pref), f"{where}: index out of prefix"
    ok = O.select_keep(pooled, n_x, w, n_keep)[: n_keep - w]
    diff = np.setxor1d(sel, ok)
    if diff.size == 0:
        return 0
    n_sel = n_keep - w
    kth = np.sort(pooled)[::-1][n_sel - 1]
    band = np.abs(pooled[diff] - kth) <= REL_BAND * abs(kth)
    assert np.all(band), (
        f"{where}: {int((~band).sum())} of {diff.size} differing positions lie outside the "
        f"{REL_BAND:g} band around the boundary score {kth!r}: "
        f"{diff[~band][:8].tolist()} with scores {pooled[diff[~band][:8]].tolist()}")
    return int(diff.size)


def score_rel_err(gpu: np.ndarray, ref: np.ndarray) -> float:
    return float(np.max(np.abs(gpu - ref) / np.maximum(np.abs(ref), 1e-300)))


def score_rel_err_p99(gpu: np.ndarray, ref: np.ndarray) -> float:
    """99th percentile of the per-position relative score error."""
    e = np.abs(gpu - ref) / np.maximum(np.abs(ref), 1e-300)
    return float(np.percentile(e, 99))
