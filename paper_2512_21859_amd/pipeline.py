"""Orchestration of the eviction + decode path over the C ABI.

Eviction happens once per request and layer after the prefill phase
(score -> select -> compact), then every decode step appends the new token's
K/V and attends over the retained cache (TimeBill Sec. 5.2 deployment; the
retained length follows Eq. N_kv).  This module only allocates device buffers
(torch) and sequences library calls; all arithmetic runs in the kernels.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

import torch

from . import _lib


SCORERS = ("snapkv", "snapkv_avg", "knorm", "h2o")


class Evictor:
    """Score / select buffers and workspace for one layer shape.

    scorer: "snapkv" (observation-window scores, max-pooled; the paper's
    eviction), "snapkv_avg" (the same scores mean-pooled), "knorm" (negated
    key norms; the window queries are not used) or "h2o" (accumulated
    attention of every prompt query: score() then takes all the prefill's
    queries [B, Hq, Lmax, d] in place of the window queries)."""

    def __init__(self, B: int, Lmax: int, Hq: int, Hkv: int, d: int, w: int, pool: int,
                 device="cuda", keep_raw: bool = False, scorer: str = "snapkv"):
        if scorer not in SCORERS:
            raise ValueError(f"scorer must be one of {SCORERS}")
        self.scorer = scorer
        self.B, self.Lmax, self.Hq, self.Hkv, self.d, self.w, self.pool = B, Lmax, Hq, Hkv, d, w, pool
        self.scores = torch.empty((B, Hkv, Lmax), dtype=torch.float32, device=device)
        self.raw = (torch.empty((B, Hkv, Lmax), dtype=torch.float32, device=device)
                    if keep_raw else None)
        self.keep_idx = torch.empty((B, Hkv, Lmax), dtype=torch.int32, device=device)
        if scorer == "knorm":
            nbytes = 0
        elif scorer == "h2o":
            nbytes = _lib.tb_workspace_bytes(_lib.TB_OP_H2O, B, Lmax, Hq, Hkv, d, 0, 0)
        else:
            nbytes = _lib.tb_workspace_bytes(_lib.TB_OP_SCORE, B, Lmax, Hq, Hkv, d, w, 0)
        self.ws = torch.empty((max(nbytes, 1),), dtype=torch.uint8, device=device)
        # long prefixes select with several blocks per KV head, which needs this
        sel = _lib.tb_workspace_bytes(_lib.TB_OP_SELECT, B, Lmax, Hq, Hkv, d, w, 0)
        self.sel_ws = torch.empty((sel,), dtype=torch.uint8, device=device) if sel else None

    def score(self, q_win: torch.Tensor, k: torch.Tensor, L: Sequence[int], stream=None) -> None:
        self.score_into(q_win, k, L, self.scores, self.raw, stream)

    def score_into(self, q_win, k, L, scores, raw=None, stream=None) -> None:
        """score() into caller-given [B, Hkv, Lmax] scores (and raw scores)."""
        if self.scorer == "knorm":
            _lib.tb_score_knorm(k, L, self.w, scores, stream)
        elif self.scorer == "h2o":
            _lib.tb_score_h2o(q_win, k, L, scores, self.ws, stream)
        else:
            _lib.tb_score_window(q_win, k, L, self.w, self.pool, scores, raw, self.ws,
                                 stream, avgpool=self.scorer == "snapkv_avg")

    def select(self, L: Sequence[int], alphas: Sequence[float], stream=None):
        return _lib.tb_select_topk(self.scores, L, self.w, alphas, self.keep_idx, self.sel_ws,
                                   stream)

    def evict(self, q_win, k, v, L, alphas, cache: "_lib.KVCache", stream=None):
        """Score, select and compact into ``cache``; returns n_keep per sequence."""
        self.score(q_win, k, L, stream)
        n_keep = self.select(L, alphas, stream)
        cache.compact_from(k, v, self.keep_idx, n_keep, stream)
        return n_keep


class StackEvictor:
    """Eviction of a stack of layers of one shape, laid out layer-major on the
    batch axis: sequence b of layer l is row l * B + b of every [layers * B,
    ...] tensor.  Each layer is scored on its own (one layer's scoring
    workspace, whose exponentials stay in the last-level cache), then one
    selection and one compaction cover the whole stack: at B = 1 and 4 KV
    heads a selection of one layer keeps 4 CUs busy, the stack's keeps
    4 * layers.  Layer by layer the results equal those of an Evictor.
    layers * B may not exceed the library's batch limit (64)."""

    def __init__(self, layers: int, B: int, Lmax: int, Hq: int, Hkv: int, d: int, w: int,
                 pool: int, device="cuda", scorer: str = "snapkv"):
        if layers < 1 or layers * B > _lib.MAX_B:
            raise ValueError(f"need 1 <= layers and layers * B <= {_lib.MAX_B}")
        self.layers, self.B = layers, B
        self.layer = Evictor(B, Lmax, Hq, Hkv, d, w, pool, device=device, scorer=scorer)
        NB = layers * B
        self.scores = torch.empty((NB, Hkv, Lmax), dtype=torch.float32, device=device)
        self.keep_idx = torch.empty((NB, Hkv, Lmax), dtype=torch.int32, device=device)
        sel = _lib.tb_workspace_bytes(_lib.TB_OP_SELECT, NB, Lmax, Hq, Hkv, d, w, 0)
        self.sel_ws = torch.empty((sel,), dtype=torch.uint8, device=device) if sel else None

    def evict(self, q_win, k, v, L: Sequence[int], alphas: Sequence[float],
              cache: "_lib.KVCache", stream=None) -> List[int]:
        """q_win [layers*B, Hq, w, d] (or the prefill's queries for h2o), k, v
        [layers*B, Hkv, Lmax, d]; L and alphas per sequence (B values, the
        same for every layer); cache has batch layers*B.  Returns n_keep per
        row of the stack."""
        B, NB = self.B, self.layers * self.B
        if k.shape[0] != NB or v.shape[0] != NB or q_win.shape[0] != NB:
            raise ValueError("q_win, k and v must hold layers * B sequences")
        if len(L) != B or len(alphas) != B:
            raise ValueError("L and alphas take one value per sequence of a layer")
        for l in range(self.layers):
            s = slice(l * B, (l + 1) * B)
            self.layer.score_into(q_win[s], k[s], L, self.scores[s], None, stream)
        Ls, als = list(L) * self.layers, list(alphas) * self.layers
        n_keep = _lib.tb_select_topk(self.scores, Ls, self.layer.w, als, self.keep_idx,
                                     self.sel_ws, stream)
        cache.compact_from(k, v, self.keep_idx, n_keep, stream)
        return n_keep


def run_decode(cache: "_lib.KVCache", q: torch.Tensor, k_new: torch.Tensor,
               v_new: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None):
    """Decode T steps: q [T,B,Hq,d], k_new/v_new [T,B,Hkv,d] -> out [T,B,Hq,d]."""
    T = q.shape[0]
    if out is None:
        out = torch.empty_like(q)
    for t in range(T):
        cache.decode(q[t], k_new[t], v_new[t], out[t], stream)
    return out


def choose_alpha(prefill_abc, step_pq, n_x: int, n_hat: int, bucket: int, k: int, n_max: int,
                 budget: float, t_predict: float = 0.0, alpha_max: float = 0.95):
    """Per-request eviction ratio (Sec. 5.2 deployment): the predicted bucket
    n_hat gives N_hat = min(N_max, n_hat * B) (Eq. predictor_inference), the
    pessimistic length N_hat_W = min(k * N_hat, N_max), and alpha* is the
    smallest ratio meeting the budget (tb_response_length and tb_alpha_star).
    Returns (alpha, feasible, N_hat_W)."""
    _, n_hat_w = _lib.tb_response_length(n_hat, bucket, k, n_max)
    alpha, feasible = _lib.tb_alpha_star(prefill_abc, step_pq, float(n_x), n_hat_w, budget,
                                         t_predict, alpha_max)
    return alpha, feasible, n_hat_w


@dataclass(frozen=True)
class TimeModel:
    """What the controller plans with (Sec. 5.1, Sec. 5.2): the prefill time
    a N^2 + b N + c and the decode-step time p N_kv + q (coefficients from
    tb_ete_fit over measured runs), the predictor's bucket size, the pessimism
    factor k, the response-length cap N_max, the predictor's own time and the
    largest ratio the deployment allows."""
    prefill_abc: Tuple[float, float, float]
    step_pq: Tuple[float, float]
    bucket: int
    k: int
    n_max: int
    t_predict: float = 0.0
    alpha_max: float = 0.95


def plan_requests(model: TimeModel, n_x: Sequence[int], budgets: Sequence[float],
                  n_hat: Sequence[int]) -> List[Tuple[float, bool, int]]:
    """choose_alpha for each request: (alpha*, feasible, N_hat_W).  A request
    whose budget cannot be met gets alpha_max with feasible False (it runs
    with the most eviction the deployment allows)."""
    if not (len(n_x) == len(budgets) == len(n_hat)):
        raise ValueError("n_x, budgets and n_hat must have one entry per request")
    return [choose_alpha(model.prefill_abc, model.step_pq, int(n), int(nh), model.bucket,
                         model.k, model.n_max, float(T), model.t_predict, model.alpha_max)
            for n, T, nh in zip(n_x, budgets, n_hat)]
