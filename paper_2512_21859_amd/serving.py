"""Multi-request serving over paged KV caches.

Each request brings its own time budget, hence its own eviction ratio
(Sec. 5.2: alpha* is solved per request from its prompt length and predicted
response length).  Requests are admitted in batches: one batched eviction
(score -> select with per-request ratios -> compaction into pages), after
which they join the running batch, where every decode step serves all active
requests in one launch per layer.

Layout: every layer has its own page pools (k_pool [P, Hkv, 32, d], v_pool
[P, Hkv, d, 32]); one block table [max_seqs, max_pages] serves all layers, so
a request owns the same page numbers in every layer.  Each layer keeps its own
kv_len [max_seqs] because every decode call appends to it.  The active
requests occupy slots 0..n-1 of the table; a retiring request's slot is
refilled by moving the last one in (its table row and lengths), so a decode
step is always one dense batch.

Pages are reserved at admission for the retained prompt plus the request's
whole response (max_new tokens), so a running request never waits for pages
and nothing is preempted.  The host holds the bookkeeping (which pages, which
slot, how long); this module allocates device buffers (torch) and sequences
library calls; every computation runs in the kernels.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from . import _lib

PAGE = _lib.V_TILE          # rows per page: one 32-row tile of every KV head


@dataclass
class Entry:
    """A request in the running batch."""
    rid: int
    pages: List[int]
    length: int              # rows now in its cache (retained prompt + appended tokens)
    left: int                # decode steps still to run
    alpha: float = 0.0
    n_x: int = 0


class SlotTable:
    """Host bookkeeping: free pages, the dense slot order and each request's
    pages and length.  No device access."""

    def __init__(self, n_pages: int, max_seqs: int, max_pages: int):
        if n_pages < 1 or max_seqs < 1 or max_pages < 1:
            raise ValueError("n_pages, max_seqs and max_pages must be >= 1")
        self.n_pages, self.max_seqs, self.max_pages = n_pages, max_seqs, max_pages
        self.free: List[int] = list(range(n_pages - 1, -1, -1))     # pop() gives page 0 first
        self.slots: List[Entry] = []

    @staticmethod
    def pages_for(rows: int) -> int:
        return -(-rows // PAGE)

    def fits(self, rows: Sequence[int]) -> bool:
        """Could requests needing these row counts all be admitted now?"""
        need = [self.pages_for(r) for r in rows]
        return (len(self.slots) + len(rows) <= self.max_seqs and
                all(n <= self.max_pages for n in need) and sum(need) <= len(self.free))

    def admit(self, rid: int, n_keep: int, max_new: int, alpha: float = 0.0,
              n_x: int = 0) -> int:
        """Reserve pages for n_keep + max_new rows and append a slot; returns it."""
        if n_keep < 1 or max_new < 0:
            raise ValueError("need n_keep >= 1 and max_new >= 0")
        if any(e.rid == rid for e in self.slots):
            raise ValueError(f"request {rid} is already running")
        n = self.pages_for(n_keep + max_new)
        if n > self.max_pages:
            raise ValueError(f"request {rid}: {n_keep + max_new} rows need {n} pages "
                             f"> max_pages {self.max_pages}")
        if len(self.slots) >= self.max_seqs:
            raise MemoryError("no free slot")
        if n > len(self.free):
            raise MemoryError(f"request {rid}: {n} pages needed, {len(self.free)} free")
        pages = [self.free.pop() for _ in range(n)]
        self.slots.append(Entry(rid, pages, n_keep, max_new, alpha, n_x))
        return len(self.slots) - 1

    def slot_of(self, rid: int) -> int:
        for s, e in enumerate(self.slots):
            if e.rid == rid:
                return s
        raise KeyError(rid)

    def retire(self, rid: int) -> Optional[int]:
        """Free the request's pages and fill its slot with the last request.
        Returns the slot the last request came from (None if nothing moved)."""
        s = self.slot_of(rid)
        self.free.extend(reversed(self.slots[s].pages))
        last = len(self.slots) - 1
        if s != last:
            self.slots[s] = self.slots[last]
        self.slots.pop()
        return last if s != last else None

    def advance(self) -> None:
        """One decode step appended a row to every running request."""
        for e in self.slots:
            if e.left <= 0:
                raise RuntimeError(f"request {e.rid} has no decode steps left")
        for e in self.slots:
            e.length += 1
            e.left -= 1

    def finished(self) -> List[int]:
        return [e.rid for e in self.slots if e.left == 0]

    def table_rows(self, lo: int = 0, hi: Optional[int] = None) -> np.ndarray:
        """Block-table rows of slots lo..hi-1; entries past a request's pages
        repeat its last page (never read: decode stays within the length)."""
        hi = len(self.slots) if hi is None else hi
        out = np.empty((hi - lo, self.max_pages), dtype=np.int32)
        for i, e in enumerate(self.slots[lo:hi]):
            out[i, :len(e.pages)] = e.pages
            out[i, len(e.pages):] = e.pages[-1]
        return out

    def lengths(self) -> np.ndarray:
        return np.array([e.length for e in self.slots], dtype=np.int32)


class Server:
    """Paged caches for n_layers layers, the batched evictor and the decode step.

    admit() takes each new request's per-layer prompt tensors; step() runs one
    decode step of every running request through all layers.
    """

    def __init__(self, n_layers: int, n_pages: int, max_seqs: int, max_pages: int, Hq: int,
                 Hkv: int, d: int, dtype: torch.dtype, w: int, pool: int, max_admit: int,
                 max_prompt: int, device="cuda"):
        self.n_layers, self.Hq, self.Hkv, self.d, self.dtype = n_layers, Hq, Hkv, d, dtype
        self.w, self.pool, self.max_admit, self.max_prompt = w, pool, max_admit, max_prompt
        self.slots = SlotTable(n_pages, max_seqs, max_pages)
        self.k_pool = torch.zeros((n_layers, n_pages, Hkv, PAGE, d), dtype=dtype, device=device)
        self.v_pool = torch.zeros((n_layers, n_pages, Hkv, d, PAGE), dtype=dtype, device=device)
        self.table = torch.zeros((max_seqs, max_pages), dtype=torch.int32, device=device)
        self.kv_len = torch.zeros((n_layers, max_seqs), dtype=torch.int32, device=device)
        # covers every batch size up to max_seqs
        dec = _lib.tb_workspace_bytes(_lib.TB_OP_DECODE, max_seqs, 0, Hq, Hkv, d, 0,
                                      max_pages * PAGE)
        self.dec_ws = torch.zeros((max(dec, 1),), dtype=torch.uint8, device=device)
        n = max_admit * Hkv * max_prompt
        self.scores_buf = torch.empty((n,), dtype=torch.float32, device=device)
        self.keep_buf = torch.empty((n,), dtype=torch.int32, device=device)
        sc = _lib.tb_workspace_bytes(_lib.TB_OP_SCORE, max_admit, max_prompt, Hq, Hkv, d, w, 0)
        self.score_ws = torch.empty((max(sc, 1),), dtype=torch.uint8, device=device)
        self.keep: Dict[int, List[torch.Tensor]] = {}       # rid -> per-layer keep_idx (kept on request)
        # static decode inputs / outputs for graph replay: row i = slot i
        self.q_in = torch.zeros((n_layers, max_seqs, Hq, d), dtype=dtype, device=device)
        self.k_in = torch.zeros((n_layers, max_seqs, Hkv, d), dtype=dtype, device=device)
        self.v_in = torch.zeros((n_layers, max_seqs, Hkv, d), dtype=dtype, device=device)
        self.o_out = torch.zeros((n_layers, max_seqs, Hq, d), dtype=dtype, device=device)
        self._graphs: Dict[int, torch.cuda.CUDAGraph] = {}

    @property
    def n_active(self) -> int:
        return len(self.slots.slots)

    def _upload(self, lo: int, hi: int, lengths: bool) -> None:
        if hi <= lo:
            return
        self.table[lo:hi].copy_(torch.from_numpy(self.slots.table_rows(lo, hi)))
        if lengths:
            ln = torch.from_numpy(self.slots.lengths()[lo:hi])
            self.kv_len[:, lo:hi].copy_(ln.unsqueeze(0).expand(self.n_layers, -1))

    def admit(self, rids: Sequence[int], L: Sequence[int], alphas: Sequence[float],
              max_new: Sequence[int], prompts: Sequence[dict], keep_sets: bool = False,
              stream=None) -> List[int]:
        """Evict and admit a batch of requests.

        prompts[l] holds layer l's q_win [b, Hq, w, d], k and v [b, Hkv, Lmax, d]
        (device, padded to Lmax = max(L)).  Every request keeps
        keep_count(L, alpha, w) rows (the same in every layer) and reserves
        pages for max_new more.  Returns n_keep per request.  keep_sets=True
        keeps each request's per-layer kept positions in self.keep.
        """
        b = len(rids)
        if not (b == len(L) == len(alphas) == len(max_new)) or b == 0:
            raise ValueError("rids, L, alphas and max_new must be non-empty and agree")
        if len(prompts) != self.n_layers:
            raise ValueError(f"need prompts for {self.n_layers} layers")
        if b > self.max_admit or max(L) > self.max_prompt:
            raise ValueError("admission batch exceeds max_admit or max_prompt")
        n_keep = [_lib.tb_keep_count(n, a, self.w) for n, a in zip(L, alphas)]
        if min(n_keep) < 1:
            raise ValueError("bad prompt length or ratio")
        if not self.slots.fits([k + m for k, m in zip(n_keep, max_new)]):
            raise MemoryError("not enough slots or pages for this batch")
        lo = self.n_active
        for i in range(b):
            self.slots.admit(rids[i], n_keep[i], max_new[i], alphas[i], L[i])
        self._upload(lo, lo + b, lengths=False)
        Lmax = prompts[0]["k"].shape[2]
        scores = self.scores_buf[: b * self.Hkv * Lmax].view(b, self.Hkv, Lmax)
        keep = self.keep_buf[: b * self.Hkv * Lmax].view(b, self.Hkv, Lmax)
        for layer, p in enumerate(prompts):
            _lib.tb_score_window(p["q_win"], p["k"], L, self.w, self.pool, scores, None,
                                 self.score_ws, stream)
            got = _lib.tb_select_topk(scores, L, self.w, alphas, keep, None, stream)
            if got != n_keep:
                raise RuntimeError(f"select kept {got}, expected {n_keep}")
            _lib.tb_compact_kv_paged(p["k"], p["v"], keep, n_keep, self.k_pool[layer],
                                     self.v_pool[layer], self.table[lo:lo + b],
                                     self.kv_len[layer, lo:lo + b], stream)
            if keep_sets:
                for i, r in enumerate(rids):
                    self.keep.setdefault(r, []).append(keep[i, :, : n_keep[i]].clone())
        return n_keep

    def step(self, q: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor,
             out: torch.Tensor, stream=None) -> None:
        """One decode step of the running batch: q, out [n_layers, n, Hq, d],
        k_new, v_new [n_layers, n, Hkv, d], row i = the request in slot i."""
        n = self.n_active
        if n == 0:
            raise RuntimeError("no running request")
        if q.shape[:2] != (self.n_layers, n) or k_new.shape[:2] != (self.n_layers, n):
            raise ValueError(f"inputs must be [{self.n_layers}, {n}, ...]")
        if any(e.left <= 0 for e in self.slots.slots):
            raise RuntimeError("retire finished requests before the next step")
        for layer in range(self.n_layers):
            _lib.tb_decode_attn_paged(q[layer], k_new[layer], v_new[layer], self.k_pool[layer],
                                      self.v_pool[layer], self.table, self.kv_len[layer],
                                      out[layer], self.dec_ws, stream)
        self.slots.advance()

    def step_graphed(self) -> None:
        """One decode step of the running batch from the static buffers: reads
        q_in / k_in / v_in[:, :n] and writes o_out[:, :n] (n = running
        requests).  The n_layers launches of a batch size are captured once in
        a graph and replayed on the current stream; the block table and the
        lengths are read from device memory at replay, so membership changes
        need no new capture."""
        n = self.n_active
        if n == 0:
            raise RuntimeError("no running request")
        if any(e.left <= 0 for e in self.slots.slots):
            raise RuntimeError("retire finished requests before the next step")
        g = self._graphs.get(n)
        if g is None:
            g = torch.cuda.CUDAGraph()
            cs = torch.cuda.Stream()
            cs.wait_stream(torch.cuda.current_stream())
            with torch.cuda.graph(g, stream=cs):
                for layer in range(self.n_layers):
                    _lib.tb_decode_attn_paged(self.q_in[layer, :n], self.k_in[layer, :n],
                                              self.v_in[layer, :n], self.k_pool[layer],
                                              self.v_pool[layer], self.table, self.kv_len[layer],
                                              self.o_out[layer, :n], self.dec_ws, cs)
            torch.cuda.current_stream().wait_stream(cs)
            self._graphs[n] = g
            # capture only records the launches: run this step now
        g.replay()
        self.slots.advance()

    def retire(self, rids: Sequence[int]) -> None:
        """Free finished requests; the last running requests move into their slots."""
        for r in rids:
            self.slots.retire(r)
            self.keep.pop(r, None)
        self._upload(0, self.n_active, lengths=True)

    def rids(self) -> List[int]:
        return [e.rid for e in self.slots.slots]
