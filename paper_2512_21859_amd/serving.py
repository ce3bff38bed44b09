"""Multi-request serving over paged KV caches.

Each request brings its own time budget, hence its own eviction ratio
(Sec. 5.2: alpha* is solved per request from its prompt length and predicted
response length).  Requests are admitted in batches: one batched eviction
(score -> select with per-request ratios -> compaction into pages), after
which they join the running batch, where every decode step serves all active
requests in one launch per layer.

Layout: every layer has its own page pools (k_pool and v_pool
[P, Hkv, 32, d]); one block table [max_seqs, max_pages] serves all layers, so
a request owns the same page numbers in every layer.  Each layer keeps its own
kv_len [max_seqs] because every decode call appends to it.  The active
requests occupy slots 0..n-1 of the table; a retiring request's slot is
refilled by moving the last one in (its table row and lengths), so a decode
step is always one dense batch.

Pages are reserved at admission for the retained prompt plus the request's
whole response (max_new tokens), so a running request never waits for pages
and nothing is preempted.

Requests can be admitted by time budget (Server.admit_budgets): the
controller gives each its ratio alpha* and pessimistic response length, as the
paper does for a single request.

Admission can also overlap decoding (Server.admit_async): the new batch's
eviction runs on a stream of its own into the top slots of the table, which
no decode step reads (a step reads slots 0..n-1 only), and the batch joins the
running one, at its end, once that eviction has finished (promote_ready).
The two streams touch disjoint table rows, lengths, pages and scratch buffers,
so a running request's step time is not held up by a whole admission.

The host holds the bookkeeping (which pages, which slot, how long); this
module allocates device buffers (torch) and sequences library calls; every
computation runs in the kernels.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from . import _lib
from .pipeline import TimeModel, plan_requests

PAGE = _lib.V_TILE          # rows per page: one 32-row tile of every KV head


class _Staging:
    """Pinned host buffers for asynchronous uploads of table rows and lengths.
    A buffer is refilled only after the copy that last read it has finished,
    so uploads never block on the stream they are queued on."""

    def __init__(self, n: int, nbytes: int):
        self.bufs = [torch.empty((nbytes,), dtype=torch.uint8, pin_memory=True) for _ in range(n)]
        self.done: List[Optional[torch.cuda.Event]] = [None] * n
        self.i = 0

    def put(self, dst: torch.Tensor, src: np.ndarray, stream) -> None:
        src = np.array(src, dtype=np.int32, order="C")          # an owned, writable copy
        i, self.i = self.i, (self.i + 1) % len(self.bufs)
        if self.done[i] is not None:
            self.done[i].synchronize()
        host = self.bufs[i][: src.nbytes].view(torch.int32).view(src.shape)
        host.copy_(torch.from_numpy(src))
        with torch.cuda.stream(stream):
            dst.copy_(host, non_blocking=True)
            ev = torch.cuda.Event()
            ev.record(stream)
        self.done[i] = ev


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
        # a batch admitted asynchronously: its eviction is still running, so it
        # holds the top slots [max_seqs - len(pending), max_seqs), which stay put
        self.pending: List[Entry] = []

    @staticmethod
    def pages_for(rows: int) -> int:
        return -(-rows // PAGE)

    def fits(self, rows: Sequence[int]) -> bool:
        """Could requests needing these row counts all be admitted now?"""
        need = [self.pages_for(r) for r in rows]
        return (len(self.slots) + len(self.pending) + len(rows) <= self.max_seqs and
                all(n <= self.max_pages for n in need) and sum(need) <= len(self.free))

    def _reserve(self, rid: int, n_keep: int, max_new: int, alpha: float, n_x: int) -> Entry:
        if n_keep < 1 or max_new < 0:
            raise ValueError("need n_keep >= 1 and max_new >= 0")
        if any(e.rid == rid for e in self.slots + self.pending):
            raise ValueError(f"request {rid} is already running")
        n = self.pages_for(n_keep + max_new)
        if n > self.max_pages:
            raise ValueError(f"request {rid}: {n_keep + max_new} rows need {n} pages "
                             f"> max_pages {self.max_pages}")
        if len(self.slots) + len(self.pending) >= self.max_seqs:
            raise MemoryError("no free slot")
        if n > len(self.free):
            raise MemoryError(f"request {rid}: {n} pages needed, {len(self.free)} free")
        return Entry(rid, [self.free.pop() for _ in range(n)], n_keep, max_new, alpha, n_x)

    def admit_pending(self, rids: Sequence[int], n_keep: Sequence[int], max_new: Sequence[int],
                      alphas: Sequence[float], n_x: Sequence[int]) -> int:
        """Reserve pages and the top slots for a batch whose eviction runs
        asynchronously; returns its first slot.  One pending batch at a time."""
        if self.pending:
            raise RuntimeError("an admitted batch is still pending")
        # checked whole first, so that a bad batch reserves nothing
        if not (len(rids) == len(n_keep) == len(max_new) == len(alphas) == len(n_x)) or not rids:
            raise ValueError("rids, n_keep, max_new, alphas and n_x must be non-empty and agree")
        running = {e.rid for e in self.slots}
        if len(set(rids)) != len(rids) or running & set(rids):
            raise ValueError("a request appears twice or is already running")
        if min(n_keep) < 1 or min(max_new) < 0:
            raise ValueError("need n_keep >= 1 and max_new >= 0")
        if any(self.pages_for(k + m) > self.max_pages for k, m in zip(n_keep, max_new)):
            raise ValueError(f"a request needs more than max_pages {self.max_pages} pages")
        if not self.fits([k + m for k, m in zip(n_keep, max_new)]):
            raise MemoryError("not enough slots or pages for this batch")
        for i, r in enumerate(rids):
            self.pending.append(self._reserve(r, n_keep[i], max_new[i], alphas[i], n_x[i]))
        return self.max_seqs - len(self.pending)

    def cancel_pending(self) -> None:
        """Drop the pending batch and free its pages."""
        for e in reversed(self.pending):
            self.free.extend(reversed(e.pages))
        self.pending = []

    def pending_rows(self) -> np.ndarray:
        """Block-table rows of the pending slots, in slot order."""
        return self._rows(self.pending)

    def promote(self) -> tuple:
        """The pending batch joins the running one at its end; returns the slot
        range [lo, hi) it now occupies."""
        lo = len(self.slots)
        self.slots.extend(self.pending)
        self.pending = []
        return lo, len(self.slots)

    def admit(self, rid: int, n_keep: int, max_new: int, alpha: float = 0.0,
              n_x: int = 0) -> int:
        """Reserve pages for n_keep + max_new rows and append a slot; returns it."""
        self.slots.append(self._reserve(rid, n_keep, max_new, alpha, n_x))
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
        return self._rows(self.slots[lo:hi])

    def _rows(self, entries: Sequence[Entry]) -> np.ndarray:
        out = np.empty((len(entries), self.max_pages), dtype=np.int32)
        for i, e in enumerate(entries):
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
        self.v_pool = torch.zeros((n_layers, n_pages, Hkv, PAGE, d), dtype=dtype, device=device)
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
        sel = _lib.tb_workspace_bytes(_lib.TB_OP_SELECT, max_admit, max_prompt, Hq, Hkv, d, w, 0)
        self.sel_ws = torch.empty((sel,), dtype=torch.uint8, device=device) if sel else None
        self.keep: Dict[int, List[torch.Tensor]] = {}       # rid -> per-layer keep_idx (kept on request)
        # static decode inputs / outputs for graph replay: row i = slot i
        self.q_in = torch.zeros((n_layers, max_seqs, Hq, d), dtype=dtype, device=device)
        self.k_in = torch.zeros((n_layers, max_seqs, Hkv, d), dtype=dtype, device=device)
        self.v_in = torch.zeros((n_layers, max_seqs, Hkv, d), dtype=dtype, device=device)
        self.o_out = torch.zeros((n_layers, max_seqs, Hq, d), dtype=dtype, device=device)
        self._graphs: Dict[int, torch.cuda.CUDAGraph] = {}
        self._staging = _Staging(8, 4 * max(n_layers, max_pages) * max_seqs)
        # Two streams taken together for overlapped admission: decode steps on
        # decode_stream, evictions on the admission stream.  Streams share a
        # few hardware queues, and two streams on one queue run one after the
        # other; streams taken one after the other from torch's pool sit on
        # different queues, where streams taken at unrelated times may not.
        self.decode_stream = torch.cuda.Stream(device=device)
        self._adm_stream = torch.cuda.Stream(device=device)
        self._adm_done: Optional[torch.cuda.Event] = None
        self._adm_refs: List[torch.Tensor] = []
        # every stream a decode step has been queued on: steps read the block
        # table and append into pages, so work that rewrites either waits for them
        self._step_streams: Dict[int, torch.cuda.Stream] = {}

    @property
    def n_active(self) -> int:
        return len(self.slots.slots)

    def _ordered(self, stream=None) -> torch.cuda.Stream:
        """The stream to queue server work on (decode_stream unless one is
        given), made to wait for the current stream (which may have produced
        the inputs) and for every stream a decode step was queued on (a
        queued step may still read the table rows or append into the pages
        this work rewrites)."""
        s = self.decode_stream if stream is None else stream
        for o in (torch.cuda.current_stream(), *self._step_streams.values()):
            if o.cuda_stream != s.cuda_stream:
                s.wait_stream(o)
        return s

    @staticmethod
    def _publish(s: torch.cuda.Stream) -> None:
        """Order the caller's current stream after the work just queued on s,
        so outputs, lengths and the table are read there in program order."""
        cur = torch.cuda.current_stream()
        if cur.cuda_stream != s.cuda_stream:
            cur.wait_stream(s)

    def _upload(self, lo: int, hi: int, lengths: bool, stream=None) -> None:
        """Table rows (and lengths, in every layer) of running slots lo..hi-1,
        queued on the stream without blocking the host."""
        if hi <= lo:
            return
        stream = self._ordered(stream)
        self._staging.put(self.table[lo:hi], self.slots.table_rows(lo, hi), stream)
        if lengths:
            ln = self.slots.lengths()[lo:hi]
            self._staging.put(self.kv_len[:, lo:hi],
                              np.broadcast_to(ln, (self.n_layers, hi - lo)), stream)

    def _check_admission(self, rids, L, alphas, max_new, prompts) -> List[int]:
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
        return n_keep

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
        if self.slots.pending:
            raise RuntimeError("an asynchronous admission is pending: promote it first")
        n_keep = self._check_admission(rids, L, alphas, max_new, prompts)
        stream = self._ordered(stream)
        lo = self.n_active
        for i in range(len(rids)):
            self.slots.admit(rids[i], n_keep[i], max_new[i], alphas[i], L[i])
        self._upload(lo, lo + len(rids), lengths=False, stream=stream)
        self._evict(rids, L, alphas, n_keep, prompts, lo, keep_sets, stream)
        self._publish(stream)
        return n_keep

    def admit_async(self, rids: Sequence[int], L: Sequence[int], alphas: Sequence[float],
                    max_new: Sequence[int], prompts: Sequence[dict],
                    keep_sets: bool = False) -> List[int]:
        """admit(), with the eviction on a separate stream so that decode steps
        queued meanwhile run alongside it (queue them on decode_stream: a
        stream created at another time may share the admission stream's
        hardware queue and then runs after it).  The eviction starts after the work
        already queued on the current stream (which may have produced the
        prompts) and after every decode step queued so far, on whatever stream
        (a queued step may still read pages freed by a retirement).  The new requests
        hold the top slots of the table until promote_ready() moves them into
        the running batch (their kept sets, with keep_sets, are complete by
        then); only one such batch may be pending.  If queueing the eviction
        fails, the batch is dropped and its pages freed."""
        if self.slots.pending:
            raise RuntimeError("an asynchronous admission is already pending")
        n_keep = self._check_admission(rids, L, alphas, max_new, prompts)
        top = self.slots.admit_pending(rids, n_keep, max_new, alphas, L)
        adm = self._adm_stream
        cur = torch.cuda.current_stream()
        for o in (cur, self.decode_stream, *self._step_streams.values()):
            adm.wait_stream(o)
        try:
            self._staging.put(self.table[top:top + len(rids)], self.slots.pending_rows(), adm)
            self._adm_refs = [x for p in prompts for x in p.values()]
            for x in self._adm_refs:        # the allocator must not reuse them before adm is done
                x.record_stream(adm)
            self._evict(rids, L, alphas, n_keep, prompts, top, keep_sets, adm)
            self._adm_done = torch.cuda.Event()
            self._adm_done.record(adm)
        except BaseException:
            # whatever was queued may still write the batch's pages: later work
            # on the current stream waits for it before the pages are reused
            cur.wait_stream(adm)
            for r in rids:
                self.keep.pop(r, None)
            self.slots.cancel_pending()
            self._adm_refs = []
            raise
        return n_keep

    def promote_ready(self, wait: bool = False, stream=None) -> int:
        """If the pending batch's eviction has finished (or wait=True), move it
        into slots n..n+b-1 of the running batch and return b; else return 0.
        The table rows and lengths are uploaded on the given (decode) stream,
        which also waits for the eviction."""
        if not self.slots.pending:
            return 0
        if not (wait or self._adm_done.query()):
            return 0
        stream = self._ordered(stream)
        stream.wait_event(self._adm_done)
        lo, hi = self.slots.promote()
        self._upload(lo, hi, lengths=True, stream=stream)
        self._publish(stream)
        self._adm_refs = []
        return hi - lo

    def admit_budgets(self, rids: Sequence[int], L: Sequence[int], budgets: Sequence[float],
                      n_hat: Sequence[int], model: TimeModel, prompts: Sequence[dict],
                      keep_sets: bool = False, overlap: bool = False):
        """Admit requests by time budget (Sec. 5.2, applied per request): each
        gets the smallest ratio alpha* whose worst-case time (prefill, then
        N_hat_W decode steps over the retained KV) fits its budget, and pages
        for N_hat_W new tokens (the pessimistic response length from its
        predicted bucket n_hat).  overlap=True admits through admit_async.
        Returns [(alpha, feasible, N_hat_W)] per request."""
        plan = plan_requests(model, L, budgets, n_hat)
        alphas = [a for a, _, _ in plan]
        max_new = [w for _, _, w in plan]
        if overlap:
            self.admit_async(rids, L, alphas, max_new, prompts, keep_sets=keep_sets)
        else:
            self.admit(rids, L, alphas, max_new, prompts, keep_sets=keep_sets)
        return plan

    def _evict(self, rids, L, alphas, n_keep, prompts, lo, keep_sets, stream) -> None:
        """Score, select and compact every layer of the requests in slots
        lo..lo+b-1, whose table rows are already on the device; everything,
        the copies of the kept sets included, is queued on `stream`."""
        with torch.cuda.stream(stream):
            self._evict_layers(rids, L, alphas, n_keep, prompts, lo, keep_sets, stream)

    def _evict_layers(self, rids, L, alphas, n_keep, prompts, lo, keep_sets, stream) -> None:
        b = len(rids)
        Lmax = prompts[0]["k"].shape[2]
        scores = self.scores_buf[: b * self.Hkv * Lmax].view(b, self.Hkv, Lmax)
        keep = self.keep_buf[: b * self.Hkv * Lmax].view(b, self.Hkv, Lmax)
        for layer, p in enumerate(prompts):
            _lib.tb_score_window(p["q_win"], p["k"], L, self.w, self.pool, scores, None,
                                 self.score_ws, stream)
            got = _lib.tb_select_topk(scores, L, self.w, alphas, keep, self.sel_ws, stream)
            if got != n_keep:
                raise RuntimeError(f"select kept {got}, expected {n_keep}")
            _lib.tb_compact_kv_paged(p["k"], p["v"], keep, n_keep, self.k_pool[layer],
                                     self.v_pool[layer], self.table[lo:lo + b],
                                     self.kv_len[layer, lo:lo + b], stream)
            if keep_sets:
                for i, r in enumerate(rids):
                    self.keep.setdefault(r, []).append(keep[i, :, : n_keep[i]].clone())

    def step(self, q: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor,
             out: torch.Tensor, stream=None) -> None:
        """One decode step of the running batch: q, out [n_layers, n, Hq, d],
        k_new, v_new [n_layers, n, Hkv, d], row i = the request in slot i.
        Queued on decode_stream unless a stream is given; either way after the
        current stream's work and after every earlier step, and the current
        stream is ordered after it (out can be read there)."""
        n = self.n_active
        if n == 0:
            raise RuntimeError("no running request")
        if any(x.shape[:2] != (self.n_layers, n) for x in (q, k_new, v_new, out)):
            raise ValueError(f"q, k_new, v_new and out must be [{self.n_layers}, {n}, ...]")
        if any(e.left <= 0 for e in self.slots.slots):
            raise RuntimeError("retire finished requests before the next step")
        s = self._ordered(stream)
        self._step_streams[s.cuda_stream] = s
        if s.cuda_stream != torch.cuda.current_stream().cuda_stream:
            for x in (q, k_new, v_new, out):    # not reused before the step has run
                x.record_stream(s)
        for layer in range(self.n_layers):
            _lib.tb_decode_attn_paged(q[layer], k_new[layer], v_new[layer], self.k_pool[layer],
                                      self.v_pool[layer], self.table, self.kv_len[layer],
                                      out[layer], self.dec_ws, s)
        self._publish(s)
        self.slots.advance()

    def capture(self, n: int) -> torch.cuda.CUDAGraph:
        """The graph of one decode step at batch size n (captured once, on a
        side stream; capture records the launches and runs nothing)."""
        if not 1 <= n <= self.slots.max_seqs:
            raise ValueError(f"batch size {n} outside 1..{self.slots.max_seqs}")
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
        return g

    def step_graphed(self, stream=None) -> None:
        """One decode step of the running batch from the static buffers: reads
        q_in / k_in / v_in[:, :n] and writes o_out[:, :n] (n = running
        requests).  The n_layers launches of a batch size are captured once in
        a graph and replayed on decode_stream (or the given stream); the block
        table and the lengths are read from device memory at replay, so
        membership changes need no new capture."""
        n = self.n_active
        if n == 0:
            raise RuntimeError("no running request")
        if any(e.left <= 0 for e in self.slots.slots):
            raise RuntimeError("retire finished requests before the next step")
        g = self.capture(n)
        s = self._ordered(stream)
        self._step_streams[s.cuda_stream] = s
        with torch.cuda.stream(s):
            g.replay()
        self._publish(s)
        self.slots.advance()

    def retire(self, rids: Sequence[int], stream=None) -> None:
        """Free finished requests; the last running requests move into their
        slots (table rows and lengths re-uploaded on decode_stream, or the
        given stream, after every queued step)."""
        for r in rids:
            self.slots.retire(r)
            self.keep.pop(r, None)
        s = self._ordered(stream)
        self._upload(0, self.n_active, lengths=True, stream=s)
        self._publish(s)

    def rids(self) -> List[int]:
        return [e.rid for e in self.slots.slots]
