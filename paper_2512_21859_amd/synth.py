"""Seeded synthetic inputs for the eviction + decode path.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic, so both the HIP path and the float64 checker can be fed
from it.  All randomness comes from ``torch.Generator('cpu')`` (fp32 normal
draws), rounded once to the workload dtype, so every consumer sees identical
values.

Seeds: 1_000_000 * workload_id + 1000 * layer + stream, with stream 0 for
K, V and window queries, 1 for heavy-hitter positions and directions, 2 for
decode-step q / k / v, 3 for per-sequence lengths and eviction ratios and 4
for the queries at every prompt position (used by the accumulated-attention
scorer).

The workloads stand in for the paper's LongBench prompts on Qwen2.5-7B-Instruct
(context up to 32768 tokens, Sec. 6.1): head shapes 28 query / 4 KV heads of
dimension 128, lengths up to the paper's context and beyond, and a small set of
"heavy hitter" keys so that the scores have the skewed shape real attention
has.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Optional, Sequence

import torch


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: shapes, window, pool, ratios, decode steps."""

    wid: int
    name: str
    dtype: torch.dtype
    B: int
    L: Optional[int]           # fixed prompt length (None: drawn per sequence)
    Hq: int
    Hkv: int
    d: int
    w: int
    pool: int
    alphas: Sequence[float]    # eviction ratios swept (per-seq ratios drawn if empty)
    T: int                     # decode steps
    layers: int = 1
    heavy: str = "none"        # "none" | "bias" | "aligned"
    heavy_frac: float = 0.0
    L_range: Optional[tuple] = None
    alpha_range: Optional[tuple] = None

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv


WORKLOADS = {
    1: Workload(1, "tiny-fp32-L512", torch.float32, 1, 512, 2, 1, 64, 16, 5,
                (0.5,), 32),
    2: Workload(2, "bf16-L8192-28q4kv", torch.bfloat16, 1, 8192, 28, 4, 128, 32, 7,
                (0.0, 0.25, 0.5, 0.75, 0.95), 256, heavy="bias", heavy_frac=0.02),
    3: Workload(3, "bf16-28layer-L32768-28q4kv", torch.bfloat16, 1, 32768, 28, 4, 128,
                32, 7, tuple(k / 20 for k in range(20)), 128, layers=28,
                heavy="bias", heavy_frac=0.02),
    4: Workload(4, "bf16-ragged16-28q4kv", torch.bfloat16, 16, None, 28, 4, 128, 32, 7,
                (), 256, heavy="bias", heavy_frac=0.02,
                L_range=(1024, 16384), alpha_range=(0.0, 0.9)),
    5: Workload(5, "bf16-L131072-32q8kv", torch.bfloat16, 1, 131072, 32, 8, 128, 64, 7,
                (0.5, 0.9, 0.98), 512, heavy="aligned", heavy_frac=0.01),
}


def seed_of(wid: int, layer: int, stream: int) -> int:
    return 1_000_000 * wid + 1000 * layer + stream


def _gen(seed: int) -> torch.Generator:
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    return g


def lengths_and_alphas(wl: Workload):
    """Per-sequence prompt lengths and eviction ratios (stream 3)."""
    if wl.L is not None:
        return [wl.L] * wl.B, None
    g = _gen(seed_of(wl.wid, 0, 3))
    lo, hi = wl.L_range
    L = torch.randint(lo, hi + 1, (wl.B,), generator=g).tolist()
    alo, ahi = wl.alpha_range
    a = (alo + (ahi - alo) * torch.rand(wl.B, generator=g, dtype=torch.float64)).tolist()
    return L, a


def make_prompt(wl: Workload, layer: int = 0, L: Optional[List[int]] = None,
                pad_value: float = 0.0):
    """Window queries and prompt K/V of one layer.

    Returns dict(q_win [B,Hq,w,d], k [B,Hkv,Lmax,d], v [B,Hkv,Lmax,d], L list,
    heavy), CPU tensors in the workload dtype; heavy[b][g] lists the planted
    heavy-hitter positions (empty without structure).  Rows j >= L[b] hold
    ``pad_value``.
    """
    if L is None:
        L, _ = lengths_and_alphas(wl)
    Lmax = max(L)
    B, Hq, Hkv, d, w = wl.B, wl.Hq, wl.Hkv, wl.d, wl.w
    g0 = _gen(seed_of(wl.wid, layer, 0))
    g1 = _gen(seed_of(wl.wid, layer, 1))
    k = torch.full((B, Hkv, Lmax, d), pad_value, dtype=torch.float32)
    v = torch.full((B, Hkv, Lmax, d), pad_value, dtype=torch.float32)
    q_win = torch.empty((B, Hq, w, d), dtype=torch.float32)
    heavy = [[[] for _ in range(Hkv)] for _ in range(B)]
    for b in range(B):
        n = L[b]
        k[b, :, :n] = torch.randn((Hkv, n, d), generator=g0)
        v[b, :, :n] = torch.randn((Hkv, n, d), generator=g0)
        q_win[b] = torch.randn((Hq, w, d), generator=g0)
        n_heavy = math.ceil(wl.heavy_frac * (n - w)) if wl.heavy != "none" else 0
        if n_heavy == 0:
            continue
        if wl.heavy == "bias":
            # a random unit direction per KV head, added with weight 2 sqrt(d)
            for gk in range(Hkv):
                u = torch.randn(d, generator=g1)
                u = u / u.norm()
                pos = torch.randperm(n - w, generator=g1)[:n_heavy]
                k[b, gk, pos] += (2.0 * math.sqrt(d)) * u
                heavy[b][gk] = sorted(pos.tolist())
        elif wl.heavy == "aligned":
            # keys replaced by 4 sqrt(d) times the unit mean of the group's window queries
            qr = q_win[b].to(wl.dtype).to(torch.float32)
            G = Hq // Hkv
            for gk in range(Hkv):
                c = qr[gk * G:(gk + 1) * G].reshape(G * w, d).mean(dim=0)
                u = c / c.norm()
                pos = torch.randperm(n - w, generator=g1)[:n_heavy]
                k[b, gk, pos] = (4.0 * math.sqrt(d)) * u
                heavy[b][gk] = sorted(pos.tolist())
    return {"q_win": q_win.to(wl.dtype), "k": k.to(wl.dtype), "v": v.to(wl.dtype),
            "L": list(L), "heavy": heavy}


def make_queries(wl: Workload, layer: int = 0, L: Optional[List[int]] = None):
    """Queries at every prompt position: [B, Hq, Lmax, d] in the workload dtype,
    N(0,1) (stream 4); rows j >= L[b] are zero."""
    if L is None:
        L, _ = lengths_and_alphas(wl)
    g4 = _gen(seed_of(wl.wid, layer, 4))
    q = torch.zeros((wl.B, wl.Hq, max(L), wl.d), dtype=torch.float32)
    for b in range(wl.B):
        q[b, :, : L[b]] = torch.randn((wl.Hq, L[b], wl.d), generator=g4)
    return q.to(wl.dtype)


def make_decode(wl: Workload, layer: int = 0, T: Optional[int] = None):
    """Per-step decode inputs: q [T,B,Hq,d], k_new and v_new [T,B,Hkv,d]."""
    T = wl.T if T is None else T
    g2 = _gen(seed_of(wl.wid, layer, 2))
    q = torch.randn((T, wl.B, wl.Hq, wl.d), generator=g2)
    kn = torch.randn((T, wl.B, wl.Hkv, wl.d), generator=g2)
    vn = torch.randn((T, wl.B, wl.Hkv, wl.d), generator=g2)
    return {"q": q.to(wl.dtype), "k_new": kn.to(wl.dtype), "v_new": vn.to(wl.dtype)}


def custom(wid: int, dtype: torch.dtype, B: int, L: Sequence[int], Hq: int, Hkv: int,
           d: int, w: int, pool: int, T: int, heavy: str = "bias",
           heavy_frac: float = 0.02) -> Workload:
    """A small workload of arbitrary shape for parity cases (seeded by ``wid``)."""
    Ls = list(L)
    wl = Workload(wid, f"custom{wid}", dtype, B, None, Hq, Hkv, d, w, pool, (), T,
                  heavy=heavy, heavy_frac=heavy_frac,
                  L_range=(min(Ls), max(Ls)), alpha_range=(0.0, 0.9))
    return wl
