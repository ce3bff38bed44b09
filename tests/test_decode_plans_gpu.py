"""Single-sequence decode at cache sizes chosen to hit every launch shape of
the split (one-, two-, four- and eight-wave partial blocks over an even share
of the tiles, and the small-cache split with at most 32 partials merged by
one wave per query head), checked against the float64 oracle at both head
dimensions."""
import numpy as np
import pytest
import torch

from oracle import timebill_oracle as O
from paper_2512_21859_amd import _lib
from tests.parity_util import DECODE_TOL, f64

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU in this container")
    _lib.load()
    torch.cuda.init()


# capacities (rows) and the block shape the plan gives 4 KV heads at each:
# one block per CU (64 per KV head), the cap/32 tiles split evenly, one wave
# per tile up to 8
CAPS = [672,      # <= 2048 rows: 21 one-tile blocks per KV head, <= 32 partials
        2304,     # 72 tiles: 64 blocks of 1-2 tiles (past the 32-partial cap)
        2816,     # 64 blocks of 1-2 tiles, one wave
        4352,     # two-wave blocks of 2-3 tiles
        8448,     # four-wave blocks of 4-5 tiles
        24640,    # eight-wave blocks of 12-13 tiles (a wave takes 1-2)
        33024]    # eight-wave blocks of 16-17 tiles (a wave takes 2-3)


@pytest.mark.parametrize("d", [128, 64])
@pytest.mark.parametrize("cap", CAPS)
def test_single_sequence_plans(cap, d):
    print(f"\n[case] decode plan cap={cap} d={d}", flush=True)
    B, Hkv, G, T = 1, 4, 7, 3
    Hq = G * Hkv
    n0 = cap - 40                          # ragged tail: the last partial is part-empty
    gen = torch.Generator().manual_seed(cap + d)
    kc = torch.randn((B, Hkv, cap, d), generator=gen).to(torch.bfloat16)
    vc = torch.randn((B, Hkv, cap, d), generator=gen).to(torch.bfloat16)
    q = torch.randn((T, B, Hq, d), generator=gen).to(torch.bfloat16)
    kn = torch.randn((T, B, Hkv, d), generator=gen).to(torch.bfloat16)
    vn = torch.randn((T, B, Hkv, d), generator=gen).to(torch.bfloat16)
    cache = _lib.KVCache(B, Hq, Hkv, cap, d, torch.bfloat16)
    cache.k.copy_(kc)
    cache.v.copy_(vc)
    cache.kv_len.fill_(n0)
    cache.host_len = [n0]
    out = torch.empty((T, B, Hq, d), dtype=torch.bfloat16, device=DEV)
    qd, knd, vnd = q.to(DEV), kn.to(DEV), vn.to(DEV)
    for t in range(T):
        cache.decode(qd[t], knd[t], vnd[t], out[t])
    torch.cuda.synchronize()
    assert cache.kv_len.cpu().tolist() == [n0 + T]
    got, kc64, vc64, kn64, vn64, q64 = f64(out), f64(kc), f64(vc), f64(kn), f64(vn), f64(q)
    for g in range(Hkv):
        for t in range(T):
            rk = np.concatenate([kc64[0, g, :n0], kn64[: t + 1, 0, g]])
            rv = np.concatenate([vc64[0, g, :n0], vn64[: t + 1, 0, g]])
            ref = O.decode_step(q64[t, 0, g * G:(g + 1) * G], rk, rv)
            err = np.abs(got[t, 0, g * G:(g + 1) * G] - ref).max()
            assert err <= DECODE_TOL[torch.bfloat16], f"g={g} t={t}: max abs err {err}"


@pytest.mark.parametrize("d", [128, 64])
@pytest.mark.parametrize("Hkv,cap", [(1, 20000),    # 256 blocks of one KV head: 256 partials, two merge rounds
                                     (2, 12032)])   # 128 partials per KV head, one round of 16 per lane
def test_many_partial_plans(Hkv, cap, d):
    print(f"\n[case] decode many partials Hkv={Hkv} cap={cap} d={d}", flush=True)
    B, G, T = 1, 8, 2
    Hq = G * Hkv
    n0 = cap - 29
    gen = torch.Generator().manual_seed(7 * cap + d + Hkv)
    kc = torch.randn((B, Hkv, cap, d), generator=gen).to(torch.bfloat16)
    vc = torch.randn((B, Hkv, cap, d), generator=gen).to(torch.bfloat16)
    q = torch.randn((T, B, Hq, d), generator=gen).to(torch.bfloat16)
    kn = torch.randn((T, B, Hkv, d), generator=gen).to(torch.bfloat16)
    vn = torch.randn((T, B, Hkv, d), generator=gen).to(torch.bfloat16)
    cache = _lib.KVCache(B, Hq, Hkv, cap, d, torch.bfloat16)
    cache.k.copy_(kc)
    cache.v.copy_(vc)
    cache.kv_len.fill_(n0)
    cache.host_len = [n0]
    out = torch.empty((T, B, Hq, d), dtype=torch.bfloat16, device=DEV)
    qd, knd, vnd = q.to(DEV), kn.to(DEV), vn.to(DEV)
    for t in range(T):
        cache.decode(qd[t], knd[t], vnd[t], out[t])
    torch.cuda.synchronize()
    assert cache.kv_len.cpu().tolist() == [n0 + T]
    got, kc64, vc64, kn64, vn64, q64 = f64(out), f64(kc), f64(vc), f64(kn), f64(vn), f64(q)
    for g in range(Hkv):
        for t in range(T):
            rk = np.concatenate([kc64[0, g, :n0], kn64[: t + 1, 0, g]])
            rv = np.concatenate([vc64[0, g, :n0], vn64[: t + 1, 0, g]])
            ref = O.decode_step(q64[t, 0, g * G:(g + 1) * G], rk, rv)
            err = np.abs(got[t, 0, g * G:(g + 1) * G] - ref).max()
            assert err <= DECODE_TOL[torch.bfloat16], f"g={g} t={t}: max abs err {err}"
