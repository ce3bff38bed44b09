"""GPU parity: the HIP path through the C ABI against the float64 oracle.

Every case prints its name before touching the GPU.  Inputs come from the
seeded generators; expected values come only from the oracle.
"""
import math

import numpy as np
import pytest
import torch

from oracle import timebill_oracle as O
from paper_2512_21859_amd import _lib, synth
from paper_2512_21859_amd.pipeline import Evictor, run_decode
from tests.parity_util import DECODE_TOL, check_keep, f64, score_rel_err, score_rel_err_p99

pytestmark = pytest.mark.gpu
DEV = "cuda"
SCORE_REL_TOL = 5e-7


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU in this container")
    _lib.load()          # raises if the library was not built
    torch.cuda.init()


def case(msg):
    print(f"\n[case] {msg}", flush=True)


# ------------------------------------------------------------------ decode only
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("G", [1, 2, 3, 4, 7, 8])
@pytest.mark.parametrize("cap,lens", [(704, [1, 523]), (20000, [19990, 4097])])
def test_decode_only(dtype, d, G, cap, lens):
    case(f"decode_only dtype={dtype} d={d} G={G} cap={cap} lens={lens}")
    B, Hkv, T = 2, 2, 3
    Hq = G * Hkv
    g = torch.Generator().manual_seed(1234 + G + d + cap)
    kc = torch.randn((B, Hkv, cap, d), generator=g).to(dtype)
    vc = torch.randn((B, Hkv, cap, d), generator=g).to(dtype)
    q = torch.randn((T + 1, B, Hq, d), generator=g).to(dtype)
    kn = torch.randn((T, B, Hkv, d), generator=g).to(dtype)
    vn = torch.randn((T, B, Hkv, d), generator=g).to(dtype)
    cache = _lib.KVCache(B, Hq, Hkv, cap, d, dtype)
    cache.k.copy_(kc)
    cache.v.copy_(vc)
    cache.kv_len.copy_(torch.tensor(lens, dtype=torch.int32))
    cache.host_len = list(lens)
    qd, knd, vnd = q.to(DEV), kn.to(DEV), vn.to(DEV)
    out = torch.empty((T + 1, B, Hq, d), dtype=dtype, device=DEV)
    for t in range(T):
        cache.decode(qd[t], knd[t], vnd[t], out[t])
    cache.decode(qd[T], None, None, out[T])            # no append
    torch.cuda.synchronize()
    assert cache.kv_len.cpu().tolist() == [n + T for n in lens]
    got = f64(out)
    tol = DECODE_TOL[dtype]
    kc64, vc64, kn64, vn64, q64 = f64(kc), f64(vc), f64(kn), f64(vn), f64(q)
    for b in range(B):
        for gg in range(Hkv):
            for t in range(T + 1):
                n = lens[b] + min(t + 1, T)
                rows_k = np.concatenate([kc64[b, gg, :lens[b]], kn64[:min(t + 1, T), b, gg]])
                rows_v = np.concatenate([vc64[b, gg, :lens[b]], vn64[:min(t + 1, T), b, gg]])
                assert rows_k.shape[0] == n
                ref = O.decode_step(q64[t, b, gg * G:(gg + 1) * G], rows_k, rows_v)
                err = np.abs(got[t, b, gg * G:(gg + 1) * G] - ref).max()
                assert err <= tol, f"b={b} g={gg} t={t}: max abs err {err}"
    # the appended rows landed in the caches
    v_rows = cache.v.cpu()
    for t in range(T):
        for b in range(B):
            assert torch.equal(cache.k[b, :, lens[b] + t].cpu(), kn[t, b])
            assert torch.equal(v_rows[b, :, lens[b] + t], vn[t, b])


# ------------------------------------------------------------------ compaction
@pytest.mark.parametrize("dtype,d", [(torch.bfloat16, 128), (torch.bfloat16, 64),
                                     (torch.float32, 64), (torch.float32, 128)])
def test_compact_exact(dtype, d):
    case(f"compact dtype={dtype} d={d}")
    B, Hkv, Lmax = 3, 2, 1000
    g = torch.Generator().manual_seed(99 + d)
    k = torch.randn((B, Hkv, Lmax, d), generator=g).to(dtype)
    v = torch.randn((B, Hkv, Lmax, d), generator=g).to(dtype)
    n_keep = [1, 517, 1000]
    cap = 1120
    keep = torch.zeros((B, Hkv, Lmax), dtype=torch.int32)
    for b in range(B):
        for gg in range(Hkv):
            sel = torch.sort(torch.randperm(Lmax, generator=g)[: n_keep[b]]).values
            keep[b, gg, : n_keep[b]] = sel.to(torch.int32)
    kd, vd = k.to(DEV), v.to(DEV)
    kc = torch.full((B, Hkv, cap, d), 3.0, dtype=dtype, device=DEV)
    vc = torch.full((B, Hkv, cap, d), 3.0, dtype=dtype, device=DEV)
    kv_len = torch.zeros((B,), dtype=torch.int32, device=DEV)
    _lib.tb_compact_kv(kd, vd, keep.to(DEV), n_keep, kc, vc, kv_len)
    torch.cuda.synchronize()
    assert kv_len.cpu().tolist() == n_keep
    k_rows, v_rows = kc.cpu(), vc.cpu()
    for b in range(B):
        for gg in range(Hkv):
            n = n_keep[b]
            idx = keep[b, gg, :n].long()
            assert torch.equal(k_rows[b, gg, :n], k[b, gg, idx])
            assert torch.equal(v_rows[b, gg, :n], v[b, gg, idx])
            # rows past n_keep are not written
            assert bool((k_rows[b, gg, n:] == 3.0).all())
            assert bool((v_rows[b, gg, n:] == 3.0).all())


# ------------------------------------------------------------------ selection
def _select_case(pooled64: np.ndarray, L, w, alphas, where):
    """pooled64 [B, Hkv, Lmax] float64 (prefix entries valid); GPU selects on fp32.
    Where some prefix is long enough, the several-blocks-per-head path (given a
    workspace) is run as well; both must give the oracle's keep_idx and leave
    the entries past n_keep untouched."""
    B, Hkv, Lmax = pooled64.shape
    p32 = torch.from_numpy(pooled64).to(torch.float32)
    p32_64 = p32.to(torch.float64).numpy()
    ref = {}
    for b in range(B):
        nk = O.keep_count(L[b], alphas[b], w)
        for gg in range(Hkv):
            ref[b, gg] = O.select_keep(p32_64[b, gg, : L[b] - w], L[b], w, nk)
    nbytes = _lib.tb_workspace_bytes(_lib.TB_OP_SELECT, B, Lmax, 0, Hkv, 0, w, 0)
    multi = nbytes > 0 and max(L) - w > 32768
    for ws in ([None, torch.full((nbytes,), 0xA5, dtype=torch.uint8, device=DEV)]
               if multi else [None]):
        keep = torch.full((B, Hkv, Lmax), -1, dtype=torch.int32, device=DEV)
        n_keep = _lib.tb_select_topk(p32.to(DEV), L, w, alphas, keep, ws)
        torch.cuda.synchronize()
        kk = keep.cpu().numpy()
        path = "one block per head" if ws is None else "several blocks per head"
        for b in range(B):
            assert n_keep[b] == O.keep_count(L[b], alphas[b], w)
            for gg in range(Hkv):
                assert np.array_equal(kk[b, gg, : n_keep[b]], ref[b, gg]), \
                    f"{where} b={b} g={gg} ({path})"
                assert (kk[b, gg, n_keep[b]:] == -1).all(), f"{where} b={b} g={gg}: wrote past n_keep"


def test_select_exact_on_oracle_scores():
    case("select on oracle pooled scores (fp32), ties by position")
    wl = synth.custom(901, torch.bfloat16, 3, [300, 4099, 9000], 8, 2, 64, 8, 7, 1)
    pr = synth.make_prompt(wl, L=[300, 4099, 9000])
    L, w = pr["L"], wl.w
    Lmax = max(L)
    pooled = np.zeros((wl.B, wl.Hkv, Lmax))
    for b in range(wl.B):
        raw = O.window_scores(f64(pr["q_win"][b]), f64(pr["k"][b]), L[b], w)
        pooled[b, :, : L[b] - w] = O.max_pool(raw, 7)
    for alphas in ([0.0, 0.0, 0.0], [0.3, 0.5, 0.7], [0.99, 0.95, 0.9], [0.1, 0.05, 0.995]):
        _select_case(pooled, L, w, alphas, f"alphas={alphas}")


@pytest.mark.parametrize("levels", [1, 2, 3, 17])
def test_select_exact_plateaus(levels):
    case(f"select with heavy ties, {levels} distinct levels")
    rng = np.random.default_rng(levels)
    B, Hkv, w = 2, 3, 4
    L = [5, 20000]
    pooled = np.zeros((B, Hkv, max(L)))
    for b in range(B):
        pooled[b, :, : L[b] - w] = rng.integers(0, levels, (Hkv, L[b] - w)) / 8.0 + 0.5
    for alphas in ([0.0, 0.1], [0.2, 0.5], [0.5, 0.999], [0.79, 0.25]):
        _select_case(pooled, L, w, alphas, f"levels={levels} alphas={alphas}")


def test_select_exact_long_prefix_and_wide_range():
    case("select beyond the LDS-cached prefix length, keys over the whole float range")
    rng = np.random.default_rng(77)
    B, Hkv, w = 2, 2, 32
    L = [40000, 33000]            # prefixes 39968 and 32968 (> 32768: read from L2 per pass)
    pooled = np.zeros((B, Hkv, max(L)))
    for b in range(B):
        n = L[b] - w
        x = 10.0 ** rng.uniform(-44, 3, (Hkv, n))          # includes fp32 subnormals
        x[:, rng.integers(0, n, n // 50)] = 0.0             # exact zeros
        x[:, 1000:1100] = x[:, 1000:1001]                   # a long plateau
        pooled[b, :, :n] = x
    for alphas in ([0.0, 0.3], [0.5, 0.9], [0.999, 0.01]):
        _select_case(pooled, L, w, alphas, f"alphas={alphas}")


def _pooled_heavy_tail(rng, n_rows, n, pool=7):
    """Window-score-like prefixes: heavy-tailed attention mass, max-pooled."""
    a = np.exp(3.0 * rng.standard_normal((n_rows, n)))
    a[:, rng.integers(0, n, max(1, n // 500))] *= 100.0
    a = a / a.sum(axis=1, keepdims=True) * 224.0
    out = a.copy()
    for s in range(1, pool // 2 + 1):
        out[:, s:] = np.maximum(out[:, s:], a[:, :-s])
        out[:, :-s] = np.maximum(out[:, :-s], a[:, s:])
    return out


@pytest.mark.parametrize("kind", ["window", "knorm", "levels3"])
def test_select_several_blocks_per_head(kind):
    """Long prefixes split over several blocks per KV head: a ragged batch in
    which a short sequence and one just past the split threshold ride along
    with a 131072-position one (the split applies above 32768 prefix
    positions; shorter prefixes of the batch take it too); ratios from none evicted (every prefix
    position kept) to a single selected position."""
    case(f"select, several blocks per head, {kind} scores")
    rng = np.random.default_rng({"window": 1, "knorm": 2, "levels3": 3}[kind])
    B, Hkv, w = 3, 2, 32
    L = [131072, 32768 + w + 1, 5000]
    pooled = np.zeros((B, Hkv, max(L)))
    for b in range(B):
        n = L[b] - w
        if kind == "window":
            pooled[b, :, :n] = _pooled_heavy_tail(rng, Hkv, n)
        elif kind == "knorm":        # negated key norms
            pooled[b, :, :n] = -np.sqrt(rng.chisquare(128, (Hkv, n)))
        else:
            pooled[b, :, :n] = rng.integers(0, 3, (Hkv, n)) / 4.0
    for alphas in ([0.5, 0.5, 0.5], [0.0, 0.9, 0.3], [0.95, 0.0, 0.999],
                   [1.0 - (w + 1) / L[0] + 1e-12, 0.25, 0.75]):   # first: n_keep = w + 1
        _select_case(pooled, L, w, alphas, f"{kind} alphas={alphas}")


def test_select_several_blocks_max_batch():
    """64 sequences (the largest batch) with prefixes from 1 to 40000
    positions, so most rows of the launch grid are short or early-exit units
    beside a few long ones, under one shared workspace."""
    case("select, several blocks per head, 64 ragged sequences")
    rng = np.random.default_rng(64)
    B, Hkv, w = 64, 2, 16
    L = [int(x) for x in rng.integers(w + 1, 40001, B)]
    L[0], L[1] = 40000, w + 1
    pooled = np.zeros((B, Hkv, max(L)))
    for b in range(B):
        n = L[b] - w
        pooled[b, :, :n] = rng.integers(0, 1000, (Hkv, n)) / 64.0   # many ties
    alphas = [float(a) for a in rng.uniform(0.0, 0.99, B)]
    alphas[2] = 0.0
    _select_case(pooled, L, w, alphas, "max batch")


@pytest.mark.parametrize("seed", range(8))
def test_select_several_blocks_random_shapes(seed):
    """Seeded random batches whose longest prefix needs several blocks per
    head: batch size, heads, window, lengths, ratios and the score
    distribution (continuous, heavy ties, negative, all equal) drawn per case."""
    rng = np.random.default_rng(1000 + seed)
    B, Hkv, w = int(rng.integers(1, 5)), int(rng.integers(1, 4)), int(rng.integers(1, 65))
    L = [int(x) for x in rng.integers(w + 1, 90001, B)]
    L[int(rng.integers(0, B))] = int(rng.integers(32768 + w + 1, 90001))
    kind = ["normal", "ties", "negative", "equal"][seed % 4]
    case(f"select random shapes seed={seed} B={B} Hkv={Hkv} w={w} L={L} kind={kind}")
    pooled = np.zeros((B, Hkv, max(L)))
    for b in range(B):
        n = L[b] - w
        if kind == "normal":
            x = np.exp(rng.normal(0.0, 2.0, (Hkv, n)))
        elif kind == "ties":
            x = rng.integers(0, 7, (Hkv, n)) * 0.25
        elif kind == "negative":
            x = -np.abs(rng.normal(0.0, 1.0, (Hkv, n)))
        else:
            x = np.full((Hkv, n), 0.375)
        pooled[b, :, :n] = x
    alphas = [float(a) for a in rng.uniform(0.0, 0.999, B)]
    _select_case(pooled, L, w, alphas, f"seed={seed}")


def test_select_exact_narrow_range():
    case("select on keys that share all but their lowest bits")
    rng = np.random.default_rng(5)
    B, Hkv, w = 1, 2, 8
    L = [3000]
    base = np.float32(0.125)
    pooled = np.zeros((B, Hkv, L[0]))
    bits = np.frombuffer(base.tobytes(), dtype=np.uint32)[0]
    low = rng.integers(0, 4, (Hkv, L[0] - w)).astype(np.uint32)      # differ in 2 bits only
    pooled[0, :, : L[0] - w] = (bits + low).view(np.float32).astype(np.float64)
    for alphas in ([0.1], [0.5], [0.97]):
        _select_case(pooled, L, w, alphas, f"alphas={alphas}")


# ------------------------------------------------------------------ scoring
@pytest.mark.parametrize("dtype,d,G,w,pool,L", [
    (torch.float32, 64, 2, 16, 5, [512]),
    (torch.float32, 128, 1, 5, 3, [70, 333]),
    (torch.bfloat16, 128, 7, 32, 7, [1000, 65, 4097]),
    (torch.bfloat16, 64, 4, 64, 1, [129, 3000]),
    (torch.bfloat16, 128, 8, 40, 9, [2100]),          # 320 rows: two row chunks
    (torch.bfloat16, 128, 16, 64, 7, [700]),          # 1024 rows: four row chunks
    # blocks with idle waves (too few blocks to pack): 6, 4 and 7 row pairs
    (torch.bfloat16, 128, 6, 32, 7, [1000, 130]),     # 192 rows
    (torch.bfloat16, 64, 5, 20, 3, [777]),            # 100 rows, the last pair partial
    (torch.float32, 128, 7, 30, 5, [300, 2049]),      # 210 rows, the last pair partial
    (torch.bfloat16, 128, 2, 64, 7, [65, 200, 4160]), # 128 rows, ragged batch
])
def test_score_matches_oracle(dtype, d, G, w, pool, L):
    _score_case(dtype, d, G, w, pool, L, 2)


def _k1_packs(R, Lmax, Hkv, B):
    """Whether the library runs K1 with packed blocks (8 units of 32 rows x
    64 keys per block over at most two key tiles) for this shape: 4, 6 or 7
    row pairs, at least two packed blocks per CU and fewer blocks per CU than
    unpacked (256 CUs)."""
    P, nt, units = -(-R // 32), -(-Lmax // 64), Hkv * B
    plain, packed = nt * units, -(-P * nt // 8) * units
    return P in (4, 6, 7) and packed >= 512 and -(-packed // 256) < -(-plain // 256)


@pytest.mark.parametrize("dtype,d,G,w,pool,Hkv,L", [
    (torch.bfloat16, 128, 7, 32, 7, 8, [4600, 3001]),   # 224 rows: 7 row pairs
    (torch.bfloat16, 64, 6, 32, 5, 8, [4096, 3333]),    # 192 rows: 6 pairs
    (torch.float32, 128, 5, 20, 3, 4, [8200, 129]),     # 100 rows: 4 pairs, the last partial
    (torch.bfloat16, 128, 7, 30, 7, 8, [5150, 999]),    # 210 rows: 7 pairs, the last partial
])
def test_score_packed_blocks_match_oracle(dtype, d, G, w, pool, Hkv, L):
    assert _k1_packs(G * w, max(L), Hkv, len(L)), "shape does not take the packed blocks"
    _score_case(dtype, d, G, w, pool, L, Hkv)


def _score_case(dtype, d, G, w, pool, L, Hkv):
    case(f"score dtype={dtype} d={d} G={G} w={w} pool={pool} Hkv={Hkv} L={L}")
    wl = synth.custom(700 + d + G + w, dtype, len(L), L, G * Hkv, Hkv, d, w, pool, 1)
    pr = synth.make_prompt(wl, L=L, pad_value=float("nan"))    # padding must never be read
    ev = Evictor(len(L), max(L), G * Hkv, Hkv, d, w, pool, keep_raw=True)
    ev.scores.fill_(-7.0)
    ev.score(pr["q_win"].to(DEV), pr["k"].to(DEV), L)
    torch.cuda.synchronize()
    sc, raw = ev.scores.cpu().numpy(), ev.raw.cpu().numpy()
    worst = 0.0
    for b in range(len(L)):
        ref_raw = O.window_scores(f64(pr["q_win"][b]), f64(pr["k"][b]), L[b], w)
        ref = O.max_pool(ref_raw, pool)
        pref = L[b] - w
        worst = max(worst, score_rel_err(raw[b, :, :pref], ref_raw),
                    score_rel_err(sc[b, :, :pref], ref))
        assert np.all(sc[b, :, pref:] == -7.0), "scores beyond the prefix were written"
    print(f"max relative score error {worst:.3e}", flush=True)
    assert worst <= SCORE_REL_TOL


# ------------------------------------------------------------------ full chains
_POOLED = {}


def _oracle_pooled(wl, layer, b, q64, k64, n_x):
    key = (wl.wid, layer, b, n_x)
    if key not in _POOLED:
        _POOLED.clear() if len(_POOLED) > 64 else None
        _POOLED[key] = O.max_pool(O.window_scores(q64, k64, n_x, wl.w), wl.pool)
    return _POOLED[key]


def _run_layer(wl, layer, L, alphas, T, check_steps, prompt=None, dec=None):
    """GPU eviction + decode for one layer; checked against the oracle."""
    pr = prompt or synth.make_prompt(wl, layer, L=L)
    dc = dec or synth.make_decode(wl, layer, T=T)
    B, Hq, Hkv, d, w = wl.B, wl.Hq, wl.Hkv, wl.d, wl.w
    Lmax = max(L)
    ev = Evictor(B, Lmax, Hq, Hkv, d, w, wl.pool)
    n_keep_host = [O.keep_count(L[b], alphas[b], w) for b in range(B)]
    cache = _lib.KVCache(B, Hq, Hkv, max(n_keep_host) + T, d, wl.dtype)
    n_keep = ev.evict(pr["q_win"].to(DEV), pr["k"].to(DEV), pr["v"].to(DEV), L, alphas, cache)
    assert n_keep == n_keep_host
    out = run_decode(cache, dc["q"].to(DEV), dc["k_new"].to(DEV), dc["v_new"].to(DEV))
    torch.cuda.synchronize()
    keep = ev.keep_idx.cpu().numpy()
    sc = ev.scores.cpu().numpy()
    got = f64(out)
    excused, worst_score, worst_dec, p99 = 0, 0.0, 0.0, 0.0
    hits, planted = 0, 0
    for b in range(B):
        q64, k64, v64 = f64(pr["q_win"][b]), f64(pr["k"][b]), f64(pr["v"][b])
        pooled = _oracle_pooled(wl, layer, b, q64, k64, L[b])
        pref = L[b] - w
        worst_score = max(worst_score, score_rel_err(sc[b, :, :pref], pooled))
        p99 = max(p99, score_rel_err_p99(sc[b, :, :pref], pooled))
        kc = np.empty((Hkv, n_keep[b], d))
        vc = np.empty((Hkv, n_keep[b], d))
        for g in range(Hkv):
            gk = keep[b, g, : n_keep[b]]
            excused += check_keep(gk, pooled[g], L[b], w, n_keep[b],
                                  f"{wl.name} layer={layer} b={b} g={g} alpha={alphas[b]}")
            hv = pr.get("heavy", [[[]] * Hkv] * B)[b][g]
            hits += int(np.isin(hv, gk).sum())
            planted += len(hv)
            kc[g], vc[g] = k64[g, gk], v64[g, gk]
        ref = O.decode_sequence(f64(dc["q"][:, b]), f64(dc["k_new"][:, b]),
                                f64(dc["v_new"][:, b]), kc, vc, steps=check_steps)
        for t, o in ref.items():
            worst_dec = max(worst_dec, float(np.abs(got[t, b] - o).max()))
    # reported, not asserted: score accuracy (max, p99) and how many planted
    # heavy hitters the selection kept (a sanity figure, not a parity check)
    recall = f"{hits / planted:.3f} of {planted}" if planted else "n/a"
    print(f"{wl.name} layer={layer} alphas={[round(a, 4) for a in alphas]}: "
          f"excused={excused} score rel err max={worst_score:.2e} p99={p99:.2e} "
          f"max decode abs err={worst_dec:.2e} heavy-hitter recall={recall}", flush=True)
    assert worst_score <= SCORE_REL_TOL
    assert worst_dec <= DECODE_TOL[wl.dtype]
    return out


def _steps(T, every=16):
    return sorted(set([0, 1, T - 1] + list(range(0, T, every))))


def test_workload1_tiny_fp32():
    wl = synth.WORKLOADS[1]
    case(wl.name)
    _run_layer(wl, 0, [wl.L], [0.5], wl.T, range(wl.T))


@pytest.mark.parametrize("alpha", synth.WORKLOADS[2].alphas)
def test_workload2_single_layer(alpha):
    """Every one of the 256 decode steps checked against the oracle."""
    wl = synth.WORKLOADS[2]
    case(f"{wl.name} alpha={alpha}")
    _run_layer(wl, 0, [wl.L], [alpha], wl.T, range(wl.T))


def test_workload4_ragged():
    """16 ragged sequences, every one of the 256 decode steps checked."""
    wl = synth.WORKLOADS[4]
    L, alphas = synth.lengths_and_alphas(wl)
    case(f"{wl.name} L={L}")
    _run_layer(wl, 0, L, alphas, wl.T, range(wl.T))


@pytest.mark.parametrize("seed", range(12))
def test_full_chain_random_shapes(seed):
    """Score, select, compact and decode on seeded random shapes: batch size,
    heads and group size, head dimension, dtype, window, pool width, ragged
    lengths, one ratio per sequence and the decode step count all drawn."""
    rs = np.random.RandomState(7000 + seed)
    dtype = [torch.bfloat16, torch.float32][rs.randint(2)]
    d = [64, 128][rs.randint(2)]
    Hkv = int(rs.choice([1, 2, 4]))
    G = int(rs.choice([1, 2, 3, 4, 7, 8]))
    B = int(rs.randint(1, 5))
    w = int(rs.choice([1, 8, 31, 32, 64]))
    pool = int(rs.choice([1, 3, 5, 7]))
    T = int(rs.randint(1, 7))
    L = [int(x) for x in rs.randint(w + 1, 2600, size=B)]
    alphas = [float(x) for x in np.round(rs.uniform(0.0, 0.95, size=B), 3)]
    wl = synth.custom(7000 + seed, dtype, B, L, G * Hkv, Hkv, d, w, pool, T)
    case(f"random chain seed={seed} {dtype} d={d} Hkv={Hkv} G={G} w={w} pool={pool} "
         f"T={T} L={L} alphas={alphas}")
    _run_layer(wl, 0, L, alphas, T, range(T))


W3_DECODE_LAYERS = (0, 13, 27)


@pytest.mark.parametrize("layer", range(synth.WORKLOADS[3].layers))
def test_workload3_layer(layer):
    """One layer of the 28-layer stack at all 20 ratios k/20: eviction
    (scores, selection, compaction) checked at every ratio; decode checked at
    the first, second, last and every 16th step on layers 0, 13 and 27, and
    at the first and last step on the others."""
    wl = synth.WORKLOADS[3]
    steps = _steps(wl.T) if layer in W3_DECODE_LAYERS else [0, wl.T - 1]
    case(f"{wl.name} layer={layer}: eviction at {len(wl.alphas)} ratios, decode steps {steps}")
    pr = synth.make_prompt(wl, layer)
    dc = synth.make_decode(wl, layer)
    for a in wl.alphas:
        _run_layer(wl, layer, [wl.L], [a], wl.T, steps, prompt=pr, dec=dc)


@pytest.mark.parametrize("alpha", synth.WORKLOADS[5].alphas)
def test_workload5_long_context(alpha):
    """L = 131072: decode checked at the first, second, last and every 16th
    of the 512 steps."""
    wl = synth.WORKLOADS[5]
    case(f"{wl.name} alpha={alpha}")
    _run_layer(wl, 0, [wl.L], [alpha], wl.T, _steps(wl.T))


# ------------------------------------------------------------------ properties
def test_determinism_and_alpha0_identity():
    wl = synth.WORKLOADS[2]
    case(f"{wl.name}: run twice bit-identical; alpha=0 compacted == raw cache")
    pr = synth.make_prompt(wl)
    dc = synth.make_decode(wl, T=16)
    qd, kd, vd = pr["q_win"].to(DEV), pr["k"].to(DEV), pr["v"].to(DEV)
    res = []
    for _ in range(2):
        ev = Evictor(1, wl.L, wl.Hq, wl.Hkv, wl.d, wl.w, wl.pool, keep_raw=True)
        cache = _lib.KVCache(1, wl.Hq, wl.Hkv, wl.L + 16, wl.d, wl.dtype)
        ev.evict(qd, kd, vd, [wl.L], [0.5], cache)
        out = run_decode(cache, dc["q"].to(DEV), dc["k_new"].to(DEV), dc["v_new"].to(DEV))
        torch.cuda.synchronize()
        n_keep = cache.host_len[0] - 16
        pref = wl.L - wl.w
        res.append((ev.scores[:, :, :pref].clone(), ev.raw[:, :, :pref].clone(),
                    ev.keep_idx[:, :, :n_keep].clone(), out.clone()))
    for x, y in zip(res[0], res[1]):     # entries beyond these are unspecified
        assert torch.equal(x, y)
    # alpha = 0: the compacted cache is the prompt cache itself
    ev = Evictor(1, wl.L, wl.Hq, wl.Hkv, wl.d, wl.w, wl.pool)
    c0 = _lib.KVCache(1, wl.Hq, wl.Hkv, wl.L + 16, wl.d, wl.dtype)
    ev.evict(qd, kd, vd, [wl.L], [0.0], c0)
    c1 = _lib.KVCache(1, wl.Hq, wl.Hkv, wl.L + 16, wl.d, wl.dtype)
    c1.k[:, :, : wl.L].copy_(kd)
    v_rows = torch.zeros((1, wl.Hkv, c1.cap, wl.d), dtype=wl.dtype, device=DEV)
    v_rows[:, :, : wl.L] = vd
    c1.v.copy_(v_rows)
    c1.kv_len.fill_(wl.L)
    c1.host_len = [wl.L]
    o0 = run_decode(c0, dc["q"].to(DEV), dc["k_new"].to(DEV), dc["v_new"].to(DEV))
    o1 = run_decode(c1, dc["q"].to(DEV), dc["k_new"].to(DEV), dc["v_new"].to(DEV))
    torch.cuda.synchronize()
    assert torch.equal(ev.keep_idx[0, :, : wl.L].cpu(),
                       torch.arange(wl.L, dtype=torch.int32).expand(wl.Hkv, wl.L))
    assert torch.equal(o0, o1)


def test_decode_graph_replay():
    wl = synth.WORKLOADS[2]
    case(f"{wl.name}: 8 decode steps captured in a graph, replayed 3 times")
    T = 8
    pr = synth.make_prompt(wl)
    dc = synth.make_decode(wl, T=T)
    qd, knd, vnd = dc["q"].to(DEV), dc["k_new"].to(DEV), dc["v_new"].to(DEV)
    ev = Evictor(1, wl.L, wl.Hq, wl.Hkv, wl.d, wl.w, wl.pool)
    cache = _lib.KVCache(1, wl.Hq, wl.Hkv, 8192, wl.d, wl.dtype)
    ev.evict(pr["q_win"].to(DEV), pr["k"].to(DEV), pr["v"].to(DEV), [wl.L], [0.75], cache)
    torch.cuda.synchronize()
    len0 = cache.kv_len.clone()
    eager = torch.empty_like(qd)
    for t in range(T):
        _lib.tb_decode_attn(qd[t], knd[t], vnd[t], cache.k, cache.v, cache.kv_len, eager[t],
                            cache.ws)
    torch.cuda.synchronize()
    graph_out = torch.empty_like(qd)
    s = torch.cuda.Stream()
    cache.kv_len.copy_(len0)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for t in range(T):
            _lib.tb_decode_attn(qd[t], knd[t], vnd[t], cache.k, cache.v, cache.kv_len,
                                graph_out[t], cache.ws, stream=s)
    torch.cuda.synchronize()
    for rep in range(3):
        cache.kv_len.copy_(len0)
        graph_out.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(graph_out, eager), f"replay {rep} differs from eager"
        assert torch.equal(cache.kv_len, len0 + T)
