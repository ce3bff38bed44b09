"""GPU parity of the scorer variants (KNorm, average-pool SnapKV) and of the
selection on signed scores, through the C ABI, against the float64 oracle.

Every case prints its name before touching the GPU; expected values come only
from the oracle.
"""
import numpy as np
import pytest
import torch

from oracle import scorers as S
from oracle import timebill_oracle as O
from paper_2512_21859_amd import _lib, synth
from paper_2512_21859_amd.pipeline import Evictor, run_decode
from tests.parity_util import DECODE_TOL, check_keep, f64, score_rel_err

pytestmark = pytest.mark.gpu
DEV = "cuda"
KNORM_REL_TOL = 1.2e-7      # one fp32 rounding of a float64 norm (6e-8), with margin
AVG_REL_TOL = 5e-7          # as for the max-pooled scores (fp32 raw scores, float64 mean)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU in this container")
    _lib.load()
    torch.cuda.init()


def case(msg):
    print(f"\n[case] {msg}", flush=True)


def _knorm_ref(pr, L, w):
    return [S.knorm_scores(f64(pr["k"][b]), L[b], w) for b in range(len(L))]


@pytest.mark.parametrize("dtype,d", [(torch.bfloat16, 128), (torch.bfloat16, 64),
                                     (torch.float32, 128), (torch.float32, 64)])
def test_knorm_scores_and_selection(dtype, d):
    L = [77, 4099, 9000]
    case(f"knorm dtype={dtype} d={d} L={L}")
    wl = synth.custom(950 + d, dtype, 3, L, 4, 2, d, 8, 7, 1)
    pr = synth.make_prompt(wl, L=L, pad_value=7.0)
    w, Lmax = wl.w, max(L)
    scores = torch.full((wl.B, wl.Hkv, Lmax), 123.0, dtype=torch.float32, device=DEV)
    _lib.tb_score_knorm(pr["k"].to(DEV), L, w, scores)
    torch.cuda.synchronize()
    sc = f64(scores)
    ref = _knorm_ref(pr, L, w)
    for b in range(wl.B):
        pref = L[b] - w
        assert score_rel_err(sc[b, :, :pref], ref[b]) <= KNORM_REL_TOL
        assert np.all(sc[b, :, pref:] == 123.0)              # untouched past the prefix
    keep = torch.full((wl.B, wl.Hkv, Lmax), -1, dtype=torch.int32, device=DEV)
    for alphas in ([0.0] * 3, [0.3, 0.5, 0.7], [0.95, 0.9, 0.99]):
        n_keep = _lib.tb_select_topk(scores, L, w, alphas, keep)
        torch.cuda.synchronize()
        kk = keep.cpu().numpy()
        for b in range(wl.B):
            for g in range(wl.Hkv):
                check_keep(kk[b, g, :n_keep[b]], ref[b][g], L[b], w, n_keep[b],
                           f"knorm b={b} g={g} alpha={alphas[b]}")


def test_select_signed_scores_exact():
    case("select on signed fp32 scores (negatives, +0 and -0, plateaus), bit-exact")
    rng = np.random.default_rng(21)
    B, Hkv, w = 2, 3, 5
    L = [300, 40000]
    x = rng.standard_normal((B, Hkv, max(L))) * 10.0 ** rng.uniform(-20, 5, (B, Hkv, max(L)))
    x[:, :, 10:20] = 0.0
    x[:, :, 20:30] = -0.0
    x[:, :, 200:260] = x[:, :, 200:201]                      # a plateau
    x[1, 1, :] = -np.abs(x[1, 1, :]) - 1e-3                   # one head all negative
    p32 = torch.from_numpy(x).to(torch.float32)
    keep = torch.full((B, Hkv, max(L)), -1, dtype=torch.int32, device=DEV)
    ref64 = p32.to(torch.float64).numpy()
    for alphas in ([0.0, 0.1], [0.5, 0.5], [0.9, 0.999], [0.97, 0.25]):
        n_keep = _lib.tb_select_topk(p32.to(DEV), L, w, alphas, keep)
        torch.cuda.synchronize()
        kk = keep.cpu().numpy()
        for b in range(B):
            for g in range(Hkv):
                want = O.select_keep(ref64[b, g, : L[b] - w], L[b], w, n_keep[b])
                assert np.array_equal(kk[b, g, : n_keep[b]], want), f"b={b} g={g} {alphas}"


@pytest.mark.parametrize("pool,L", [(7, [300, 5000]), (1, [200, 90]), (9, [14, 700])])
def test_avgpool_scores_and_selection(pool, L):
    case(f"average-pool window scores pool={pool} L={L}")
    wl = synth.custom(960 + pool, torch.bfloat16, len(L), L, 8, 2, 64, 8, pool, 1)
    pr = synth.make_prompt(wl, L=L)
    w, Lmax = wl.w, max(L)
    ev = Evictor(wl.B, Lmax, wl.Hq, wl.Hkv, wl.d, w, pool, keep_raw=True, scorer="snapkv_avg")
    ev.score(pr["q_win"].to(DEV), pr["k"].to(DEV), L)
    torch.cuda.synchronize()
    sc, raw = f64(ev.scores), f64(ev.raw)
    refs = []
    for b in range(wl.B):
        pref = L[b] - w
        a = O.window_scores(f64(pr["q_win"][b]), f64(pr["k"][b]), L[b], w)
        refs.append(S.avg_pool(a, pool))
        assert score_rel_err(raw[b, :, :pref], a) <= AVG_REL_TOL
        assert score_rel_err(sc[b, :, :pref], refs[b]) <= AVG_REL_TOL
    for alpha in (0.25, 0.5, 0.9):
        n_keep = ev.select(L, [alpha] * wl.B)
        torch.cuda.synchronize()
        kk = ev.keep_idx.cpu().numpy()
        for b in range(wl.B):
            for g in range(wl.Hkv):
                check_keep(kk[b, g, :n_keep[b]], refs[b][g], L[b], w, n_keep[b],
                           f"avgpool b={b} g={g} alpha={alpha}")


@pytest.mark.parametrize("scorer", ["knorm", "snapkv_avg"])
def test_scorer_end_to_end_decode(scorer):
    """Variant scores feed the same select, compact and decode (L = 8192 workload shape)."""
    wl = synth.WORKLOADS[2]
    T, alpha = 8, 0.5
    case(f"{scorer} end to end: {wl.name} alpha={alpha}, {T} decode steps")
    pr = synth.make_prompt(wl)
    dc = synth.make_decode(wl, T=T)
    L, w = [wl.L], wl.w
    ev = Evictor(1, wl.L, wl.Hq, wl.Hkv, wl.d, w, wl.pool, scorer=scorer)
    cache = _lib.KVCache(1, wl.Hq, wl.Hkv, _lib.tb_keep_count(wl.L, alpha, w) + T, wl.d, wl.dtype)
    n_keep = ev.evict(pr["q_win"].to(DEV), pr["k"].to(DEV), pr["v"].to(DEV), L, [alpha], cache)
    out = run_decode(cache, dc["q"].to(DEV), dc["k_new"].to(DEV), dc["v_new"].to(DEV))
    torch.cuda.synchronize()
    q64, k64, v64 = f64(pr["q_win"][0]), f64(pr["k"][0]), f64(pr["v"][0])
    if scorer == "knorm":
        ref = S.knorm_scores(k64, wl.L, w)
    else:
        ref = S.avg_pool(O.window_scores(q64, k64, wl.L, w), wl.pool)
    kk = ev.keep_idx.cpu().numpy()
    for g in range(wl.Hkv):
        check_keep(kk[0, g, :n_keep[0]], ref[g], wl.L, w, n_keep[0], f"{scorer} g={g}")
    # decode against the oracle on the GPU's own kept set
    kept = kk[0, :, :n_keep[0]]
    kc = np.stack([k64[g, kept[g]] for g in range(wl.Hkv)])
    vc = np.stack([v64[g, kept[g]] for g in range(wl.Hkv)])
    res = O.decode_sequence(f64(dc["q"][:, 0]), f64(dc["k_new"][:, 0]), f64(dc["v_new"][:, 0]),
                            kc, vc)
    want = np.stack([res[t] for t in range(T)])
    err = float(np.max(np.abs(f64(out[:, 0]) - want)))
    print(f"{scorer}: max decode abs err {err:.2e}")
    assert err <= DECODE_TOL[wl.dtype]


@pytest.mark.parametrize("alpha", synth.WORKLOADS[5].alphas)
def test_knorm_long_context(alpha):
    wl = synth.WORKLOADS[5]
    case(f"knorm {wl.name} alpha={alpha}")
    pr = synth.make_prompt(wl)
    L, w = [wl.L], wl.w
    scores = torch.empty((1, wl.Hkv, wl.L), dtype=torch.float32, device=DEV)
    _lib.tb_score_knorm(pr["k"].to(DEV), L, w, scores)
    keep = torch.empty((1, wl.Hkv, wl.L), dtype=torch.int32, device=DEV)
    n_keep = _lib.tb_select_topk(scores, L, w, [alpha], keep)
    torch.cuda.synchronize()
    ref = S.knorm_scores(f64(pr["k"][0]), wl.L, w)
    assert score_rel_err(f64(scores)[0, :, : wl.L - w], ref) <= KNORM_REL_TOL
    kk = keep.cpu().numpy()
    for g in range(wl.Hkv):
        check_keep(kk[0, g, :n_keep[0]], ref[g], wl.L, w, n_keep[0], f"knorm L=131072 g={g}")


# ------------------------------------------------------------------ H2O
def _h2o_gpu(q, k, L):
    B, Hq, Lmax, d = q.shape
    Hkv = k.shape[1]
    ws = torch.empty((_lib.tb_workspace_bytes(_lib.TB_OP_H2O, B, Lmax, Hq, Hkv, d, 0, 0),),
                     dtype=torch.uint8, device=DEV)
    scores = torch.full((B, Hkv, Lmax), 123.0, dtype=torch.float32, device=DEV)
    _lib.tb_score_h2o(q.to(DEV), k.to(DEV), L, scores, ws)
    torch.cuda.synchronize()
    return f64(scores)


@pytest.mark.parametrize("dtype,d,Hq,Hkv,L", [
    (torch.bfloat16, 128, 14, 2, [1000, 257]),
    (torch.float32, 64, 4, 2, [300]),
    (torch.bfloat16, 64, 3, 3, [37, 64, 65]),
    # 5 KV heads x 2 sequences: units that are not whole rounds of the 8 XCDs
    (torch.bfloat16, 128, 10, 5, [700, 1300]),
])
def test_h2o_scores_and_selection(dtype, d, Hq, Hkv, L):
    case(f"h2o dtype={dtype} d={d} Hq={Hq} Hkv={Hkv} L={L}")
    wl = synth.custom(970 + d + Hq, dtype, len(L), L, Hq, Hkv, d, 16, 1, 1)
    pr = synth.make_prompt(wl, L=L, pad_value=5.0)
    q = synth.make_queries(wl, L=L)
    sc = _h2o_gpu(q, pr["k"], L)
    G, w = Hq // Hkv, min(16, min(L) - 1)
    for b in range(len(L)):
        ref = S.h2o_scores(f64(q[b]), f64(pr["k"][b]), L[b])
        assert score_rel_err(sc[b, :, : L[b]], ref) <= AVG_REL_TOL
        np.testing.assert_allclose(sc[b, :, : L[b]].sum(axis=1), G * L[b], rtol=1e-6)
        assert np.all(sc[b, :, L[b]:] == 123.0)
        keep = torch.full((1, Hkv, L[b]), -1, dtype=torch.int32, device=DEV)
        for alpha in (0.3, 0.7):
            n_keep = _lib.tb_select_topk(torch.from_numpy(sc[b:b + 1, :, : L[b]]).float().to(DEV),
                                         [L[b]], w, [alpha], keep)
            torch.cuda.synchronize()
            kk = keep.cpu().numpy()
            for g in range(Hkv):
                check_keep(kk[0, g, :n_keep[0]], ref[g, : L[b] - w], L[b], w, n_keep[0],
                           f"h2o b={b} g={g} alpha={alpha}")


def test_h2o_full_size_sampled():
    """L = 8192 workload shape: every KV head's scores total G * L, and the last
    64 columns (which only need the statistics of the last 64 query rows) match
    the oracle computed column by column."""
    wl = synth.WORKLOADS[2]
    case(f"h2o full size {wl.name}: total mass and the last 64 columns")
    pr = synth.make_prompt(wl)
    q = synth.make_queries(wl)
    L = wl.L
    sc = _h2o_gpu(q, pr["k"], [L])[0]
    G = wl.Hq // wl.Hkv
    np.testing.assert_allclose(sc[:, :L].sum(axis=1), G * L, rtol=1e-6)
    q64, k64 = f64(q[0]), f64(pr["k"][0])
    tail = 64
    want = np.zeros((wl.Hkv, tail))
    for h in range(wl.Hq):
        g = h // G
        s = (q64[h, L - tail:] @ k64[g, :L].T) / np.sqrt(wl.d)          # rows L-64 .. L-1
        rows = np.arange(L - tail, L)[:, None]
        s = np.where(np.arange(L)[None, :] <= rows, s, -np.inf)
        p = np.exp(s - s.max(axis=1, keepdims=True))
        p /= p.sum(axis=1, keepdims=True)
        want[g] += p[:, L - tail:].sum(axis=0)                           # columns L-64 .. L-1
    assert score_rel_err(sc[:, L - tail: L], want) <= AVG_REL_TOL


def test_h2o_end_to_end_decode():
    wl = synth.custom(990, torch.bfloat16, 1, [1500], 8, 2, 128, 32, 1, 6)
    L, T, alpha = [1500], 6, 0.6
    case(f"h2o end to end L={L} alpha={alpha}, {T} decode steps")
    pr = synth.make_prompt(wl, L=L)
    dc = synth.make_decode(wl, T=T)
    q = synth.make_queries(wl, L=L)
    ev = Evictor(1, L[0], wl.Hq, wl.Hkv, wl.d, wl.w, 1, scorer="h2o")
    cache = _lib.KVCache(1, wl.Hq, wl.Hkv, _lib.tb_keep_count(L[0], alpha, wl.w) + T, wl.d,
                         wl.dtype)
    n_keep = ev.evict(q.to(DEV), pr["k"].to(DEV), pr["v"].to(DEV), L, [alpha], cache)
    out = run_decode(cache, dc["q"].to(DEV), dc["k_new"].to(DEV), dc["v_new"].to(DEV))
    torch.cuda.synchronize()
    k64, v64 = f64(pr["k"][0]), f64(pr["v"][0])
    ref = S.h2o_scores(f64(q[0]), k64, L[0])[:, : L[0] - wl.w]
    kk = ev.keep_idx.cpu().numpy()
    for g in range(wl.Hkv):
        check_keep(kk[0, g, :n_keep[0]], ref[g], L[0], wl.w, n_keep[0], f"h2o g={g}")
    kept = kk[0, :, :n_keep[0]]
    kc = np.stack([k64[g, kept[g]] for g in range(wl.Hkv)])
    vc = np.stack([v64[g, kept[g]] for g in range(wl.Hkv)])
    res = O.decode_sequence(f64(dc["q"][:, 0]), f64(dc["k_new"][:, 0]), f64(dc["v_new"][:, 0]),
                            kc, vc)
    want = np.stack([res[t] for t in range(T)])
    assert float(np.max(np.abs(f64(out[:, 0]) - want))) <= DECODE_TOL[wl.dtype]


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("scorer", ["knorm", "snapkv_avg"])
def test_scorer_chain_random_shapes(scorer, seed):
    """Variant scores through select, compact and decode on seeded random
    shapes: dtype, head dimension, KV heads and group size, window, pool
    width, ragged lengths with one ratio per sequence, decode step count."""
    rs = np.random.RandomState(9300 + seed + (100 if scorer == "knorm" else 0))
    dtype = [torch.bfloat16, torch.float32][rs.randint(2)]
    d = [64, 128][rs.randint(2)]
    Hkv = int(rs.choice([1, 2, 4]))
    G = int(rs.choice([1, 2, 4, 7, 8]))
    B = int(rs.randint(1, 4))
    w = int(rs.choice([1, 8, 32]))
    pool = int(rs.choice([1, 3, 7]))
    T = int(rs.randint(1, 5))
    L = [int(x) for x in rs.randint(w + 1, 3000, size=B)]
    alphas = [float(x) for x in np.round(rs.uniform(0.0, 0.95, size=B), 3)]
    case(f"{scorer} random chain seed={seed} {dtype} d={d} Hkv={Hkv} G={G} w={w} "
         f"pool={pool} T={T} L={L} alphas={alphas}")
    wl = synth.custom(9300 + seed, dtype, B, L, G * Hkv, Hkv, d, w, pool, T)
    pr = synth.make_prompt(wl, L=L)
    dc = synth.make_decode(wl, T=T)
    ev = Evictor(B, max(L), wl.Hq, Hkv, d, w, pool, scorer=scorer)
    n_host = [_lib.tb_keep_count(L[b], alphas[b], w) for b in range(B)]
    cache = _lib.KVCache(B, wl.Hq, Hkv, max(n_host) + T, d, dtype)
    n_keep = ev.evict(pr["q_win"].to(DEV), pr["k"].to(DEV), pr["v"].to(DEV), L, alphas, cache)
    assert n_keep == n_host
    out = run_decode(cache, dc["q"].to(DEV), dc["k_new"].to(DEV), dc["v_new"].to(DEV))
    torch.cuda.synchronize()
    kk = ev.keep_idx.cpu().numpy()
    worst = 0.0
    for b in range(B):
        q64, k64, v64 = f64(pr["q_win"][b]), f64(pr["k"][b]), f64(pr["v"][b])
        if scorer == "knorm":
            ref = S.knorm_scores(k64, L[b], w)
        else:
            ref = S.avg_pool(O.window_scores(q64, k64, L[b], w), pool)
        for g in range(Hkv):
            check_keep(kk[b, g, :n_keep[b]], ref[g], L[b], w, n_keep[b], f"{scorer} b={b} g={g}")
        kept = kk[b, :, :n_keep[b]]
        kc = np.stack([k64[g, kept[g]] for g in range(Hkv)])
        vc = np.stack([v64[g, kept[g]] for g in range(Hkv)])
        res = O.decode_sequence(f64(dc["q"][:, b]), f64(dc["k_new"][:, b]), f64(dc["v_new"][:, b]),
                                kc, vc)
        for t in range(T):
            worst = max(worst, float(np.max(np.abs(f64(out[t, b]) - res[t]))))
    print(f"{scorer}: max decode abs err {worst:.2e}", flush=True)
    assert worst <= DECODE_TOL[dtype]
