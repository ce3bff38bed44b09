"""GPU parity of the paged caches and of the multi-request server.

Paged compaction and decode must give bit-for-bit what the contiguous entry
points give on the same rows (the tile arithmetic is shared; only where a
tile lives differs), with sequences' pages scattered through the pool, pages
owned by nobody left untouched, and table entries past a sequence's length
holding junk.  The server test runs a stream of requests with per-request
ratios through admission, decode and retirement (slots move, pages are
reused) and checks every output against the float64 oracle; the
graph-replayed server step must equal the per-call step bit for bit, and so
must a server whose admissions overlap its decode steps.
"""
import numpy as np
import pytest
import torch

from oracle import timebill_oracle as O
from paper_2512_21859_amd import _lib, synth
from paper_2512_21859_amd.serving import PAGE, Server
from tests.parity_util import DECODE_TOL, check_keep, f64

pytestmark = pytest.mark.gpu
DEV = "cuda"
FILL = 0.5


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU in this container")
    _lib.load()
    torch.cuda.init()


def case(msg):
    print(f"\n[case] {msg}", flush=True)


def _gather_rows(pool, pages, g, n):
    return torch.cat([pool[p, g] for p in pages], dim=0)[:n]


@pytest.mark.parametrize("dtype,d,G", [(torch.bfloat16, 128, 7), (torch.bfloat16, 128, 8),
                                       (torch.bfloat16, 64, 1), (torch.float32, 128, 4),
                                       (torch.float32, 64, 3)])
def test_paged_equals_contiguous(dtype, d, G):
    case(f"paged_vs_contiguous dtype={dtype} d={d} G={G}")
    B, Hkv, Lmax, T = 3, 2, 1000, 40
    Hq = G * Hkv
    n_keep = [1, 517, 1000]                        # 517 + 40 crosses a page boundary
    max_pages = 36                                 # 1152 rows >= 1000 + 40
    gen = torch.Generator().manual_seed(77 + d + G)
    k = torch.randn((B, Hkv, Lmax, d), generator=gen).to(dtype)
    v = torch.randn((B, Hkv, Lmax, d), generator=gen).to(dtype)
    keep = torch.zeros((B, Hkv, Lmax), dtype=torch.int32)
    for b in range(B):
        for g in range(Hkv):
            keep[b, g, : n_keep[b]] = torch.sort(
                torch.randperm(Lmax, generator=gen)[: n_keep[b]]).values.to(torch.int32)
    q = torch.randn((T + 1, B, Hq, d), generator=gen).to(dtype)
    kn = torch.randn((T, B, Hkv, d), generator=gen).to(dtype)
    vn = torch.randn((T, B, Hkv, d), generator=gen).to(dtype)

    # pages scattered through a pool larger than needed; each row ends in junk entries
    need = [-(-(n + T) // PAGE) for n in n_keep]
    n_pages = sum(need) + 13
    perm = torch.randperm(n_pages, generator=gen).tolist()
    pages, at = [], 0
    for n in need:
        pages.append(perm[at:at + n])
        at += n
    unused = perm[at:]
    table = torch.empty((B, max_pages), dtype=torch.int32)
    for b in range(B):
        junk = [-7, 10 ** 6, n_pages][b]
        table[b] = torch.tensor(pages[b] + [junk] * (max_pages - need[b]), dtype=torch.int32)
    k_pool = torch.full((n_pages, Hkv, PAGE, d), FILL, dtype=dtype, device=DEV)
    v_pool = torch.full((n_pages, Hkv, PAGE, d), FILL, dtype=dtype, device=DEV)
    cap = max_pages * PAGE
    kc = torch.full((B, Hkv, cap, d), FILL, dtype=dtype, device=DEV)
    vc = torch.full((B, Hkv, cap, d), FILL, dtype=dtype, device=DEV)
    len_p = torch.zeros((B,), dtype=torch.int32, device=DEV)
    len_c = torch.zeros((B,), dtype=torch.int32, device=DEV)
    kd, vd, keepd, tabd = k.to(DEV), v.to(DEV), keep.to(DEV), table.to(DEV)

    _lib.tb_compact_kv(kd, vd, keepd, n_keep, kc, vc, len_c)
    _lib.tb_compact_kv_paged(kd, vd, keepd, n_keep, k_pool, v_pool, tabd, len_p)
    ws = torch.zeros((_lib.tb_workspace_bytes(_lib.TB_OP_DECODE, B, 0, Hq, Hkv, d, 0, cap),),
                     dtype=torch.uint8, device=DEV)
    ws_p = torch.zeros_like(ws)
    qd, knd, vnd = q.to(DEV), kn.to(DEV), vn.to(DEV)
    out_c = torch.empty((T + 1, B, Hq, d), dtype=dtype, device=DEV)
    out_p = torch.empty_like(out_c)
    for t in range(T + 1):
        a, b_ = (knd[t], vnd[t]) if t < T else (None, None)
        _lib.tb_decode_attn(qd[t], a, b_, kc, vc, len_c, out_c[t], ws)
        _lib.tb_decode_attn_paged(qd[t], a, b_, k_pool, v_pool, tabd, len_p, out_p[t], ws_p)
    torch.cuda.synchronize()

    assert len_p.tolist() == len_c.tolist() == [n + T for n in n_keep]
    assert torch.equal(out_p, out_c), "paged decode differs from the contiguous decode"
    for b in range(B):
        n = n_keep[b] + T
        for g in range(Hkv):
            assert torch.equal(_gather_rows(k_pool, pages[b], g, n), kc[b, g, :n])
            for t, p in enumerate(pages[b]):
                assert torch.equal(v_pool[p, g], vc[b, g, PAGE * t:PAGE * (t + 1)]), \
                    f"b={b} g={g} tile {t}"
    for p in unused:
        assert bool((k_pool[p] == FILL).all()) and bool((v_pool[p] == FILL).all()), \
            f"page {p} owned by nobody was written"

    # the oracle on sampled steps: kept prompt rows then the appended ones
    got, k64, v64, q64 = f64(out_p), f64(k), f64(v), f64(q)
    kn64, vn64 = f64(kn), f64(vn)
    for b in range(B):
        for g in range(Hkv):
            idx = keep[b, g, : n_keep[b]].long().numpy()
            for t in (0, T // 2, T - 1, T):
                s = min(t + 1, T)
                rk = np.concatenate([k64[b, g, idx], kn64[:s, b, g]])
                rv = np.concatenate([v64[b, g, idx], vn64[:s, b, g]])
                ref = O.decode_step(q64[t, b, g * G:(g + 1) * G], rk, rv)
                err = np.abs(got[t, b, g * G:(g + 1) * G] - ref).max()
                assert err <= DECODE_TOL[dtype], f"b={b} g={g} t={t}: max abs err {err}"


def test_server_stream_matches_oracle():
    """Ten requests with their own ratios and response lengths arrive over
    time; admission waits for slots and pages; finished requests retire and
    their pages are reused."""
    n_req, layers, Hq, Hkv, d, w, pool = 10, 2, 28, 4, 128, 32, 7
    G = Hq // Hkv
    gen = torch.Generator().manual_seed(2512)
    L = torch.randint(200, 2500, (n_req,), generator=gen).tolist()
    alphas = (0.9 * torch.rand(n_req, generator=gen, dtype=torch.float64)).tolist()
    max_new = torch.randint(3, 41, (n_req,), generator=gen).tolist()
    arrive = sorted(torch.randint(0, 30, (n_req,), generator=gen).tolist())
    case(f"server stream L={L} max_new={max_new} arrive={arrive}")
    wl = synth.custom(61, torch.bfloat16, n_req, L, Hq, Hkv, d, w, pool, max(max_new))
    prompts = [synth.make_prompt(wl, layer, L) for layer in range(layers)]
    dec = [synth.make_decode(wl, layer) for layer in range(layers)]

    srv = Server(layers, n_pages=260, max_seqs=5, max_pages=80, Hq=Hq, Hkv=Hkv, d=d,
                 dtype=torch.bfloat16, w=w, pool=pool, max_admit=3, max_prompt=max(L))
    queue = list(range(n_req))
    done_steps = {r: 0 for r in range(n_req)}
    n_keep_of, keep_of = {}, {}
    outs = {r: [] for r in range(n_req)}
    step, moved = 0, 0
    while queue or srv.n_active:
        for r in srv.slots.finished():
            if srv.rids().index(r) != srv.n_active - 1:
                moved += 1
            keep_of[r] = [t.cpu() for t in srv.keep[r]]
            srv.retire([r])
        batch = []
        while (queue and arrive[queue[0]] <= step and len(batch) < srv.max_admit and
               srv.slots.fits([_lib.tb_keep_count(L[r], alphas[r], w) + max_new[r]
                               for r in batch + [queue[0]]])):
            batch.append(queue.pop(0))
        if batch:
            bl = [L[r] for r in batch]
            lm = max(bl)
            pr = [{key: prompts[layer][key][batch][:, :, :lm].contiguous().to(DEV)
                   for key in ("q_win", "k", "v")} for layer in range(layers)]
            for layer in range(layers):
                pr[layer]["q_win"] = prompts[layer]["q_win"][batch].contiguous().to(DEV)
            nk = srv.admit(batch, bl, [alphas[r] for r in batch],
                           [max_new[r] for r in batch], pr, keep_sets=True)
            n_keep_of.update(zip(batch, nk))
        if srv.n_active:
            rid = srv.rids()
            qs = torch.stack([torch.stack([dec[layer]["q"][done_steps[r], r] for r in rid])
                              for layer in range(layers)]).to(DEV)
            ks = torch.stack([torch.stack([dec[layer]["k_new"][done_steps[r], r] for r in rid])
                              for layer in range(layers)]).to(DEV)
            vs = torch.stack([torch.stack([dec[layer]["v_new"][done_steps[r], r] for r in rid])
                              for layer in range(layers)]).to(DEV)
            out = torch.empty_like(qs)
            srv.step(qs, ks, vs, out)
            o = out.cpu()
            for i, r in enumerate(rid):
                outs[r].append(o[:, i])
                done_steps[r] += 1
        step += 1
        assert step < 500, "stream did not drain"
    torch.cuda.synchronize()
    assert moved > 0, "no slot move was exercised"
    assert len(srv.slots.free) == srv.slots.n_pages

    tol = DECODE_TOL[torch.bfloat16]
    for r in range(n_req):
        assert len(outs[r]) == max_new[r]
        for layer in range(layers):
            k64 = f64(prompts[layer]["k"][r])
            v64 = f64(prompts[layer]["v"][r])
            q64 = f64(prompts[layer]["q_win"][r])
            pooled = O.max_pool(O.window_scores(q64, k64, L[r], w), pool)
            keep = keep_of[r][layer].numpy()
            assert keep.shape == (Hkv, n_keep_of[r])
            for g in range(Hkv):
                check_keep(keep[g], pooled[g], L[r], w, n_keep_of[r], f"r={r} l={layer} g={g}")
            dq, dk, dv = (f64(dec[layer][x][:, r]) for x in ("q", "k_new", "v_new"))
            for s in range(max_new[r]):
                got = f64(outs[r][s][layer])
                for g in range(Hkv):
                    rk = np.concatenate([k64[g, keep[g]], dk[: s + 1, g]])
                    rv = np.concatenate([v64[g, keep[g]], dv[: s + 1, g]])
                    ref = O.decode_step(dq[s, g * G:(g + 1) * G], rk, rv)
                    err = np.abs(got[g * G:(g + 1) * G] - ref).max()
                    assert err <= tol, f"r={r} layer={layer} g={g} step={s}: err {err}"


def test_server_graph_step_equals_eager():
    """The graph-replayed step (one captured graph per batch size, reused as
    requests come and go) gives bit for bit what the per-call step gives."""
    n_req, layers, Hq, Hkv, d, w, pool = 7, 3, 28, 4, 128, 32, 7
    gen = torch.Generator().manual_seed(77)
    L = torch.randint(200, 1500, (n_req,), generator=gen).tolist()
    alphas = (0.8 * torch.rand(n_req, generator=gen, dtype=torch.float64)).tolist()
    max_new = torch.randint(2, 12, (n_req,), generator=gen).tolist()
    case(f"server graph vs eager L={L} max_new={max_new}")
    wl = synth.custom(62, torch.bfloat16, n_req, L, Hq, Hkv, d, w, pool, max(max_new))
    prompts = [synth.make_prompt(wl, layer, L) for layer in range(layers)]
    dec = [synth.make_decode(wl, layer) for layer in range(layers)]
    kw = dict(n_pages=200, max_seqs=4, max_pages=64, Hq=Hq, Hkv=Hkv, d=d, dtype=torch.bfloat16,
              w=w, pool=pool, max_admit=2, max_prompt=max(L))
    srv_e, srv_g = Server(layers, **kw), Server(layers, **kw)
    queue, done_steps, steps = list(range(n_req)), {r: 0 for r in range(n_req)}, 0
    sizes = set()
    while queue or srv_e.n_active:
        for r in srv_e.slots.finished():
            srv_e.retire([r])
            srv_g.retire([r])
        batch = []
        while (queue and len(batch) < 2 and srv_e.slots.fits(
                [_lib.tb_keep_count(L[r], alphas[r], w) + max_new[r] for r in batch + [queue[0]]])):
            batch.append(queue.pop(0))
        if batch:
            bl = [L[r] for r in batch]
            pr = [{key: prompts[layer][key][batch][:, :, :max(bl)].contiguous().to(DEV)
                   for key in ("k", "v")} for layer in range(layers)]
            for layer in range(layers):
                pr[layer]["q_win"] = prompts[layer]["q_win"][batch].contiguous().to(DEV)
            for srv in (srv_e, srv_g):
                srv.admit(batch, bl, [alphas[r] for r in batch], [max_new[r] for r in batch], pr)
        if not srv_e.n_active:
            continue
        assert srv_e.rids() == srv_g.rids()
        rid, n = srv_e.rids(), srv_e.n_active
        sizes.add(n)
        qs = torch.stack([torch.stack([dec[l]["q"][done_steps[r], r] for r in rid])
                          for l in range(layers)]).to(DEV)
        ks = torch.stack([torch.stack([dec[l]["k_new"][done_steps[r], r] for r in rid])
                          for l in range(layers)]).to(DEV)
        vs = torch.stack([torch.stack([dec[l]["v_new"][done_steps[r], r] for r in rid])
                          for l in range(layers)]).to(DEV)
        out = torch.empty_like(qs)
        srv_e.step(qs, ks, vs, out)
        srv_g.q_in[:, :n].copy_(qs)
        srv_g.k_in[:, :n].copy_(ks)
        srv_g.v_in[:, :n].copy_(vs)
        srv_g.step_graphed()
        torch.cuda.synchronize()
        assert torch.equal(out, srv_g.o_out[:, :n]), f"step {steps}: graph replay differs"
        for r in rid:
            done_steps[r] += 1
        steps += 1
        assert steps < 200
    assert len(sizes) >= 3, f"batch sizes seen: {sizes}"
    assert torch.equal(srv_e.kv_len, srv_g.kv_len)


def test_server_async_admission_equals_serialized():
    """Admission on its own stream while the running batch keeps decoding
    (graph-replayed) and retiring: with the batch promoted two steps after its
    eviction was queued, every step's outputs, the kept positions and the
    lengths equal, bit for bit, those of a server that admits the same batch
    serially at the promotion step."""
    n_req, layers, Hq, Hkv, d, w, pool = 9, 2, 28, 4, 128, 32, 7
    lag = 2
    gen = torch.Generator().manual_seed(4242)
    L = torch.randint(300, 3000, (n_req,), generator=gen).tolist()
    alphas = (0.9 * torch.rand(n_req, generator=gen, dtype=torch.float64)).tolist()
    max_new = torch.randint(2, 14, (n_req,), generator=gen).tolist()
    case(f"server async admission L={L} max_new={max_new}")
    wl = synth.custom(63, torch.bfloat16, n_req, L, Hq, Hkv, d, w, pool, max(max_new))
    prompts = [synth.make_prompt(wl, layer, L) for layer in range(layers)]
    dec = [synth.make_decode(wl, layer) for layer in range(layers)]
    kw = dict(n_pages=240, max_seqs=5, max_pages=96, Hq=Hq, Hkv=Hkv, d=d, dtype=torch.bfloat16,
              w=w, pool=pool, max_admit=3, max_prompt=max(L))
    srv_a, srv_s = Server(layers, **kw), Server(layers, **kw)
    with torch.cuda.stream(srv_a.decode_stream):  # steps on a queue of their own
        _async_vs_serial(srv_a, srv_s, L, alphas, max_new, prompts, dec, layers, w, lag)


def _async_vs_serial(srv_a, srv_s, L, alphas, max_new, prompts, dec, layers, w, lag):
    n_req = len(L)
    queue, done_steps, steps = list(range(n_req)), {r: 0 for r in range(n_req)}, 0
    pend = None                                  # (batch, prompts, step it joins)
    overlapped = retired_while_pending = 0
    while queue or srv_a.n_active or pend:
        for r in srv_a.slots.finished():
            assert torch.equal(torch.stack(srv_a.keep[r]), torch.stack(srv_s.keep[r]))
            srv_a.retire([r])
            srv_s.retire([r])
            retired_while_pending += pend is not None
        if pend and steps == pend[2]:
            batch, pr, _ = pend
            torch.cuda.synchronize()             # the eviction has finished: the poll sees it
            assert srv_a.promote_ready() == len(batch)
            srv_s.admit(batch, [L[r] for r in batch], [alphas[r] for r in batch],
                        [max_new[r] for r in batch], pr, keep_sets=True)
            pend = None
        if pend is None and queue:
            batch = []
            while (queue and len(batch) < 3 and srv_a.slots.fits(
                    [_lib.tb_keep_count(L[r], alphas[r], w) + max_new[r]
                     for r in batch + [queue[0]]])):
                batch.append(queue.pop(0))
            if batch:
                bl = [L[r] for r in batch]
                pr = [{key: prompts[layer][key][batch][:, :, :max(bl)].contiguous().to(DEV)
                       for key in ("k", "v")} for layer in range(layers)]
                for layer in range(layers):
                    pr[layer]["q_win"] = prompts[layer]["q_win"][batch].contiguous().to(DEV)
                srv_a.admit_async(batch, bl, [alphas[r] for r in batch],
                                  [max_new[r] for r in batch], pr, keep_sets=True)
                with pytest.raises(RuntimeError):
                    srv_a.admit(batch, bl, [alphas[r] for r in batch],
                                [max_new[r] for r in batch], pr)
                pend = (batch, pr, steps + lag)
        if srv_a.n_active:
            assert srv_a.rids() == srv_s.rids()
            rid, n = srv_a.rids(), srv_a.n_active
            qs = torch.stack([torch.stack([dec[l]["q"][done_steps[r], r] for r in rid])
                              for l in range(layers)]).to(DEV)
            ks = torch.stack([torch.stack([dec[l]["k_new"][done_steps[r], r] for r in rid])
                              for l in range(layers)]).to(DEV)
            vs = torch.stack([torch.stack([dec[l]["v_new"][done_steps[r], r] for r in rid])
                              for l in range(layers)]).to(DEV)
            out = torch.empty_like(qs)
            srv_s.step(qs, ks, vs, out)
            srv_a.q_in[:, :n].copy_(qs)
            srv_a.k_in[:, :n].copy_(ks)
            srv_a.v_in[:, :n].copy_(vs)
            srv_a.step_graphed()
            overlapped += pend is not None
            torch.cuda.synchronize()
            assert torch.equal(out, srv_a.o_out[:, :n]), f"step {steps}: outputs differ"
            assert torch.equal(srv_a.kv_len[:, :n], srv_s.kv_len[:, :n])
            for r in rid:
                done_steps[r] += 1
        steps += 1
        assert steps < 300, "stream did not drain"
    torch.cuda.synchronize()
    assert all(done_steps[r] == max_new[r] for r in range(n_req))
    assert overlapped >= 3, "no decode step ran beside an eviction"
    assert retired_while_pending >= 1, "no retirement happened while a batch was pending"
    assert len(srv_a.slots.free) == srv_a.slots.n_pages


def _rows(srv, r, layers):
    """The K and V rows of request r in every layer, gathered from its pages
    (queued on its server's decode stream, after the work queued there)."""
    e = next(x for x in srv.slots.slots if x.rid == r)
    with torch.cuda.stream(srv.decode_stream):
        out = []
        for layer in range(layers):
            for g in range(srv.Hkv):
                out.append(_gather_rows(srv.k_pool[layer], e.pages, g, e.length).clone())
                out.append(_gather_rows(srv.v_pool[layer], e.pages, g, e.length).clone())
        return out


def test_server_explicit_stream_admission_after_retire():
    """Decode steps queued with an explicit stream= outside any stream
    context, and each retirement followed at once, with no host
    synchronisation, by an overlapped admission whose batch reuses the pages
    just freed: the admission must wait for the queued steps (one may still
    append into a freed page).  Every step's outputs and the new requests'
    kept rows in their pages equal, bit for bit, those of a server that
    synchronises and admits serially."""
    n_req, layers, Hq, Hkv, d, w, pool = 8, 2, 28, 4, 128, 32, 7
    gen = torch.Generator().manual_seed(515)
    L = torch.randint(2000, 6000, (n_req,), generator=gen).tolist()
    alphas = (0.5 * torch.rand(n_req, generator=gen, dtype=torch.float64)).tolist()
    max_new = torch.randint(3, 9, (n_req,), generator=gen).tolist()
    case(f"server explicit-stream admission after retire L={L} max_new={max_new}")
    wl = synth.custom(65, torch.bfloat16, n_req, L, Hq, Hkv, d, w, pool, max(max_new))
    prompts = [synth.make_prompt(wl, layer, L) for layer in range(layers)]
    dec = [synth.make_decode(wl, layer) for layer in range(layers)]
    need = max(_lib.tb_keep_count(n, a, w) + m for n, a, m in zip(L, alphas, max_new))
    pages = -(-need // PAGE)
    kw = dict(n_pages=3 * pages, max_seqs=3, max_pages=pages, Hq=Hq, Hkv=Hkv, d=d,
              dtype=torch.bfloat16, w=w, pool=pool, max_admit=2, max_prompt=max(L))
    srv_a, srv_s = Server(layers, **kw), Server(layers, **kw)

    def prompt_of(batch):
        bl = max(L[r] for r in batch)
        pr = [{key: prompts[layer][key][batch][:, :, :bl].contiguous().to(DEV)
               for key in ("k", "v")} for layer in range(layers)]
        for layer in range(layers):
            pr[layer]["q_win"] = prompts[layer]["q_win"][batch].contiguous().to(DEV)
        return pr

    def args(batch):
        return (batch, [L[r] for r in batch], [alphas[r] for r in batch],
                [max_new[r] for r in batch], prompt_of(batch))

    queue, done = list(range(n_req)), {r: 0 for r in range(n_req)}
    outs_a, outs_s, rows_a, rows_s = [], [], {}, {}
    first = [queue.pop(0), queue.pop(0)]
    srv_a.admit(*args(first))
    srv_s.admit(*args(first))
    pend, steps, reused = None, 0, 0
    while queue or srv_a.n_active or pend:
        fin = srv_a.slots.finished()
        if fin:
            freed = {p for e in srv_a.slots.slots if e.rid in fin for p in e.pages}
            srv_a.retire(fin)                    # queued behind the steps, no sync
            srv_s.retire(fin)
        else:
            freed = set()
        if pend is not None and steps >= pend[1]:
            assert srv_a.promote_ready(wait=True) == len(pend[0])
            torch.cuda.synchronize()
            srv_s.admit(*args(pend[0]))
            torch.cuda.synchronize()
            for r in pend[0]:
                rows_a[r], rows_s[r] = _rows(srv_a, r, layers), _rows(srv_s, r, layers)
            pend = None
        if pend is None and queue and srv_a.slots.fits(
                [_lib.tb_keep_count(L[queue[0]], alphas[queue[0]], w) + max_new[queue[0]]]):
            batch = [queue.pop(0)]
            srv_a.admit_async(*args(batch))      # right behind the retirement
            taken = set(srv_a.slots.pending[0].pages)
            reused += bool(taken & freed)
            pend = (batch, steps + 1)
        n = srv_a.n_active
        if n:
            rid = srv_a.rids()
            assert rid == srv_s.rids()
            qs = torch.stack([torch.stack([dec[l]["q"][done[r], r] for r in rid])
                              for l in range(layers)]).to(DEV)
            ks = torch.stack([torch.stack([dec[l]["k_new"][done[r], r] for r in rid])
                              for l in range(layers)]).to(DEV)
            vs = torch.stack([torch.stack([dec[l]["v_new"][done[r], r] for r in rid])
                              for l in range(layers)]).to(DEV)
            oa, os_ = torch.empty_like(qs), torch.empty_like(qs)
            srv_a.step(qs, ks, vs, oa, stream=srv_a.decode_stream)    # explicit, no context
            srv_s.step(qs, ks, vs, os_)
            outs_a.append(oa)
            outs_s.append(os_)
            for r in rid:
                done[r] += 1
        steps += 1
        assert steps < 200, "stream did not drain"
    torch.cuda.synchronize()
    assert reused >= 1, "no admission took a page freed by the retirement before it"
    for t, (a, b) in enumerate(zip(outs_a, outs_s)):
        assert torch.equal(a, b), f"step {t}: outputs differ"
    assert set(rows_a) == set(range(2, n_req))
    for r in rows_a:
        for x, y in zip(rows_a[r], rows_s[r]):
            assert torch.equal(x, y), f"request {r}: kept rows differ"
    assert all(done[r] == max_new[r] for r in range(n_req))


def test_server_async_admission_rolls_back_on_error():
    """An admission whose eviction fails while being queued (layer 1's keys
    in the wrong dtype, caught on the host after layer 0 was queued) leaves
    nothing pending and every page free; the same batch admitted correctly
    afterwards decodes exactly as on a server that never saw the failure."""
    n_req, layers, Hq, Hkv, d, w, pool = 3, 2, 28, 4, 128, 32, 7
    L, alphas, max_new = [900, 1500, 700], [0.5, 0.2, 0.8], [3, 3, 3]
    case(f"server async admission rollback L={L}")
    wl = synth.custom(64, torch.bfloat16, n_req, L, Hq, Hkv, d, w, pool, max(max_new))
    prompts = [synth.make_prompt(wl, layer, L) for layer in range(layers)]
    dec = [synth.make_decode(wl, layer) for layer in range(layers)]
    kw = dict(n_pages=120, max_seqs=4, max_pages=48, Hq=Hq, Hkv=Hkv, d=d, dtype=torch.bfloat16,
              w=w, pool=pool, max_admit=3, max_prompt=max(L))
    srv, ref = Server(layers, **kw), Server(layers, **kw)
    rids = list(range(n_req))
    pr = [{key: prompts[layer][key].contiguous().to(DEV) for key in ("q_win", "k", "v")}
          for layer in range(layers)]
    bad = [dict(pr[0]), dict(pr[1])]
    bad[1]["k"] = bad[1]["k"].float()
    with pytest.raises(ValueError):
        srv.admit_async(rids, L, alphas, max_new, bad, keep_sets=True)
    assert not srv.slots.pending and not srv.keep
    assert len(srv.slots.free) == srv.slots.n_pages
    srv.admit_async(rids, L, alphas, max_new, pr, keep_sets=True)
    assert srv.promote_ready(wait=True) == n_req
    ref.admit(rids, L, alphas, max_new, pr, keep_sets=True)
    for t in range(max(max_new)):
        qs = torch.stack([dec[l]["q"][t, :n_req] for l in range(layers)]).to(DEV)
        ks = torch.stack([dec[l]["k_new"][t, :n_req] for l in range(layers)]).to(DEV)
        vs = torch.stack([dec[l]["v_new"][t, :n_req] for l in range(layers)]).to(DEV)
        o1, o2 = torch.empty_like(qs), torch.empty_like(qs)
        srv.step(qs, ks, vs, o1)
        ref.step(qs, ks, vs, o2)
        torch.cuda.synchronize()
        assert torch.equal(o1, o2), f"step {t}"
    for r in rids:
        assert torch.equal(torch.stack(srv.keep[r]), torch.stack(ref.keep[r]))


@pytest.mark.parametrize("overlap", [False, True])
def test_server_admits_by_budget(overlap):
    """Requests admitted by time budget carry the controller's ratio and
    pessimistic length: each keeps keep_count(L, alpha*) rows under the
    selection acceptance rule, reserves N_hat_W steps, and its first decode
    step matches the oracle over the kept rows."""
    from paper_2512_21859_amd.pipeline import TimeModel
    n_req, layers, Hq, Hkv, d, w, pool = 4, 1, 28, 4, 128, 32, 7
    L = [1200, 2600, 900, 3100]
    budgets = [60.0, 40.0, 1.0e4, 25.0]                    # tight to loose
    n_hat = [2, 3, 1, 2]
    model = TimeModel(prefill_abc=(1e-7, 2e-3, 1.0), step_pq=(2e-3, 0.5), bucket=4, k=2,
                      n_max=16, t_predict=0.5, alpha_max=0.9)
    case(f"server admission by budget overlap={overlap}")
    wl = synth.custom(65, torch.bfloat16, n_req, L, Hq, Hkv, d, w, pool, 16)
    prompts = [synth.make_prompt(wl, 0, L)]
    dec = synth.make_decode(wl, 0)
    srv = Server(layers, n_pages=400, max_seqs=4, max_pages=120, Hq=Hq, Hkv=Hkv, d=d,
                 dtype=torch.bfloat16, w=w, pool=pool, max_admit=4, max_prompt=max(L))
    pr = [{key: prompts[0][key].contiguous().to(DEV) for key in ("q_win", "k", "v")}]
    rids = list(range(n_req))
    with torch.cuda.stream(srv.decode_stream):
        plan = srv.admit_budgets(rids, L, budgets, n_hat, model, pr, keep_sets=True,
                                 overlap=overlap)
        if overlap:
            assert srv.promote_ready(wait=True) == n_req
        alphas = [a for a, _, _ in plan]
        assert len(set(alphas)) > 1, f"budgets should give different ratios: {plan}"
        for i, (a, feas, nw) in enumerate(plan):
            e = srv.slots.slots[i]
            assert e.rid == i and e.alpha == a and e.left == nw
            assert e.length == _lib.tb_keep_count(L[i], a, w)
        qs = dec["q"][0, :n_req].unsqueeze(0).to(DEV)
        ks = dec["k_new"][0, :n_req].unsqueeze(0).to(DEV)
        vs = dec["v_new"][0, :n_req].unsqueeze(0).to(DEV)
        out = torch.empty_like(qs)
        srv.step(qs, ks, vs, out)
        torch.cuda.synchronize()
    G = Hq // Hkv
    for i in range(n_req):
        n_keep = _lib.tb_keep_count(L[i], alphas[i], w)
        k64, v64, q64 = (f64(prompts[0][x][i]) for x in ("k", "v", "q_win"))
        pooled = O.max_pool(O.window_scores(q64, k64, L[i], w), pool)
        keep = srv.keep[i][0].cpu().numpy()
        got = f64(out[0, i])
        for g in range(Hkv):
            check_keep(keep[g], pooled[g], L[i], w, n_keep, f"r={i} g={g}")
            rk = np.concatenate([k64[g, keep[g]], f64(dec["k_new"][0, i, g])[None]])
            rv = np.concatenate([v64[g, keep[g]], f64(dec["v_new"][0, i, g])[None]])
            ref = O.decode_step(f64(dec["q"][0, i, g * G:(g + 1) * G]), rk, rv)
            assert np.abs(got[g * G:(g + 1) * G] - ref).max() <= DECODE_TOL[torch.bfloat16]


def test_paged_decode_clamps_table_entries():
    """Block-table entries outside the pool are clamped into it before use
    (the ABI's stated behaviour): a sequence whose table names pages -7 and 9
    in a 6-page pool attends over pages 0 and 5 there.  The appended row lands
    in a valid page."""
    case("paged decode with out-of-pool table entries")
    Hkv, G, d, n_pages, max_pages, n0 = 2, 4, 128, 6, 4, 100
    Hq = Hkv * G
    gen = torch.Generator().manual_seed(31)
    k_pool = torch.randn((n_pages, Hkv, PAGE, d), generator=gen).to(torch.bfloat16)
    v_pool = torch.randn((n_pages, Hkv, PAGE, d), generator=gen).to(torch.bfloat16)
    q = torch.randn((1, Hq, d), generator=gen).to(torch.bfloat16)
    kn = torch.randn((1, Hkv, d), generator=gen).to(torch.bfloat16)
    vn = torch.randn((1, Hkv, d), generator=gen).to(torch.bfloat16)
    table = torch.tensor([[-7, 9, 2, 3]], dtype=torch.int32)
    used = [0, 5, 2, 3]                                    # the clamped pages, tile by tile
    kp, vp = k_pool.to(DEV), v_pool.to(DEV)
    kv_len = torch.tensor([n0], dtype=torch.int32, device=DEV)
    out = torch.empty((1, Hq, d), dtype=torch.bfloat16, device=DEV)
    cap = max_pages * PAGE
    ws = torch.zeros((_lib.tb_workspace_bytes(_lib.TB_OP_DECODE, 1, 0, Hq, Hkv, d, 0, cap),),
                     dtype=torch.uint8, device=DEV)
    _lib.tb_decode_attn_paged(q.to(DEV), kn.to(DEV), vn.to(DEV), kp, vp, table.to(DEV), kv_len,
                              out, ws)
    torch.cuda.synchronize()
    assert kv_len.cpu().tolist() == [n0 + 1]
    got = f64(out[0])
    for g in range(Hkv):
        k_rows = torch.cat([k_pool[p, g] for p in used])[:n0]
        v_rows = torch.cat([v_pool[p, g] for p in used])[:n0]
        rk = np.concatenate([f64(k_rows), f64(kn[0, g])[None]])
        rv = np.concatenate([f64(v_rows), f64(vn[0, g])[None]])
        ref = O.decode_step(f64(q[0, g * G:(g + 1) * G]), rk, rv)
        assert np.abs(got[g * G:(g + 1) * G] - ref).max() <= DECODE_TOL[torch.bfloat16]
