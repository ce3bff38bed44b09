"""Stacked eviction (pipeline.StackEvictor): the layers of a stack are scored
one by one, then selected and compacted in one call each.  Every layer must
get exactly what the per-layer Evictor gives it: the same keep counts, kept
positions, compacted cache rows and lengths, for ragged batches, per-sequence
ratios and every scorer (window, averaged window, key norm, H2O); a decode step
over a layer's rows of the stacked cache must equal the decode over that
layer's own cache, bit for bit."""
import pytest
import torch

from paper_2512_21859_amd import _lib, synth
from paper_2512_21859_amd.pipeline import Evictor, StackEvictor

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU in this container")
    _lib.load()
    torch.cuda.init()


def case(msg):
    print(f"\n[case] {msg}", flush=True)


@pytest.mark.parametrize("scorer", ["snapkv", "snapkv_avg", "knorm"])
@pytest.mark.parametrize("layers,L,alphas", [(3, [3000, 2100], [0.3, 0.8]),
                                             (28, [4100], [0.55])])
def test_stack_equals_per_layer(scorer, layers, L, alphas):
    B, Hq, Hkv, d, w, pool, T = len(L), 8, 2, 128, 32, 7, 3
    case(f"{layers} layers, L={L}, alphas={alphas}, scorer={scorer}")
    wl = synth.custom(2300 + layers, torch.bfloat16, B, L, Hq, Hkv, d, w, pool, T)
    Lmax = max(L)
    prompts = [synth.make_prompt(wl, layer, L) for layer in range(layers)]
    st = {x: torch.cat([p[x] for p in prompts]).to(DEV) for x in ("q_win", "k", "v")}
    n_keep = [_lib.tb_keep_count(L[b], alphas[b], w) for b in range(B)]
    cap = max(n_keep) + T

    sev = StackEvictor(layers, B, Lmax, Hq, Hkv, d, w, pool, scorer=scorer)
    cs = _lib.KVCache(layers * B, Hq, Hkv, cap, d, wl.dtype)
    nk_s = sev.evict(st["q_win"], st["k"], st["v"], L, alphas, cs)
    assert nk_s == n_keep * layers

    ev = Evictor(B, Lmax, Hq, Hkv, d, w, pool, scorer=scorer)
    dec = synth.make_decode(wl, 0, T=1)
    for layer in range(layers):
        r = slice(layer * B, (layer + 1) * B)
        cl = _lib.KVCache(B, Hq, Hkv, cap, d, wl.dtype)
        nk = ev.evict(st["q_win"][r], st["k"][r], st["v"][r], L, alphas, cl)
        assert nk == n_keep
        torch.cuda.synchronize()
        assert torch.equal(cs.kv_len[r].cpu(), cl.kv_len.cpu())
        for b in range(B):
            n = nk[b]
            assert torch.equal(sev.keep_idx[layer * B + b, :, :n - w], ev.keep_idx[b, :, :n - w])
            assert torch.equal(cs.k[layer * B + b, :, :n], cl.k[b, :, :n])
            assert torch.equal(cs.v[layer * B + b, :, :n], cl.v[b, :, :n])
        if layer in (0, layers - 1):
            q, kn, vn = (dec[x][0].to(DEV) for x in ("q", "k_new", "v_new"))
            o_s = torch.empty((B, Hq, d), dtype=wl.dtype, device=DEV)
            o_l = torch.empty_like(o_s)
            _lib.tb_decode_attn(q, kn, vn, cs.k[r], cs.v[r], cs.kv_len[r], o_s, cs.ws)
            cl.decode(q, kn, vn, o_l)
            torch.cuda.synchronize()
            assert torch.equal(o_s, o_l)
            assert torch.equal(cs.kv_len[r].cpu(), cl.kv_len.cpu())


def test_stack_rejects_bad_shapes():
    """A stack larger than the batch limit, and inputs that do not hold
    layers * B sequences, are refused before any call."""
    with pytest.raises(ValueError):
        StackEvictor(65, 1, 256, 4, 2, 64, 8, 3)
    sev = StackEvictor(2, 1, 256, 4, 2, 64, 8, 3)
    k = torch.zeros((3, 2, 256, 64), dtype=torch.bfloat16, device=DEV)
    q = torch.zeros((3, 4, 8, 64), dtype=torch.bfloat16, device=DEV)
    cache = _lib.KVCache(2, 4, 2, 256, 64, torch.bfloat16)
    with pytest.raises(ValueError):
        sev.evict(q, k, k, [256], [0.5], cache)


def test_stack_equals_per_layer_h2o():
    """H2O takes every prompt query (q [layers*B, Hq, Lmax, d]) in place of
    the window queries; the stacked eviction must still equal the per-layer
    one, layer by layer."""
    layers, L, alphas = 3, [900, 640], [0.5, 0.25]
    B, Hq, Hkv, d, w, pool, T = len(L), 8, 2, 128, 32, 1, 2
    case(f"{layers} layers, L={L}, alphas={alphas}, scorer=h2o")
    wl = synth.custom(2400, torch.bfloat16, B, L, Hq, Hkv, d, w, pool, T)
    Lmax = max(L)
    prompts = [synth.make_prompt(wl, layer, L) for layer in range(layers)]
    q = torch.cat([synth.make_queries(wl, layer, L) for layer in range(layers)]).to(DEV)
    k = torch.cat([p["k"] for p in prompts]).to(DEV)
    v = torch.cat([p["v"] for p in prompts]).to(DEV)
    n_keep = [_lib.tb_keep_count(L[b], alphas[b], w) for b in range(B)]
    cap = max(n_keep) + T
    sev = StackEvictor(layers, B, Lmax, Hq, Hkv, d, w, pool, scorer="h2o")
    cs = _lib.KVCache(layers * B, Hq, Hkv, cap, d, wl.dtype)
    assert sev.evict(q, k, v, L, alphas, cs) == n_keep * layers
    ev = Evictor(B, Lmax, Hq, Hkv, d, w, pool, scorer="h2o")
    for layer in range(layers):
        r = slice(layer * B, (layer + 1) * B)
        cl = _lib.KVCache(B, Hq, Hkv, cap, d, wl.dtype)
        assert ev.evict(q[r], k[r], v[r], L, alphas, cl) == n_keep
        torch.cuda.synchronize()
        for b in range(B):
            n = n_keep[b]
            assert torch.equal(sev.keep_idx[layer * B + b, :, :n - w], ev.keep_idx[b, :, :n - w])
            assert torch.equal(cs.k[layer * B + b, :, :n], cl.k[b, :, :n])
            assert torch.equal(cs.v[layer * B + b, :, :n], cl.v[b, :, :n])
