"""GPU parity of the causal prefill attention (and its window-statistics
by-product) through the C ABI against the float64 oracle."""
import numpy as np
import pytest
import torch

from oracle import timebill_oracle as O
from paper_2512_21859_amd import _lib, synth
from tests.parity_util import DECODE_TOL, f64

pytestmark = pytest.mark.gpu
DEV = "cuda"
TOL = DECODE_TOL[torch.bfloat16]     # bf16 inputs/outputs, P rounded to bf16 (as decode)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU in this container")
    _lib.load()
    torch.cuda.init()


def case(msg):
    print(f"\n[case] {msg}", flush=True)


def _run(wl, L, w=0):
    pr = synth.make_prompt(wl, L=L)
    q = synth.make_queries(wl, L=L)
    out = torch.full(q.shape, 3.0, dtype=q.dtype, device=DEV)
    ws = (torch.full((wl.B, wl.Hq, w, 2), -5.0, dtype=torch.float32, device=DEV)
          if w else None)
    _lib.tb_prefill_attn(q.to(DEV), pr["k"].to(DEV), pr["v"].to(DEV), L, out, w, ws)
    torch.cuda.synchronize()
    return pr, q, out, ws


@pytest.mark.parametrize("d,Hq,Hkv,L,w", [
    (128, 14, 2, [300, 129], 32),
    (64, 8, 2, [1, 64, 200], 1),
    (128, 7, 1, [1000], 64),
    (64, 16, 2, [777, 2049], 32),      # d = 64 over many blocks, ragged tails
    # KV-head counts that do not divide the 8 XCDs of the block order, and
    # (tile, batch, KV head) unit counts that are not whole XCD rounds
    (128, 9, 3, [700, 1500, 33], 32),
    (64, 10, 5, [1200, 513], 16),
    (128, 16, 8, [1025], 32),
])
def test_prefill_matches_oracle(d, Hq, Hkv, L, w):
    case(f"prefill d={d} Hq={Hq} Hkv={Hkv} L={L} w={w}")
    _check_against_oracle(synth.custom(1300 + d + Hq, torch.bfloat16, len(L), L, Hq, Hkv, d, w, 1, 1), L, w)


@pytest.mark.parametrize("seed", range(6))
def test_prefill_random_shapes(seed):
    """Seeded random shapes: head dimension, KV heads, group size, batch,
    ragged lengths (including lengths below the window) and window size."""
    rs = np.random.RandomState(9100 + seed)
    d = [64, 128][rs.randint(2)]
    Hkv = int(rs.choice([1, 2, 4]))
    G = int(rs.choice([1, 2, 3, 4, 7, 8]))
    B = int(rs.randint(1, 4))
    w = int(rs.choice([0, 1, 16, 32, 64]))
    L = [int(x) for x in rs.randint(max(w, 1), 1500, size=B)]
    case(f"prefill random seed={seed} d={d} Hkv={Hkv} G={G} L={L} w={w}")
    _check_against_oracle(synth.custom(9100 + seed, torch.bfloat16, B, L, G * Hkv, Hkv, d, w, 1, 1), L, w)


def _check_against_oracle(wl, L, w):
    pr, q, out, ws = _run(wl, L, w)
    got = f64(out)
    wst = ws.cpu().numpy() if ws is not None else None
    worst = 0.0
    for b in range(len(L)):
        ref = O.prefill_attention(f64(q[b]), f64(pr["k"][b]), f64(pr["v"][b]), L[b])
        worst = max(worst, float(np.abs(got[b, :, : L[b]] - ref).max()))
        assert np.all(got[b, :, L[b]:] == 3.0), "rows past L were written"
        ww = min(w, L[b])
        if ww and ww == w:
            st = O.prefill_window_stats(f64(q[b]), f64(pr["k"][b]), L[b], w)
            assert np.all(np.abs(wst[b, ..., 0] - st[..., 0]) <= 1e-5 * (1 + np.abs(st[..., 0])))
            assert np.all(np.abs(wst[b, ..., 1] / st[..., 1] - 1) <= 1e-4)
    print(f"max abs error {worst:.2e}", flush=True)
    assert worst <= TOL


def test_prefill_full_size_sampled_rows():
    wl = synth.WORKLOADS[2]
    L = [wl.L]
    case(f"prefill at {wl.name}: sampled rows against the oracle, rerun bit-identical")
    pr, q, out, ws = _run(wl, L, wl.w)
    rows = [0, 1, 31, 32, 63, 64, 127, 128, 129, 4095, 4096, 8000, wl.L - wl.w, wl.L - 1]
    ref = O.prefill_attention(f64(q[0]), f64(pr["k"][0]), f64(pr["v"][0]), wl.L, rows)
    err = float(np.abs(f64(out)[0][:, rows] - ref).max())
    print(f"max abs error over sampled rows {err:.2e}", flush=True)
    assert err <= TOL
    st = O.prefill_window_stats(f64(q[0]), f64(pr["k"][0]), wl.L, wl.w)
    wst = ws.cpu().numpy()[0]
    assert np.all(np.abs(wst[..., 0] - st[..., 0]) <= 1e-5 * (1 + np.abs(st[..., 0])))
    assert np.all(np.abs(wst[..., 1] / st[..., 1] - 1) <= 1e-4)
    out2 = torch.empty_like(out)
    _lib.tb_prefill_attn(q.to(DEV), pr["k"].to(DEV), pr["v"].to(DEV), L, out2)
    torch.cuda.synchronize()
    assert torch.equal(out, out2)


@pytest.mark.parametrize("d,Hq,Hkv,L,w", [
    # longest prompt >= 8192: the 8-wave, 256-row blocks with 128-key stages;
    # ragged batch, tails that are not whole blocks or stages, d = 64 and 128
    (64, 8, 2, [8300, 1000, 4097], 32),
    (128, 7, 1, [300, 8193], 64),
    (128, 12, 3, [9001], 16),
])
def test_prefill_long_ragged_sampled_rows(d, Hq, Hkv, L, w):
    case(f"prefill long ragged d={d} Hq={Hq} Hkv={Hkv} L={L} w={w}: sampled rows")
    wl = synth.custom(4400 + d + Hq, torch.bfloat16, len(L), L, Hq, Hkv, d, w, 1, 1)
    pr, q, out, ws = _run(wl, L, w)
    got = f64(out)
    wst = ws.cpu().numpy()
    worst = 0.0
    for b, n in enumerate(L):
        rows = sorted({r for r in (0, 1, 63, 64, 127, 128, 255, 256, 257, 4095, 4096,
                                   8063, 8191, 8192, n - 129, n - 128, n - w, n - 2, n - 1)
                       if 0 <= r < n})
        ref = O.prefill_attention(f64(q[b]), f64(pr["k"][b]), f64(pr["v"][b]), n, rows)
        worst = max(worst, float(np.abs(got[b][:, rows] - ref).max()))
        assert np.all(got[b, :, n:] == 3.0), "rows past L were written"
        st = O.prefill_window_stats(f64(q[b]), f64(pr["k"][b]), n, w)
        assert np.all(np.abs(wst[b, ..., 0] - st[..., 0]) <= 1e-5 * (1 + np.abs(st[..., 0])))
        assert np.all(np.abs(wst[b, ..., 1] / st[..., 1] - 1) <= 1e-4)
    print(f"max abs error over sampled rows {worst:.2e}", flush=True)
    assert worst <= TOL
