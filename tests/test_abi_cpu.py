"""C ABI checks that need no GPU: the library loads, exports every declared
symbol, computes n_keep like the oracle, sizes workspaces, and rejects bad
arguments before any HIP call (only calls that fail validation are made)."""
import ctypes
import json
import os
import re
import subprocess

import pytest

from oracle import timebill_oracle as O
from paper_2512_21859_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "timebill.h")


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def _declared():
    text = open(HEADER).read()
    decl = r"^(?:int32_t|int64_t|size_t|double|tb_status|const char\*)\s+(tb_[a-z0-9_]+)\("
    return sorted(set(re.findall(decl, text, re.M)))


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert set(names) == set(_lib.EXPORTED), names
    nm = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB_PATH], capture_output=True,
                        text=True, check=True).stdout
    exported = set(re.findall(r" T (\S+)$", nm, re.M))
    for n in names:
        assert n in exported, f"{n} not exported"
        assert hasattr(lib, n)
    # nothing else: internal code is built with hidden visibility
    assert exported == set(names), sorted(exported - set(names))


def test_keep_count_matches_oracle_and_table(lib):
    with open(os.path.join(ROOT, "tests", "golden", "n_keep_table.json")) as f:
        tab = json.load(f)
    for case in tab["cases"]:
        alphas = case.get("alphas") or [k / 20 for k in case["alphas_k_over_20"]]
        assert [_lib.tb_keep_count(case["n_x"], a, case["w"]) for a in alphas] == case["n_keep"]
    for L in (2, 3, 17, 1000, 131072):
        for a in (0.0, 0.05, 0.3333, 0.5, 0.9, 0.999):
            for w in (1, 2, 16):
                if w < L:
                    assert _lib.tb_keep_count(L, a, w) == O.keep_count(L, a, w)
    assert _lib.tb_keep_count(10, 1.0, 2) == -1
    assert _lib.tb_keep_count(10, -0.5, 2) == -1
    assert _lib.tb_keep_count(10, 0.5, 10) == -1


def test_workspace_sizes(lib):
    s = _lib.tb_workspace_bytes(_lib.TB_OP_SCORE, 1, 8192, 28, 4, 128, 32, 0)
    assert s >= 4 * 128 * 224 * 64 * 4                     # the per-tile exponentials
    assert _lib.tb_workspace_bytes(_lib.TB_OP_SELECT, 1, 8192, 28, 4, 128, 32, 0) == 0
    # prefixes past 32768 positions may select with several blocks per head
    assert _lib.tb_workspace_bytes(_lib.TB_OP_SELECT, 1, 32768 + 32, 0, 4, 0, 32, 0) == 0
    sel = _lib.tb_workspace_bytes(_lib.TB_OP_SELECT, 3, 32768 + 33, 0, 4, 0, 32, 0)
    assert sel > 0 and sel % (3 * 4) == 0
    assert sel == _lib.tb_workspace_bytes(_lib.TB_OP_SELECT, 3, 131072, 0, 4, 0, 64, 0)
    assert _lib.tb_workspace_bytes(_lib.TB_OP_SELECT, 0, 131072, 0, 4, 0, 64, 0) == 0
    d = _lib.tb_workspace_bytes(_lib.TB_OP_DECODE, 1, 0, 28, 4, 128, 0, 8448)
    assert d > 8 and d % 256 == 0
    assert _lib.tb_workspace_bytes(_lib.TB_OP_DECODE, 1, 0, 28, 5, 128, 0, 8448) == 0
    assert b"bad sizes" in lib.tb_last_error()
    assert _lib.tb_workspace_bytes(9, 1, 1, 1, 1, 64, 1, 1) == 0


def test_decode_workspace_covers_smaller_batches(lib):
    """The decode split depends on the batch size; the reported workspace for B
    covers every batch of at most B sequences, so it never shrinks as B grows."""
    for Hq, Hkv, d in ((28, 4, 128), (32, 8, 128), (2, 1, 64)):
        for cap in (32, 672, 2112, 8448, 16640, 32896, 131136):
            sizes = [_lib.tb_workspace_bytes(_lib.TB_OP_DECODE, B, 0, Hq, Hkv, d, 0, cap)
                     for B in range(1, 40)]
            assert all(s > 0 for s in sizes)
            assert sizes == sorted(sizes), (Hq, Hkv, d, cap)


FAKE = ctypes.c_void_p(0x1000)     # never dereferenced: every call below fails validation


def _i32(*v):
    return (ctypes.c_int32 * len(v))(*v)


def _score(lib, fn=None, **kw):
    a = dict(q=FAKE, k=FAKE, B=1, L=_i32(100), Lmax=100, Hq=4, Hkv=2, d=128, w=8, pool=7,
             dt=_lib.TB_BF16, sc=FAKE, raw=None, ws=FAKE, wsb=1 << 40)
    a.update(kw)
    fn = lib.tb_score_window if fn is None else fn
    return fn(a["q"], a["k"], a["B"], a["L"], a["Lmax"], a["Hq"], a["Hkv"],
                               a["d"], a["w"], a["pool"], a["dt"], a["sc"], a["raw"], a["ws"],
                               a["wsb"], None)


def test_score_validation(lib):
    E = _lib
    assert _score(lib, q=None) == E.TB_EINVAL
    assert _score(lib, B=0) == E.TB_EINVAL
    assert _score(lib, B=65, L=_i32(*([100] * 65))) == E.TB_EUNSUPPORTED
    assert _score(lib, Hq=5) == E.TB_EINVAL
    assert _score(lib, d=96) == E.TB_EUNSUPPORTED
    assert _score(lib, dt=7) == E.TB_EUNSUPPORTED
    assert _score(lib, w=0) == E.TB_EINVAL
    assert _score(lib, pool=4) == E.TB_EINVAL
    assert _score(lib, pool=131) == E.TB_EUNSUPPORTED
    assert _score(lib, w=100) == E.TB_EINVAL            # w must be < L
    assert _score(lib, L=_i32(101)) == E.TB_EINVAL      # L > Lmax
    assert _score(lib, Hq=40, Hkv=1, w=32) == E.TB_EUNSUPPORTED   # G*w > 1024
    assert _score(lib, Hq=64, Hkv=1, w=1 << 27, L=_i32((1 << 27) + 1),
                  Lmax=(1 << 27) + 1) == E.TB_EUNSUPPORTED          # G*w would wrap an int
    assert _lib.tb_workspace_bytes(_lib.TB_OP_SCORE, 1, 1 << 28, 64, 1, 128, 1 << 27, 0) == 0
    assert _score(lib, wsb=16) == E.TB_EWORKSPACE
    assert b"workspace" in lib.tb_last_error()


def test_score_avgpool_validation(lib):
    """The average-pool entry validates exactly like tb_score_window."""
    E = _lib
    for kw, want in [(dict(q=None), E.TB_EINVAL), (dict(pool=4), E.TB_EINVAL),
                     (dict(w=100), E.TB_EINVAL), (dict(Hq=40, Hkv=1, w=32), E.TB_EUNSUPPORTED),
                     (dict(wsb=16), E.TB_EWORKSPACE)]:
        assert _score(lib, fn=lib.tb_score_window_avgpool, **kw) == want, kw
    assert b"tb_score_window_avgpool: workspace" in lib.tb_last_error()


def test_score_knorm_validation(lib):
    E = _lib

    def call(k=FAKE, B=1, L=100, Lmax=100, Hkv=2, d=128, w=8, dt=_lib.TB_BF16, sc=FAKE):
        return lib.tb_score_knorm(k, B, _i32(L), Lmax, Hkv, d, w, dt, sc, None)

    assert call(k=None) == E.TB_EINVAL
    assert call(sc=None) == E.TB_EINVAL
    assert call(B=0) == E.TB_EINVAL
    assert call(d=96) == E.TB_EUNSUPPORTED
    assert call(dt=7) == E.TB_EUNSUPPORTED
    assert call(w=0) == E.TB_EINVAL
    assert call(w=100) == E.TB_EINVAL
    assert call(L=101) == E.TB_EINVAL
    assert b"L[0]" in lib.tb_last_error()


def test_score_h2o_validation(lib):
    E = _lib

    def call(q=FAKE, k=FAKE, B=1, L=100, Lmax=100, Hq=4, Hkv=2, d=128, dt=_lib.TB_BF16,
             sc=FAKE, ws=FAKE, wsb=1 << 30):
        return lib.tb_score_h2o(q, k, B, _i32(L), Lmax, Hq, Hkv, d, dt, sc, ws, wsb, None)

    assert call(q=None) == E.TB_EINVAL
    assert call(B=0) == E.TB_EINVAL
    assert call(Hq=5) == E.TB_EINVAL
    assert call(d=96) == E.TB_EUNSUPPORTED
    assert call(L=0) == E.TB_EINVAL
    assert call(L=101) == E.TB_EINVAL
    need = _lib.tb_workspace_bytes(_lib.TB_OP_H2O, 1, 100, 4, 2, 128, 0, 0)
    assert need >= 3 * 4 * 100 * 8
    assert call(wsb=need - 1) == E.TB_EWORKSPACE
    assert call(ws=None) == E.TB_EWORKSPACE


def test_prefill_validation(lib):
    E = _lib

    def call(q=FAKE, B=1, L=100, Lmax=100, Hq=4, Hkv=2, d=128, dt=_lib.TB_BF16, out=FAKE,
             w=8, ws=FAKE):
        return lib.tb_prefill_attn(q, FAKE, FAKE, B, _i32(L), Lmax, Hq, Hkv, d, dt, out, w, ws,
                                   None)

    assert call(q=None) == E.TB_EINVAL
    assert call(out=None) == E.TB_EINVAL
    assert call(dt=_lib.TB_F32) == E.TB_EUNSUPPORTED
    assert b"bf16 only" in lib.tb_last_error()
    assert call(Hq=5) == E.TB_EINVAL
    assert call(d=96) == E.TB_EUNSUPPORTED
    assert call(L=0) == E.TB_EINVAL
    assert call(L=101) == E.TB_EINVAL
    assert call(w=0) == E.TB_EINVAL                     # window statistics need w >= 1
    assert call(w=101, L=100) == E.TB_EINVAL            # and w <= L
    assert call(w=0, ws=None, B=0) == E.TB_EINVAL


def test_select_validation(lib):
    E = _lib
    n_keep = (ctypes.c_int32 * 1)()

    def call(alpha=0.5, L=100, Lmax=100, w=8, B=1, keep=FAKE):
        a = (ctypes.c_double * 1)(alpha)
        return lib.tb_select_topk(FAKE, B, _i32(L), Lmax, 2, w, a, keep, n_keep, None, 0, None)

    assert call(alpha=1.0) == E.TB_EINVAL
    assert call(alpha=-0.1) == E.TB_EINVAL
    assert call(alpha=float("nan")) == E.TB_EINVAL
    assert call(L=101) == E.TB_EINVAL
    assert call(w=100) == E.TB_EINVAL
    assert call(B=0) == E.TB_EINVAL
    assert call(keep=None) == E.TB_EINVAL


def test_select_workspace_validation(lib):
    """A workspace is needed only where a prefix is long enough for several
    blocks per head; then it must be large enough and aligned.  Checked
    before anything is enqueued."""
    E = _lib
    n_keep = (ctypes.c_int32 * 2)()
    L, w, Hkv = [40000, 20000], 32, 2            # the first prefix (39968) is long enough
    need = _lib.tb_workspace_bytes(_lib.TB_OP_SELECT, 2, 40000, 0, Hkv, 0, w, 0)

    def call(ws, nbytes, L=L):
        a = (ctypes.c_double * 2)(0.5, 0.5)
        return lib.tb_select_topk(FAKE, 2, _i32(*L), 40000, Hkv, w, a, FAKE, n_keep,
                                  ws, nbytes, None)

    assert call(FAKE, need - 1) == E.TB_EWORKSPACE
    assert b"workspace" in lib.tb_last_error()
    assert call(ctypes.c_void_p(0x1002), need) == E.TB_EINVAL          # misaligned
    assert b"aligned" in lib.tb_last_error()


def test_compact_validation(lib):
    E = _lib

    def call(n=50, cap=64, Lmax=100, d=128, dt=_lib.TB_BF16, kc=FAKE):
        return lib.tb_compact_kv(FAKE, FAKE, FAKE, 1, _i32(n), Lmax, 2, d, dt, cap, kc, FAKE,
                                 FAKE, None, 0, None)

    assert call(n=65) == E.TB_EINVAL          # beyond cap
    assert call(cap=60) == E.TB_EINVAL        # cap not a whole number of 32-row tiles
    assert call(n=0) == E.TB_EINVAL
    assert call(n=101, cap=200) == E.TB_EINVAL  # beyond Lmax
    assert call(d=32) == E.TB_EUNSUPPORTED
    assert call(kc=None) == E.TB_EINVAL


def test_decode_validation(lib):
    E = _lib

    def call(Hq=28, Hkv=4, d=128, cap=128, wsb=1 << 30, kn=FAKE, vn=FAKE, ws=FAKE):
        return lib.tb_decode_attn(FAKE, kn, vn, FAKE, FAKE, FAKE, 1, Hq, Hkv, d, cap,
                                  _lib.TB_BF16, FAKE, ws, wsb, None)

    assert call(kn=None) == E.TB_EINVAL       # k_new without v_new
    assert call(Hq=36, Hkv=4) == E.TB_EUNSUPPORTED   # G = 9
    assert call(Hq=30) == E.TB_EINVAL
    assert call(d=256) == E.TB_EUNSUPPORTED
    assert call(cap=0) == E.TB_EINVAL
    assert call(cap=100) == E.TB_EINVAL       # cap not a whole number of 32-row tiles
    assert call(wsb=8) == E.TB_EWORKSPACE
    assert call(ws=None) == E.TB_EINVAL


def test_decode_noalloc_validation(lib):
    """The entry point without a workspace validates like tb_decode_attn and
    refuses, before any HIP call, a call whose workspace need exceeds the
    library's 16 MiB scratch."""
    E = _lib

    def call(B=1, Hq=28, Hkv=4, d=128, cap=128, kn=FAKE, vn=FAKE, q=FAKE):
        return lib.tb_decode_attn_noalloc(q, kn, vn, FAKE, FAKE, FAKE, B, Hq, Hkv, d, cap,
                                          _lib.TB_BF16, FAKE, None)

    assert call(q=None) == E.TB_EINVAL
    assert call(kn=None) == E.TB_EINVAL
    assert call(Hq=36, Hkv=4) == E.TB_EUNSUPPORTED
    assert call(cap=100) == E.TB_EINVAL
    big = dict(B=64, Hq=64, Hkv=8, d=128, cap=65536)
    assert _lib.tb_workspace_bytes(_lib.TB_OP_DECODE, 64, 0, 64, 8, 128, 0, 65536) > 16 << 20
    assert call(**big) == E.TB_EWORKSPACE
    assert b"scratch" in lib.tb_last_error()


def test_compact_paged_validation(lib):
    E = _lib

    def call(n=50, max_pages=2, n_pages=8, table=FAKE, kp=FAKE, d=128):
        return lib.tb_compact_kv_paged(FAKE, FAKE, FAKE, 1, _i32(n), 100, 2, d, _lib.TB_BF16,
                                       kp, FAKE, n_pages, table, max_pages, FAKE, None)

    assert call(table=None) == E.TB_EINVAL
    assert b"block table" in lib.tb_last_error()
    assert call(max_pages=0) == E.TB_EINVAL
    assert call(n_pages=0) == E.TB_EINVAL
    assert call(max_pages=1 << 27) == E.TB_EUNSUPPORTED
    assert call(max_pages=(1 << 25) + 1) == E.TB_EUNSUPPORTED   # capacity would pass 2^30 rows
    assert call(max_pages=1 << 26) == E.TB_EUNSUPPORTED         # 2^26 * 32 overflows int32
    assert call(n=65) == E.TB_EINVAL          # beyond max_pages * 32 rows
    assert call(kp=None) == E.TB_EINVAL
    assert call(d=32) == E.TB_EUNSUPPORTED


def test_decode_paged_validation(lib):
    E = _lib

    def call(Hq=28, Hkv=4, d=128, max_pages=4, n_pages=8, table=FAKE, wsb=1 << 30, kn=FAKE,
             vn=FAKE):
        return lib.tb_decode_attn_paged(FAKE, kn, vn, FAKE, FAKE, n_pages, table, max_pages, FAKE,
                                        1, Hq, Hkv, d, _lib.TB_BF16, FAKE, FAKE, wsb, None)

    assert call(table=None) == E.TB_EINVAL
    assert call(n_pages=0) == E.TB_EINVAL
    assert call(kn=None) == E.TB_EINVAL
    assert call(Hq=36) == E.TB_EUNSUPPORTED
    assert call(d=256) == E.TB_EUNSUPPORTED
    need = _lib.tb_workspace_bytes(_lib.TB_OP_DECODE, 1, 0, 28, 4, 128, 0, 4 * 32)
    assert call(wsb=need - 1) == E.TB_EWORKSPACE
    assert b"tb_decode_attn_paged: workspace" in lib.tb_last_error()


def test_binding_refuses_cpu_tensors():
    import torch
    with pytest.raises(ValueError):
        _lib._dev(torch.zeros(3), "x")
