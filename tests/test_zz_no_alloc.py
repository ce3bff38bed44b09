"""The decode entry point that allocates nothing (library-held scratch in
place of a workspace) against tb_decode_attn: two calls in a row on one GPU,
the second with a smaller input, must give bit-identical outputs, caches and
lengths (same kernels and launch plan; only where the partials live differs).
"""
import pytest
import torch

from paper_2512_21859_amd import _lib

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU in this container")
    _lib.load()
    torch.cuda.init()


def _pair(seed, B, Hq, Hkv, d, cap, lens, dtype):
    """Two identical caches (one per entry point) filled with seeded values."""
    g = torch.Generator().manual_seed(seed)
    kc = torch.randn((B, Hkv, cap, d), generator=g).to(dtype)
    vc = torch.randn((B, Hkv, cap, d), generator=g).to(dtype)
    caches = []
    for _ in range(2):
        c = _lib.KVCache(B, Hq, Hkv, cap, d, dtype)
        c.k.copy_(kc)
        c.v.copy_(vc)
        c.kv_len.copy_(torch.tensor(lens, dtype=torch.int32))
        c.host_len = list(lens)
        caches.append(c)
    return caches


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_noalloc_equals_workspace_call(dtype):
    # (B, Hq, Hkv, d, cap, lens, steps): the second call is smaller
    cases = [(2, 28, 4, 128, 8448, [8000, 3100], 3), (1, 8, 2, 64, 640, [300], 2)]
    for i, (B, Hq, Hkv, d, cap, lens, T) in enumerate(cases):
        print(f"\n[case] noalloc call {i}: dtype={dtype} B={B} Hq={Hq} Hkv={Hkv} d={d} "
              f"cap={cap} lens={lens} steps={T}", flush=True)
        assert _lib.tb_workspace_bytes(_lib.TB_OP_DECODE, B, 0, Hq, Hkv, d, 0, cap) \
            <= 16 << 20
        c_ws, c_sc = _pair(100 + i, B, Hq, Hkv, d, cap, lens, dtype)
        g = torch.Generator().manual_seed(200 + i)
        q = torch.randn((T, B, Hq, d), generator=g).to(dtype).to(DEV)
        kn = torch.randn((T, B, Hkv, d), generator=g).to(dtype).to(DEV)
        vn = torch.randn((T, B, Hkv, d), generator=g).to(dtype).to(DEV)
        o_ws = torch.empty((T, B, Hq, d), dtype=dtype, device=DEV)
        o_sc = torch.full((T, B, Hq, d), float("nan"), dtype=dtype, device=DEV)
        for t in range(T):
            _lib.tb_decode_attn(q[t], kn[t], vn[t], c_ws.k, c_ws.v, c_ws.kv_len, o_ws[t],
                                c_ws.ws)
            _lib.tb_decode_attn_noalloc(q[t], kn[t], vn[t], c_sc.k, c_sc.v, c_sc.kv_len,
                                        o_sc[t])
        torch.cuda.synchronize()
        assert torch.equal(o_ws, o_sc), f"call {i}: outputs differ"
        assert torch.equal(c_ws.kv_len, c_sc.kv_len)
        assert c_sc.kv_len.cpu().tolist() == [n + T for n in lens]
        assert torch.equal(c_ws.k, c_sc.k) and torch.equal(c_ws.v, c_sc.v)
