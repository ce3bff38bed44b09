"""ctypes binding of libtimebill.so (the C ABI declared in include/timebill.h).

Argument marshalling only: every step of the path runs in the HIP kernels.
The functions carry the C names and take torch tensors (device memory) plus
plain Python values; work is enqueued on the current torch stream.  There is
no fallback: without the built library every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtimebill.so")

TB_OK, TB_EINVAL, TB_EUNSUPPORTED, TB_EWORKSPACE, TB_EHIP, TB_EINTERNAL = range(6)
MAX_B = 64          # sequences per call (include/timebill.h: B <= 64)
TB_F32, TB_BF16 = 0, 1
TB_OP_SCORE, TB_OP_SELECT, TB_OP_COMPACT, TB_OP_DECODE, TB_OP_H2O = range(5)
V_TILE = 32          # rows per tile (and per page) of the compact caches; cap is a multiple

EXPORTED = ("tb_keep_count", "tb_last_error", "tb_workspace_bytes", "tb_score_window",
            "tb_score_window_avgpool", "tb_score_knorm", "tb_score_h2o", "tb_prefill_attn",
            "tb_select_topk", "tb_compact_kv_paged", "tb_decode_attn_paged", "tb_compact_kv", "tb_decode_attn", "tb_decode_attn_noalloc", "tb_ete_fit", "tb_wcet",
            "tb_alpha_star", "tb_response_length", "tb_predictor_length")

_lib = None


class TimebillError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"status {status}: {msg}")
        self.status = status


def load() -> ctypes.CDLL:
    """Load the library once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, dbl, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_double, ctypes.c_size_t
    p_i32 = ctypes.POINTER(ctypes.c_int32)
    p_dbl = ctypes.POINTER(ctypes.c_double)
    lib.tb_keep_count.argtypes = [i32, dbl, i32]
    lib.tb_keep_count.restype = i32
    lib.tb_last_error.argtypes = []
    lib.tb_last_error.restype = ctypes.c_char_p
    lib.tb_workspace_bytes.argtypes = [i32] * 8
    lib.tb_workspace_bytes.restype = sz
    lib.tb_score_window.argtypes = [vp, vp, i32, p_i32, i32, i32, i32, i32, i32, i32, i32,
                                    vp, vp, vp, sz, vp]
    lib.tb_score_window.restype = i32
    lib.tb_score_window_avgpool.argtypes = lib.tb_score_window.argtypes
    lib.tb_score_window_avgpool.restype = i32
    lib.tb_score_knorm.argtypes = [vp, i32, p_i32, i32, i32, i32, i32, i32, vp, vp]
    lib.tb_score_knorm.restype = i32
    lib.tb_score_h2o.argtypes = [vp, vp, i32, p_i32, i32, i32, i32, i32, i32, vp, vp, sz, vp]
    lib.tb_score_h2o.restype = i32
    lib.tb_prefill_attn.argtypes = [vp, vp, vp, i32, p_i32, i32, i32, i32, i32, i32, vp, i32, vp,
                                    vp]
    lib.tb_prefill_attn.restype = i32
    lib.tb_compact_kv_paged.argtypes = [vp, vp, vp, i32, p_i32, i32, i32, i32, i32, vp, vp, i32,
                                        vp, i32, vp, vp]
    lib.tb_compact_kv_paged.restype = i32
    lib.tb_decode_attn_paged.argtypes = [vp, vp, vp, vp, vp, i32, vp, i32, vp, i32, i32, i32, i32,
                                         i32, vp, vp, sz, vp]
    lib.tb_decode_attn_paged.restype = i32
    lib.tb_select_topk.argtypes = [vp, i32, p_i32, i32, i32, i32, p_dbl, vp, p_i32, vp, sz, vp]
    lib.tb_select_topk.restype = i32
    lib.tb_compact_kv.argtypes = [vp, vp, vp, i32, p_i32, i32, i32, i32, i32, i32, vp, vp, vp,
                                  vp, sz, vp]
    lib.tb_compact_kv.restype = i32
    lib.tb_decode_attn.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, vp, vp,
                                   sz, vp]
    lib.tb_decode_attn.restype = i32
    lib.tb_decode_attn_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32,
                                           vp, vp]
    lib.tb_decode_attn_noalloc.restype = i32
    lib.tb_ete_fit.argtypes = [p_dbl, p_dbl, i32, i32, p_dbl]
    lib.tb_ete_fit.restype = i32
    lib.tb_wcet.argtypes = [p_dbl, p_dbl, dbl, dbl, i32]
    lib.tb_wcet.restype = dbl
    lib.tb_alpha_star.argtypes = [p_dbl, p_dbl, dbl, i32, dbl, dbl, dbl, p_i32]
    lib.tb_alpha_star.restype = dbl
    lib.tb_response_length.argtypes = [i32, i32, i32, i32, p_i32]
    lib.tb_response_length.restype = i32
    lib.tb_predictor_length.argtypes = [p_dbl, p_dbl, dbl, ctypes.c_int64]
    lib.tb_predictor_length.restype = ctypes.c_int64
    _lib = lib
    return lib


def _check(status: int) -> None:
    if status != TB_OK:
        raise TimebillError(status, load().tb_last_error().decode())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return TB_BF16
    if t.dtype == torch.float32:
        return TB_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _dev(t: Optional[torch.Tensor], name: str, dtype=None) -> int:
    if t is None:
        return 0
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    return t.data_ptr()


def _stream(stream) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _i32_array(vals: Sequence[int]):
    return (ctypes.c_int32 * len(vals))(*[int(v) for v in vals])


def tb_keep_count(L: int, alpha: float, w: int) -> int:
    return int(load().tb_keep_count(int(L), float(alpha), int(w)))


def tb_workspace_bytes(op: int, B: int, Lmax: int, Hq: int, Hkv: int, d: int, w: int,
                       cap: int) -> int:
    return int(load().tb_workspace_bytes(op, B, Lmax, Hq, Hkv, d, w, cap))


def tb_score_window(q_win: torch.Tensor, k: torch.Tensor, L: Sequence[int], w: int, pool: int,
                    scores: torch.Tensor, raw_scores: Optional[torch.Tensor] = None,
                    ws: Optional[torch.Tensor] = None, stream=None, avgpool: bool = False) -> None:
    """q_win [B,Hq,w,d], k [B,Hkv,Lmax,d] (bf16/fp32); scores [B,Hkv,Lmax] fp32.
    avgpool=True calls tb_score_window_avgpool (mean instead of max)."""
    B, Hq, w_, d = q_win.shape
    _, Hkv, Lmax, d2 = k.shape
    if w_ != w or d2 != d or k.shape[0] != B or k.dtype != q_win.dtype:
        raise ValueError("q_win / k shapes or dtypes disagree")
    if tuple(scores.shape) != (B, Hkv, Lmax):
        raise ValueError("scores must be [B, Hkv, Lmax]")
    if raw_scores is not None and tuple(raw_scores.shape) != (B, Hkv, Lmax):
        raise ValueError("raw_scores must be [B, Hkv, Lmax]")
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    fn = load().tb_score_window_avgpool if avgpool else load().tb_score_window
    _check(fn(
        _dev(q_win, "q_win"), _dev(k, "k"), B, _i32_array(L), Lmax, Hq, Hkv, d, w, pool,
        _dtype_code(k), _dev(scores, "scores", torch.float32),
        _dev(raw_scores, "raw_scores", torch.float32), _dev(ws, "ws"), ws_bytes,
        _stream(stream)))


def tb_score_knorm(k: torch.Tensor, L: Sequence[int], w: int, scores: torch.Tensor,
                   stream=None) -> None:
    """k [B,Hkv,Lmax,d] (bf16/fp32) -> scores [B,Hkv,Lmax] fp32 = -||k_j|| (prefix)."""
    B, Hkv, Lmax, d = k.shape
    if tuple(scores.shape) != (B, Hkv, Lmax):
        raise ValueError("scores must be [B, Hkv, Lmax]")
    _check(load().tb_score_knorm(_dev(k, "k"), B, _i32_array(L), Lmax, Hkv, d, w,
                                 _dtype_code(k), _dev(scores, "scores", torch.float32),
                                 _stream(stream)))


def tb_score_h2o(q: torch.Tensor, k: torch.Tensor, L: Sequence[int], scores: torch.Tensor,
                 ws: torch.Tensor, stream=None) -> None:
    """q [B,Hq,Lmax,d] (all prompt queries), k [B,Hkv,Lmax,d] -> scores [B,Hkv,Lmax]
    fp32: the attention mass each key receives from every prompt query."""
    B, Hq, Lmax, d = q.shape
    _, Hkv, Lmax2, d2 = k.shape
    if Lmax2 != Lmax or d2 != d or k.shape[0] != B or k.dtype != q.dtype:
        raise ValueError("q / k shapes or dtypes disagree")
    if tuple(scores.shape) != (B, Hkv, Lmax):
        raise ValueError("scores must be [B, Hkv, Lmax]")
    _check(load().tb_score_h2o(_dev(q, "q"), _dev(k, "k"), B, _i32_array(L), Lmax, Hq, Hkv, d,
                               _dtype_code(k), _dev(scores, "scores", torch.float32),
                               _dev(ws, "ws"), ws.numel() * ws.element_size(), _stream(stream)))


def tb_prefill_attn(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, L: Sequence[int],
                    out: torch.Tensor, w: int = 0, window_stats: Optional[torch.Tensor] = None,
                    stream=None) -> None:
    """Causal GQA prefill attention: q [B,Hq,Lmax,d], k/v [B,Hkv,Lmax,d] (bf16) ->
    out [B,Hq,Lmax,d]; window_stats [B,Hq,w,2] fp32 gets (M, Z) of the last w rows."""
    B, Hq, Lmax, d = q.shape
    _, Hkv, Lmax2, d2 = k.shape
    if tuple(v.shape) != tuple(k.shape) or Lmax2 != Lmax or d2 != d or k.shape[0] != B:
        raise ValueError("q / k / v shapes disagree")
    if tuple(out.shape) != tuple(q.shape):
        raise ValueError("out must match q")
    if window_stats is not None and tuple(window_stats.shape) != (B, Hq, w, 2):
        raise ValueError("window_stats must be [B, Hq, w, 2]")
    _check(load().tb_prefill_attn(_dev(q, "q"), _dev(k, "k"), _dev(v, "v"), B, _i32_array(L),
                                  Lmax, Hq, Hkv, d, _dtype_code(q), _dev(out, "out"), w,
                                  _dev(window_stats, "window_stats", torch.float32),
                                  _stream(stream)))


def tb_select_topk(scores: torch.Tensor, L: Sequence[int], w: int, alpha: Sequence[float],
                   keep_idx: torch.Tensor, ws: Optional[torch.Tensor] = None,
                   stream=None) -> List[int]:
    """scores [B,Hkv,Lmax] fp32 -> keep_idx [B,Hkv,Lmax] int32; returns n_keep per sequence."""
    B, Hkv, Lmax = scores.shape
    if tuple(keep_idx.shape) != (B, Hkv, Lmax):
        raise ValueError("keep_idx must be [B, Hkv, Lmax]")
    n_keep = (ctypes.c_int32 * B)()
    alphas = (ctypes.c_double * B)(*[float(a) for a in alpha])
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(load().tb_select_topk(
        _dev(scores, "scores", torch.float32), B, _i32_array(L), Lmax, Hkv, w, alphas,
        _dev(keep_idx, "keep_idx", torch.int32), n_keep, _dev(ws, "ws"), ws_bytes,
        _stream(stream)))
    return list(n_keep)


def _dbl_array(vals: Sequence[float]):
    return (ctypes.c_double * len(vals))(*[float(v) for v in vals])


def tb_ete_fit(n: Sequence[float], t: Sequence[float], degree: int) -> List[float]:
    """Least-squares coefficients, highest power first ({p, q} or {a, b, c})."""
    coef = (ctypes.c_double * (degree + 1))()
    if load().tb_ete_fit(_dbl_array(n), _dbl_array(t), len(n), degree, coef) != 0:
        raise ValueError("tb_ete_fit: bad arguments or singular system")
    return list(coef)


def tb_wcet(prefill_abc: Sequence[float], step_pq: Sequence[float], n_x: float, alpha: float,
            n_hat_w: int) -> float:
    return float(load().tb_wcet(_dbl_array(prefill_abc), _dbl_array(step_pq), n_x, alpha,
                                n_hat_w))


def tb_alpha_star(prefill_abc: Sequence[float], step_pq: Sequence[float], n_x: float,
                  n_hat_w: int, budget: float, t_predict: float, alpha_max: float):
    """Returns (alpha*, feasible)."""
    feas = ctypes.c_int32(0)
    a = load().tb_alpha_star(_dbl_array(prefill_abc), _dbl_array(step_pq), n_x, n_hat_w, budget,
                             t_predict, alpha_max, ctypes.byref(feas))
    return float(a), bool(feas.value)


def tb_response_length(n_hat: int, bucket: int, k: int, n_max: int):
    """Returns (N_hat, N_hat_W) for predicted bucket index n_hat."""
    nh = ctypes.c_int32(0)
    nw = load().tb_response_length(int(n_hat), int(bucket), int(k), int(n_max), ctypes.byref(nh))
    if nw < 0:
        raise ValueError("tb_response_length: bad arguments")
    return int(nh.value), int(nw)


def _check_caches(k_cache, v_cache, B, Hkv, d):
    cap = k_cache.shape[2]
    if tuple(k_cache.shape) != (B, Hkv, cap, d):
        raise ValueError("k_cache must be [B, Hkv, cap, d]")
    if cap % V_TILE or tuple(v_cache.shape) != (B, Hkv, cap, d):
        raise ValueError("v_cache must be [B, Hkv, cap, d] with cap a multiple of 32")
    return cap


def tb_compact_kv(k: torch.Tensor, v: torch.Tensor, keep_idx: torch.Tensor,
                  n_keep: Sequence[int], k_cache: torch.Tensor, v_cache: torch.Tensor,
                  kv_len: torch.Tensor, stream=None) -> None:
    """k, v [B,Hkv,Lmax,d] -> k_cache, v_cache [B,Hkv,cap,d]; kv_len [B] int32
    set to n_keep."""
    B, Hkv, Lmax, d = k.shape
    if v.shape != k.shape:
        raise ValueError("k and v shapes disagree")
    cap = _check_caches(k_cache, v_cache, B, Hkv, d)
    if k_cache.dtype != k.dtype or v_cache.dtype != k.dtype or v.dtype != k.dtype:
        raise TypeError("k, v and caches must share a dtype")
    _check(load().tb_compact_kv(
        _dev(k, "k"), _dev(v, "v"), _dev(keep_idx, "keep_idx", torch.int32), B,
        _i32_array(n_keep), Lmax, Hkv, d, _dtype_code(k), cap, _dev(k_cache, "k_cache"),
        _dev(v_cache, "v_cache"), _dev(kv_len, "kv_len", torch.int32), None, 0,
        _stream(stream)))


def tb_decode_attn(q: torch.Tensor, k_new: Optional[torch.Tensor], v_new: Optional[torch.Tensor],
                   k_cache: torch.Tensor, v_cache: torch.Tensor, kv_len: torch.Tensor,
                   out: torch.Tensor, ws: torch.Tensor, stream=None) -> None:
    """q, out [B,Hq,d]; k_new, v_new [B,Hkv,d] or None; caches as in tb_compact_kv."""
    B, Hq, d = q.shape
    Hkv = k_cache.shape[1]
    cap = _check_caches(k_cache, v_cache, B, Hkv, d)
    if out.shape != q.shape:
        raise ValueError("out must match q")
    for t, name in ((k_new, "k_new"), (v_new, "v_new")):
        if t is not None and tuple(t.shape) != (B, Hkv, d):
            raise ValueError(f"{name} must be [B, Hkv, d]")
    if any(t is not None and t.dtype != q.dtype for t in (k_new, v_new, k_cache, v_cache, out)):
        raise TypeError("decode tensors must share a dtype")
    _check(load().tb_decode_attn(
        _dev(q, "q"), _dev(k_new, "k_new"), _dev(v_new, "v_new"), _dev(k_cache, "k_cache"),
        _dev(v_cache, "v_cache"), _dev(kv_len, "kv_len", torch.int32), B, Hq, Hkv, d, cap,
        _dtype_code(q), _dev(out, "out"), _dev(ws, "ws"), ws.numel() * ws.element_size(),
        _stream(stream)))


def tb_decode_attn_noalloc(q: torch.Tensor, k_new: Optional[torch.Tensor],
                           v_new: Optional[torch.Tensor], k_cache: torch.Tensor,
                           v_cache: torch.Tensor, kv_len: torch.Tensor, out: torch.Tensor,
                           stream=None) -> None:
    """tb_decode_attn with the library's scratch in place of a workspace."""
    B, Hq, d = q.shape
    Hkv = k_cache.shape[1]
    cap = _check_caches(k_cache, v_cache, B, Hkv, d)
    if out.shape != q.shape:
        raise ValueError("out must match q")
    for t, name in ((k_new, "k_new"), (v_new, "v_new")):
        if t is not None and tuple(t.shape) != (B, Hkv, d):
            raise ValueError(f"{name} must be [B, Hkv, d]")
    if any(t is not None and t.dtype != q.dtype for t in (k_new, v_new, k_cache, v_cache, out)):
        raise TypeError("decode tensors must share a dtype")
    _check(load().tb_decode_attn_noalloc(
        _dev(q, "q"), _dev(k_new, "k_new"), _dev(v_new, "v_new"), _dev(k_cache, "k_cache"),
        _dev(v_cache, "v_cache"), _dev(kv_len, "kv_len", torch.int32), B, Hq, Hkv, d, cap,
        _dtype_code(q), _dev(out, "out"), _stream(stream)))


class KVCache:
    """Compact caches of one layer plus the host-side lengths the library cannot see.

    Allocation happens here (torch device memory); every computation is a
    call into the library.  ``cap`` is rounded up to whole 32-row tiles; ``k``
    and ``v`` are row-major.  ``decode`` refuses an append past ``cap``.
    """

    def __init__(self, B: int, Hq: int, Hkv: int, cap: int, d: int, dtype: torch.dtype,
                 device="cuda"):
        cap = -(-cap // V_TILE) * V_TILE          # whole 32-row tiles
        self.B, self.Hq, self.Hkv, self.cap, self.d = B, Hq, Hkv, cap, d
        self.k = torch.empty((B, Hkv, cap, d), dtype=dtype, device=device)
        self.v = torch.empty((B, Hkv, cap, d), dtype=dtype, device=device)
        self.kv_len = torch.zeros((B,), dtype=torch.int32, device=device)
        nbytes = tb_workspace_bytes(TB_OP_DECODE, B, 0, Hq, Hkv, d, 0, cap)
        self.ws = torch.zeros((max(nbytes, 1),), dtype=torch.uint8, device=device)
        self.host_len = [0] * B

    def compact_from(self, k: torch.Tensor, v: torch.Tensor, keep_idx: torch.Tensor,
                     n_keep: Sequence[int], stream=None) -> None:
        if max(n_keep) > self.cap:
            raise ValueError("n_keep exceeds the cache capacity")
        tb_compact_kv(k, v, keep_idx, n_keep, self.k, self.v, self.kv_len, stream)
        self.host_len = list(n_keep)

    def decode(self, q, k_new, v_new, out, stream=None) -> None:
        if k_new is not None and max(self.host_len) + 1 > self.cap:
            raise ValueError("append would exceed the cache capacity")
        tb_decode_attn(q, k_new, v_new, self.k, self.v, self.kv_len, out, self.ws, stream)
        if k_new is not None:
            self.host_len = [n + 1 for n in self.host_len]


def tb_predictor_length(prefill_abc: Sequence[float], predict_abc: Sequence[float], n_x: float,
                        max_len: int) -> int:
    """Largest predictor input length N_p <= max_len whose predicted time fits
    within the predicted prefill time (-1: none fits)."""
    r = load().tb_predictor_length(_dbl_array(prefill_abc), _dbl_array(predict_abc), float(n_x),
                                   int(max_len))
    if r == -2:
        raise ValueError("tb_predictor_length: bad arguments")
    return int(r)



def _check_pools(k_pool, v_pool, block_table, dtype):
    n_pages, Hkv, t, d = k_pool.shape
    if t != V_TILE or tuple(v_pool.shape) != (n_pages, Hkv, V_TILE, d):
        raise ValueError("pools must be k_pool and v_pool [P, Hkv, 32, d]")
    if k_pool.dtype != dtype or v_pool.dtype != dtype:
        raise TypeError("pools must share the inputs' dtype")
    if block_table.dim() != 2:
        raise ValueError("block_table must be [B, max_pages]")
    return n_pages, Hkv, d, block_table.shape[1]


def tb_compact_kv_paged(k: torch.Tensor, v: torch.Tensor, keep_idx: torch.Tensor,
                        n_keep: Sequence[int], k_pool: torch.Tensor, v_pool: torch.Tensor,
                        block_table: torch.Tensor, kv_len: torch.Tensor, stream=None) -> None:
    """k, v [B,Hkv,Lmax,d] -> the pages block_table [B, max_pages] names in
    k_pool [P,Hkv,32,d] / v_pool [P,Hkv,d,32]; kv_len [B] int32 set to n_keep."""
    B, Hkv, Lmax, d = k.shape
    if v.shape != k.shape or v.dtype != k.dtype:
        raise ValueError("k and v disagree")
    n_pages, ph, pd, max_pages = _check_pools(k_pool, v_pool, block_table, k.dtype)
    if (ph, pd) != (Hkv, d) or block_table.shape[0] != B:
        raise ValueError("pool or block table shape does not match k")
    _check(load().tb_compact_kv_paged(
        _dev(k, "k"), _dev(v, "v"), _dev(keep_idx, "keep_idx", torch.int32), B,
        _i32_array(n_keep), Lmax, Hkv, d, _dtype_code(k), _dev(k_pool, "k_pool"),
        _dev(v_pool, "v_pool"), n_pages, _dev(block_table, "block_table", torch.int32),
        max_pages, _dev(kv_len, "kv_len", torch.int32), _stream(stream)))


def tb_decode_attn_paged(q: torch.Tensor, k_new: Optional[torch.Tensor],
                         v_new: Optional[torch.Tensor], k_pool: torch.Tensor,
                         v_pool: torch.Tensor, block_table: torch.Tensor, kv_len: torch.Tensor,
                         out: torch.Tensor, ws: torch.Tensor, stream=None) -> None:
    """q, out [B,Hq,d]; k_new, v_new [B,Hkv,d] or None; pools and table as in
    tb_compact_kv_paged (only the first B table rows and lengths are used)."""
    B, Hq, d = q.shape
    n_pages, Hkv, pd, max_pages = _check_pools(k_pool, v_pool, block_table, q.dtype)
    if pd != d or block_table.shape[0] < B or kv_len.numel() < B:
        raise ValueError("pool, block table or kv_len does not match q")
    if out.shape != q.shape or out.dtype != q.dtype:
        raise ValueError("out must match q")
    for t, name in ((k_new, "k_new"), (v_new, "v_new")):
        if t is not None and (tuple(t.shape) != (B, Hkv, d) or t.dtype != q.dtype):
            raise ValueError(f"{name} must be [B, Hkv, d] of q's dtype")
    _check(load().tb_decode_attn_paged(
        _dev(q, "q"), _dev(k_new, "k_new"), _dev(v_new, "v_new"), _dev(k_pool, "k_pool"),
        _dev(v_pool, "v_pool"), n_pages, _dev(block_table, "block_table", torch.int32),
        max_pages, _dev(kv_len, "kv_len", torch.int32), B, Hq, Hkv, d, _dtype_code(q),
        _dev(out, "out"), _dev(ws, "ws"), ws.numel() * ws.element_size(), _stream(stream)))
