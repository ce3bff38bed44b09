"""Benchmark of the eviction + decode hot path on one MI355X.

Headline workload: a 28-layer stack with the Qwen2.5-7B attention shape
(28 query / 4 KV heads of dimension 128, bf16), a prompt of L = 32768 tokens
(the paper's context), independent random K/V per layer, observation window
32, max-pool 7, swept over the eviction ratios alpha = k/20, k = 0..19, with
128 decode tokens per ratio.  Inputs are seeded synthetic tensors already
resident in HBM when timing starts.

One step = for every alpha: evict every layer (score each layer's window,
then select and compact all 28 layers in one call each, the layers stacked
on the batch axis: once per request, as after a prefill), then 128 decode
tokens, one
token being the decode step (append + attention) of all 28 layers in order,
replayed from a HIP graph captured once per ratio.  The metric is decode
tokens per second over the whole step (eviction included); per-ratio rows
give the eviction time, the time per token and the achieved bandwidth, and
the per-token time is fitted with the execution-time model's decode-step form
t = p N_kv + q.

The roofline entry is for the decode call (tb_decode_attn: the split-K partial
kernel decode_mfma_kernel and its merge kernel), the dominant work:
algorithmic bytes per call (K and V rows of the cache plus q, the new K/V row
and the output) divided by the average call duration, measured with HIP
events recorded on the stream the graphs replay on (the gaps between the two
kernels included).  The CPU baseline is the float64 oracle on this host, on a
bounded sample of the same workload.
"""
import os

# The CPU baseline's BLAS threads: the host's CPUs available to this process,
# capped by a thread count the environment already sets; fixed before numpy
# (imported by torch) loads its thread pools.
_HOST_CPUS = len(os.sched_getaffinity(0))
_BLAS_THREADS = min(_HOST_CPUS, int(os.environ.get("OMP_NUM_THREADS", _HOST_CPUS) or _HOST_CPUS))
for _v in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
    os.environ[_v] = str(_BLAS_THREADS)

import argparse
import json
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def _parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="minimum CPU time of the oracle baseline sample")
    ap.add_argument("--no-single", action="store_true",
                    help="skip the single-layer L=8192 ratio sweep (and its cold-cache run)")
    ap.add_argument("--no-long-context", action="store_true",
                    help="skip the supplementary long-context decode measurement")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the 2 GiB read / copy bandwidth ceilings")
    ap.add_argument("--no-prefill", action="store_true",
                    help="skip the prefill-attention sweep")
    ap.add_argument("--no-scorers", action="store_true",
                    help="skip the scorer-variant timings")
    ap.add_argument("--no-paged", action="store_true",
                    help="skip the paged-cache batch and serving-stream measurements")
    ap.add_argument("--only", choices=("headline", "single", "long", "ceiling", "scorers",
                                       "prefill", "paged", "counters"),
                    help="run one measurement alone and print its JSON (for profiling that "
                         "workload by itself; 'headline' is the timed sweep without the "
                         "CPU baseline)")
    ap.add_argument("--tokens", type=int, default=None,
                    help="decode tokens per ratio in the headline sweep (default: the "
                         "workload's 128; fewer only for counter runs, which record per-call "
                         "figures)")
    ap.add_argument("--pmc-calibration", action="store_true",
                    help="first copy 512 MiB device-to-device twice (a kernel of known "
                         "traffic for scaling hardware byte counters)")
    return ap.parse_args()


def _decode_bytes(Hq, Hkv, d, n_rows, esz=2):
    """Algorithmic HBM bytes of one decode launch over n_rows cached rows."""
    return (2 * Hkv * n_rows * d + 2 * Hq * d + 2 * Hkv * d) * esz


def _evict_bytes(Hq, Hkv, d, L, w, n_keep, esz=2):
    score = Hkv * L * d * esz + Hq * w * d * esz + Hkv * (L - w) * 4
    select = Hkv * (L - w) * 4 + Hkv * n_keep * 4
    compact = 2 * 2 * Hkv * n_keep * d * esz + Hkv * n_keep * 4
    return score + select + compact


def code_sha256(text):
    """sha256 of a C++ source with its comments and whitespace removed, so
    that edits to comments alone do not count as a change of the code."""
    import hashlib
    import re
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return hashlib.sha256("".join(text.split()).encode()).hexdigest()


def measured_traffic():
    """HBM bytes per decode call of the headline sweep from the committed counter
    runs, or None when the decode kernels or their launch plan have changed
    since the counters were taken (the record holds code_sha256 of each source
    it depends on)."""
    path = os.path.join(ROOT, "profiles", "decode_traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f)
        for src, sha in rec["sources_code_sha256"].items():
            with open(os.path.join(ROOT, src)) as f:
                if code_sha256(f.read()) != sha:
                    return None
    except (OSError, KeyError, ValueError, AttributeError):
        return None
    return rec["traffic_bytes_per_call"]


def cpu_baseline(min_seconds):
    """The float64 oracle on this host, on a bounded sample of the headline
    workload: whole evictions (window scores, pooling, selection, compaction)
    of layers 0, 1, ... and decode steps 0, 16, ..., 112, 127 of those layers at
    ratios spread over the sweep, until min_seconds have passed.  Scaled to the
    whole sweep: every ratio's eviction of all 28 layers costs the sampled mean
    eviction, and a decode step is fitted linearly in the retained length from
    the sampled steps; tokens/s = 20 * 128 tokens / that total."""
    import numpy as np
    from oracle import timebill_oracle as O
    from paper_2512_21859_amd import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:       # pragma: no cover - reporting only
        threads = _BLAS_THREADS
    wl = synth.WORKLOADS[3]
    L, w, pool, T, nl = wl.L, wl.w, wl.pool, wl.T, wl.layers
    check = sorted(set(range(0, T, 16)) | {T - 1})
    sample_alphas = [wl.alphas[i] for i in (0, 10, 19, 5, 15, 2, 17)]
    evict_s, steps = [], []          # eviction seconds; (retained rows, seconds) per step
    t0 = time.perf_counter()
    layers_done, alphas_done = 0, []
    for layer in range(nl):
        pr = synth.make_prompt(wl, layer)
        dc = synth.make_decode(wl, layer)
        q64, k64, v64 = (pr[x][0].double().numpy() for x in ("q_win", "k", "v"))
        qs, kn, vn = (dc[x][:, 0].double().numpy() for x in ("q", "k_new", "v_new"))
        for a in sample_alphas:
            c0 = time.perf_counter()
            pooled = O.max_pool(O.window_scores(q64, k64, L, w), pool)
            nk = O.keep_count(L, a, w)
            keep = [O.select_keep(pooled[g], L, w, nk) for g in range(k64.shape[0])]
            kc = np.stack([O.compact(k64[g], v64[g], keep[g])[0] for g in range(len(keep))])
            vc = np.stack([O.compact(k64[g], v64[g], keep[g])[1] for g in range(len(keep))])
            evict_s.append(time.perf_counter() - c0)
            alphas_done.append(a)
            for t in check:
                c1 = time.perf_counter()
                O.decode_sequence(qs, kn, vn, kc, vc, steps=[t])
                steps.append((nk + t + 1, time.perf_counter() - c1))
            if time.perf_counter() - t0 >= min_seconds:
                break
        layers_done = layer + 1
        if time.perf_counter() - t0 >= min_seconds:
            break
    wall = time.perf_counter() - t0
    x = np.array([n for n, _ in steps], dtype=np.float64)
    y = np.array([s for _, s in steps], dtype=np.float64)
    slope, icpt = np.polyfit(x, y, 1) if np.ptp(x) > 0 else (0.0, float(y.mean()))
    ev_mean = float(np.mean(evict_s))
    total = 0.0
    for a in wl.alphas:
        nk = O.keep_count(L, a, w)
        total += nl * ev_mean + nl * sum(slope * (nk + t + 1) + icpt for t in range(T))
    tokens = len(wl.alphas) * T
    return {"value": tokens / total, "unit": "tokens/s", "cores": int(threads),
            "host_cpus": _HOST_CPUS, "blas_threads": _BLAS_THREADS, "kind": "oracle",
            "stage_ms": {"eviction_per_layer": round(ev_mean * 1e3, 1),
                         "decode_step_per_layer_at_32768_rows": round(
                             (slope * 32768 + icpt) * 1e3, 2)},
            "sample": (f"float64 numpy oracle on the host, {wall:.1f} s of CPU work: "
                       f"{len(evict_s)} whole evictions of one layer (window scores, "
                       f"pooling, selection, compaction) over {layers_done} layer(s) at "
                       f"ratios {sorted(set(alphas_done))}, and "
                       f"{len(steps)} single decode steps (steps {check} of each); scaled to "
                       f"the whole sweep (20 ratios x 28 layers x 128 tokens) with the mean "
                       f"eviction and a least-squares line of step time against retained "
                       f"length")}


def long_context(torch, _lib, synth, Evictor, dev, steps=64, alpha=0.5):
    """Supplementary: decode at the long-context shape (L = 131072, 32 q / 8 kv
    heads, alpha = 0.5, ~65.5k retained rows per head, ~268 MB of K/V per step),
    where a step is bandwidth-bound rather than latency-bound."""
    wl = synth.WORKLOADS[5]
    B, Hq, Hkv, d, w, L = wl.B, wl.Hq, wl.Hkv, wl.d, wl.w, wl.L
    pr = synth.make_prompt(wl)
    dc = synth.make_decode(wl, T=steps)
    q_win, k, v = (pr[x].to(dev) for x in ("q_win", "k", "v"))
    qd, knd, vnd = (dc[x].to(dev) for x in ("q", "k_new", "v_new"))
    del pr
    stream = torch.cuda.current_stream()
    ev = Evictor(B, L, Hq, Hkv, d, w, wl.pool, device=dev)
    nk = _lib.tb_keep_count(L, alpha, w)
    cache = _lib.KVCache(B, Hq, Hkv, nk + steps, d, wl.dtype, device=dev)
    out = torch.empty((steps, B, Hq, d), dtype=wl.dtype, device=dev)
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    ev.evict(q_win, k, v, [L], [alpha], cache, stream)          # warm-up
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    cs = torch.cuda.Stream()
    with torch.cuda.graph(g, stream=cs):
        for t in range(steps):
            _lib.tb_decode_attn(qd[t], knd[t], vnd[t], cache.k, cache.v, cache.kv_len, out[t],
                                cache.ws, stream=cs)
    torch.cuda.synchronize()
    ev_ms, de_ms = [], []
    for _ in range(3):
        e0.record(stream)
        ev.evict(q_win, k, v, [L], [alpha], cache, stream)
        e1.record(stream)
        g.replay()
        e2.record(stream)
        torch.cuda.synchronize()
        ev_ms.append(e0.elapsed_time(e1))
        de_ms.append(e1.elapsed_time(e2))
    ev_t, de_t = min(ev_ms), min(de_ms)
    sc_t = _best_ms(torch, lambda: ev.score(q_win, k, [L], stream))
    se_t = _best_ms(torch, lambda: ev.select([L], [alpha], stream))
    co_t = _best_ms(torch, lambda: cache.compact_from(k, v, ev.keep_idx, [nk], stream))
    dbytes = sum(_decode_bytes(Hq, Hkv, d, nk + t + 1) for t in range(steps)) / steps
    per_step_us = de_t * 1e3 / steps
    cbytes = 2 * 2 * Hkv * nk * d * 2
    return {
        "workload": "bf16, B=1, L=131072, 32 q / 8 kv heads, d=128, w=64, pool 7, "
                    f"alpha={alpha}, {steps} decode steps",
        "n_keep": nk,
        "decode_us_per_step": round(per_step_us, 2),
        "decode_GBps": round(dbytes / (per_step_us * 1e-6) / 1e9, 1),
        "decode_frac_of_8TBps": round(dbytes / (per_step_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
        "bytes_per_step": round(dbytes),
        "evict_us": round(ev_t * 1e3, 1),
        "score_us": round(sc_t * 1e3, 1),
        "select_us": round(se_t * 1e3, 1),
        "compact_us": round(co_t * 1e3, 1),
        "compaction_bytes": cbytes,
        "compact_GBps": round(cbytes / (co_t * 1e-3) / 1e9, 1),
        "compact_frac_of_8TBps": round(cbytes / (co_t * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "timing": "best of 3: HIP events around the eviction and around a graph of the decode steps",
    }


def _best_ms(torch, fn, reps=3, stream=None):
    """Best of ``reps`` HIP-event timings of fn() on the current stream, in ms."""
    stream = torch.cuda.current_stream() if stream is None else stream
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    best = float("inf")
    for _ in range(reps):
        e0.record(stream)
        fn()
        e1.record(stream)
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1))
    return best


def hbm_ceiling(torch, dev, nbytes=2 << 30):
    """Practical bandwidth ceilings over 2 GiB buffers, best of 5: a streaming
    read (the benchmark's own probe kernel, libtbbench.so: 16-byte
    nontemporal loads, grid sizes 1-16 blocks per CU tried) and a
    device-to-device copy (torch copy_)."""
    import ctypes
    x = torch.ones((nbytes // 4,), dtype=torch.float32, device=dev)
    y = torch.empty_like(x)
    y.copy_(x)
    torch.cuda.synchronize()
    cp = _best_ms(torch, lambda: y.copy_(x), reps=5)
    del y
    probe = ctypes.CDLL(os.path.join(ROOT, "paper_2512_21859_amd", "libtbbench.so"))
    probe.tbb_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                      ctypes.c_int, ctypes.c_void_p]
    probe.tbb_stream_read.restype = ctypes.c_int
    sink = torch.zeros((16 * 256,), dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()
    rd_best, rd_blocks = float("inf"), 0
    for blocks in (256, 512, 1024, 2048, 4096):
        def run():
            if probe.tbb_stream_read(x.data_ptr(), nbytes, sink.data_ptr(), blocks,
                                     stream.cuda_stream) != 0:
                raise RuntimeError("stream-read probe failed")
        run()
        t = _best_ms(torch, run, reps=5)
        if t < rd_best:
            rd_best, rd_blocks = t, blocks
    by_size = read_floor_by_size(torch, probe, x, sink)
    del x, sink
    torch.cuda.empty_cache()
    return {"read_GBps": round(nbytes / (rd_best * 1e-3) / 1e9, 1),
            "read_blocks": rd_blocks,
            "copy_GBps": round(2 * nbytes / (cp * 1e-3) / 1e9, 1),
            "bytes": nbytes,
            "how": "streaming-read probe kernel (16-byte nontemporal loads, best grid) and "
                   "torch copy_ (read + write) over 2 GiB buffers, HIP events, best of 5",
            "read_by_size": by_size}


def read_floor_by_size(torch, probe, x, sink, sizes_mib=(4, 8, 16, 32, 64, 128, 256)):
    """The streaming-read probe at the sizes one decode or compaction call
    moves (64 MiB ~ one layer's K and V at L = 32768), launched back to back
    from a graph over disjoint windows of the 2 GiB buffer (at least 1 GiB per
    replay, so the 256 MB last-level cache holds none of it): the time per
    launch is what a single launch that only streams its bytes costs,
    dispatch and ramp included.  Best grid of 256 / 512 / 1024 blocks, best
    of 5 replays."""
    total = x.numel() * x.element_size()
    rows = []
    for mib in sizes_mib:
        size = mib << 20
        n = max(16, -(-(1 << 30) // size))
        if n * size > total:
            n = total // size
        best = (float("inf"), 0)
        for blocks in (256, 512, 1024):
            cs = torch.cuda.Stream()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=cs):
                for i in range(n):
                    if probe.tbb_stream_read(x.data_ptr() + i * size, size, sink.data_ptr(), blocks,
                                             cs.cuda_stream) != 0:
                        raise RuntimeError("stream-read probe failed")
            g.replay()
            torch.cuda.synchronize()
            t = _best_ms(torch, g.replay, reps=5) / n
            if t < best[0]:
                best = (t, blocks)
            del g
        rows.append({"MiB": mib, "us_per_launch": round(best[0] * 1e3, 2), "blocks": best[1],
                     "GBps": round(size / (best[0] * 1e-3) / 1e9, 1),
                     "frac_of_8TBps": round(size / (best[0] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)})
    return rows


FP64_PEAK_TFLOPS = 78.6


def mfma_ceiling(torch, dev):
    """Practical matrix-core rates, best of 5 over grids of 1-8 blocks of 4
    waves per CU: the benchmark's probe kernel (libtbbench.so) runs eight
    independent accumulation chains per wave on register operands for the
    float64 16x16x4 shape (the window scorer's products) and the bf16
    16x16x32 shape (the prefill's and decode's products)."""
    import ctypes
    probe = ctypes.CDLL(os.path.join(ROOT, "paper_2512_21859_amd", "libtbbench.so"))
    probe.tbb_mfma_peak.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                    ctypes.c_void_p]
    probe.tbb_mfma_peak.restype = ctypes.c_int
    stream = torch.cuda.current_stream()
    out = {}
    # (kind, flops per instruction, iterations: about 1-2 ms at the datasheet peak
    # on the largest grid)
    for name, kind, flops, iters, peak in (("fp64_16x16x4", 0, 16 * 16 * 4 * 2, 1200,
                                            FP64_PEAK_TFLOPS),
                                           ("bf16_16x16x32", 1, 16 * 16 * 32 * 2, 4000,
                                            BF16_PEAK_TFLOPS)):
        best_rate, best_blocks = 0.0, 0
        for per_cu in (1, 2, 4, 8):
            blocks = 256 * per_cu
            sink = torch.empty((blocks * 256,), dtype=torch.float64, device=dev)

            def run():
                if probe.tbb_mfma_peak(kind, blocks, iters, sink.data_ptr(), stream.cuda_stream) != 0:
                    raise RuntimeError("matrix-core probe failed")
            run()
            t = _best_ms(torch, run, reps=5)
            rate = blocks * 4 * iters * 8 * flops / (t * 1e-3) / 1e12
            if rate > best_rate:
                best_rate, best_blocks = rate, blocks
            del sink
        out[name] = {"TFLOPs": round(best_rate, 1), "blocks": best_blocks,
                     "frac_of_datasheet": round(best_rate / peak, 4)}
    out["how"] = ("probe kernel: 8 independent accumulation chains per wave on register "
                  "operands, 256 threads per block, best grid and best of 5 (HIP events)")
    return out


def cold_decode(torch, _lib, Evictor, dev, wl, q_win, k, v, qd, knd, vnd,
                target_bytes=1 << 30):
    """Decode at ratio 0 for the L = 8192 workload with the step's cache
    rotated over enough copies (>= 1 GiB in total) that every step reads its
    cache from HBM rather than the 256 MB last-level cache."""
    B, Hq, Hkv, d, w, L, T = wl.B, wl.Hq, wl.Hkv, wl.d, wl.w, wl.L, wl.T
    per_cache = 2 * Hkv * (L + T) * d * 2
    R = -(-target_bytes // per_cache)
    ev = Evictor(B, L, Hq, Hkv, d, w, wl.pool, device=dev)
    caches = [_lib.KVCache(B, Hq, Hkv, L + T, d, wl.dtype, device=dev) for _ in range(R)]
    out = torch.empty((T, B, Hq, d), dtype=wl.dtype, device=dev)
    stream = torch.cuda.current_stream()

    def reset():
        for c in caches:
            ev.evict(q_win, k, v, [L], [0.0], c, stream)

    reset()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    cs = torch.cuda.Stream()
    with torch.cuda.graph(g, stream=cs):
        for t in range(T):
            c = caches[t % R]
            _lib.tb_decode_attn(qd[t], knd[t], vnd[t], c.k, c.v, c.kv_len, out[t], c.ws,
                                stream=cs)
    torch.cuda.synchronize()
    best = float("inf")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for _ in range(3):
        reset()
        e0.record(stream)
        g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1))
    # rows attended at step t: L + (number of earlier appends to that cache) + 1
    dbytes = sum(_decode_bytes(Hq, Hkv, d, L + t // R + 1) for t in range(T))
    us = best * 1e3 / T
    del caches, ev
    torch.cuda.empty_cache()
    return {"workload": f"bf16, B=1, L={L}, 28 q / 4 kv heads, d=128, ratio 0, {T} decode "
                        f"steps rotating over {R} caches ({R * per_cache / 2**30:.2f} GiB)",
            "decode_us_per_step": round(us, 3),
            "decode_GBps": round(dbytes / T / (us * 1e-6) / 1e9, 1),
            "decode_frac_of_8TBps": round(dbytes / T / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "timing": "best of 3: HIP events around a graph of the decode steps"}


def scorer_variants(torch, _lib, synth, Evictor, dev, reps=10):
    """Supplementary: scoring time of each scorer (max-pool window scores, the
    mean-pooled variant, KNorm, and at L = 8192 H2O) at the L = 8192, one
    layer of the L = 32768 and the L = 131072 shapes, from a graph of `reps`
    scoring calls (2 for H2O); KNorm's bandwidth counts one read of K plus the
    fp32 scores written; the window scorers' fp64 rate counts the window
    products 2 Hq w L d over the whole scoring call."""
    out = {}
    for wid in (2, 3, 5):
        wl = synth.WORKLOADS[wid]
        B, Hq, Hkv, d, w, L = wl.B, wl.Hq, wl.Hkv, wl.d, wl.w, wl.L
        pr = synth.make_prompt(wl)
        q_win, k = pr["q_win"].to(dev), pr["k"].to(dev)
        del pr
        # H2O needs the queries of every prompt position and ~2 Hq L^2 d float64
        # flops per call: measured at L = 8192 only (L = 131072 would be 141 TFLOP)
        scorers = ("snapkv", "snapkv_avg", "knorm") + (("h2o",) if L <= 8192 else ())
        q_all = synth.make_queries(wl).to(dev) if "h2o" in scorers else None
        row = {}
        for scorer in scorers:
            ev = Evictor(B, L, Hq, Hkv, d, w, wl.pool, device=dev, scorer=scorer)
            qin = q_all if scorer == "h2o" else q_win
            n = 2 if scorer == "h2o" else reps
            cs = torch.cuda.Stream()
            ev.score(qin, k, [L], cs)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=cs):
                for _ in range(n):
                    ev.score(qin, k, [L], cs)
            torch.cuda.synchronize()
            us = _best_ms(torch, g.replay) * 1e3 / n
            row[scorer] = {"us": round(us, 2)}
            if scorer in ("snapkv", "snapkv_avg"):
                flops = 2 * Hq * w * L * d
                row[scorer]["fp64_TFLOPs"] = round(flops / (us * 1e-6) / 1e12, 2)
            if scorer == "knorm":
                nbytes = Hkv * L * d * 2 + Hkv * (L - w) * 4
                row[scorer]["GBps"] = round(nbytes / (us * 1e-6) / 1e9, 1)
                row[scorer]["frac_of_8TBps"] = round(nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)
            if scorer == "h2o":
                # two passes over the causal pairs (i >= j), 2 d flops per pair and head
                flops = 2 * 2 * Hq * d * (L * (L + 1) // 2)
                row[scorer]["fp64_TFLOPs"] = round(flops / (us * 1e-6) / 1e12, 2)
                row[scorer]["frac_of_78.6"] = round(flops / (us * 1e-6) / 1e12 / 78.6, 4)
            del g, ev
        del q_all
        out[f"L{L}_{Hq}q{Hkv}kv"] = row
        del q_win, k
        torch.cuda.empty_cache()
    out["timing"] = f"best of 3 replays of a graph of {reps} scoring calls, divided by {reps}"
    return out


BF16_PEAK_TFLOPS = 2500.0


PREFILL_LENGTHS = (256, 512, 1024) + tuple(2048 * k for k in range(1, 17))


def prefill_sweep(torch, _lib, synth, dev, lengths=PREFILL_LENGTHS):
    """Supplementary: causal prefill attention (28 q / 4 kv heads, d = 128, bf16)
    at 19 prompt lengths over the paper's profiling range (256 .. 32768: every
    2048 plus three short prompts), the time fitted with the paper's
    prefill-phase form a N^2 + b N + c (tb_ete_fit, degree 2; attention only,
    where the paper times the whole model's prefill) and the bf16 matrix-core
    rate (causal flops 4 Hq d N(N+1)/2)."""
    Lmax = max(lengths)
    wl = synth.custom(2000, torch.bfloat16, 1, [Lmax], 28, 4, 128, 32, 7, 1)
    pr = synth.make_prompt(wl, L=[Lmax])
    q = synth.make_queries(wl, L=[Lmax]).to(dev)
    k, v = pr["k"].to(dev), pr["v"].to(dev)
    del pr
    out = torch.empty_like(q)
    Hq, d = wl.Hq, wl.d
    rows = []
    for n in lengths:
        reps = max(2, min(20, (1 << 25) // (n * n // 64)))
        cs = torch.cuda.Stream()
        _lib.tb_prefill_attn(q, k, v, [n], out, stream=cs)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cs):
            for _ in range(reps):
                _lib.tb_prefill_attn(q, k, v, [n], out, stream=cs)
        torch.cuda.synchronize()
        us = _best_ms(torch, g.replay) * 1e3 / reps
        flops = 4 * Hq * d * (n * (n + 1) // 2)
        rows.append({"n": n, "us": round(us, 2), "TFLOPs": round(flops / (us * 1e-6) / 1e12, 1),
                     "frac_of_bf16_peak": round(flops / (us * 1e-6) / 1e12 / BF16_PEAK_TFLOPS, 4)})
        del g
    a, b_, c = _lib.tb_ete_fit([r["n"] for r in rows], [r["us"] for r in rows], 2)
    pred = [a * r["n"] ** 2 + b_ * r["n"] + c for r in rows]
    ape = [abs(f - r["us"]) / r["us"] for f, r in zip(pred, rows)]
    mape = 100.0 * sum(ape) / len(rows)
    long_ape = [e for e, r in zip(ape, rows) if r["n"] >= 2048]
    mape_long = 100.0 * sum(long_ape) / len(long_ape)
    del q, k, v, out
    torch.cuda.empty_cache()
    return {"workload": "causal prefill attention, bf16, B=1, 28 q / 4 kv heads, d=128",
            "per_length": rows,
            "prefill_time_fit": {"a_us_per_n2": a, "b_us_per_n": b_, "c_us": c, "mape_pct": mape,
                                 "mape_pct_n_ge_2048": mape_long, "points": len(rows),
                                 "note": "attention only (the paper's 1.22% is for a whole-model "
                                         "prefill on an A40: context, not a target)"},
            "timing": "best of 3 replays of a graph of repeated calls (2..20 by length)"}


def _pct(xs, q):
    xs = sorted(xs)
    return xs[min(len(xs) - 1, int(q * (len(xs) - 1) + 0.5))]


LLC_BYTES = 256 << 20      # MI355X last-level (Infinity) cache


def headline(torch, _lib, synth, Evictor, dev, steps, warmup, tokens=None):
    """The 28-layer L = 32768 sweep (module docstring).  Returns the headline
    fields of the JSON line."""
    from paper_2512_21859_amd.pipeline import StackEvictor
    wl = synth.WORKLOADS[3]
    T, nl = (wl.T if tokens is None else tokens), wl.layers
    B, Hq, Hkv, d, w, L = wl.B, wl.Hq, wl.Hkv, wl.d, wl.w, wl.L
    # the layers' prompt tensors and caches are stacked layer-major on the
    # batch axis ([nl * B, ...]); each layer's entries are views of its rows
    stack = {}
    lay = [dict() for _ in range(nl)]
    for layer in range(nl):
        pr = synth.make_prompt(wl, layer)
        dc = synth.make_decode(wl, layer, T=T)
        for x in ("q_win", "k", "v"):
            if x not in stack:
                stack[x] = torch.empty((nl * B,) + tuple(pr[x].shape[1:]), dtype=pr[x].dtype,
                                       device=dev)
            stack[x][layer * B:(layer + 1) * B].copy_(pr[x])
            lay[layer][x] = stack[x][layer * B:(layer + 1) * B]
        lay[layer].update({x: dc[x].to(dev) for x in ("q", "k_new", "v_new")})
        del pr, dc
    ev = Evictor(B, L, Hq, Hkv, d, w, wl.pool, device=dev)
    sev = StackEvictor(nl, B, L, Hq, Hkv, d, w, wl.pool, device=dev)
    stream = torch.cuda.current_stream()
    alphas = list(wl.alphas)
    n_keep = {a: _lib.tb_keep_count(L, a, w) for a in alphas}
    caches = {a: _lib.KVCache(nl * B, Hq, Hkv, n_keep[a] + T, d, wl.dtype, device=dev)
              for a in alphas}
    out = torch.empty((T, nl, B, Hq, d), dtype=wl.dtype, device=dev)

    def evict_all(a):
        # every layer scored on its own, then one selection and one compaction
        # for the stack (a layer's selection alone keeps Hkv CUs busy); one
        # stream for everything: spreading the layers' evictions over side
        # streams measured slower (every later decode dispatch slowed down)
        sev.evict(stack["q_win"], stack["k"], stack["v"], [L] * B, [a] * B, caches[a], stream)

    # one graph per ratio: T tokens x 28 layers of decode calls (lengths live on
    # the device, so every replay after an eviction starts from n_keep)
    graphs = {}
    cap_stream = torch.cuda.Stream()
    for a in alphas:
        evict_all(a)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cap_stream):
            c = caches[a]
            for t in range(T):
                for layer in range(nl):
                    x, r = lay[layer], slice(layer * B, (layer + 1) * B)
                    _lib.tb_decode_attn(x["q"][t], x["k_new"][t], x["v_new"][t], c.k[r], c.v[r],
                                        c.kv_len[r], out[t, layer], c.ws, stream=cap_stream)
        graphs[a] = g
    torch.cuda.synchronize()

    def step(evs=None):
        for i, a in enumerate(alphas):
            if evs is not None:
                evs[3 * i].record(stream)
            evict_all(a)
            if evs is not None:
                evs[3 * i + 1].record(stream)
            graphs[a].replay()
            if evs is not None:
                evs[3 * i + 2].record(stream)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    n_al = len(alphas)
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(3 * n_al)]
              for _ in range(steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record(stream)
    for s_ in range(steps):
        step(events[s_])
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = t_start.elapsed_time(t_end)

    rows = []
    hbm_bytes = hbm_ms = hbm_calls = 0.0
    all_bytes = all_ms = 0.0
    for i, a in enumerate(alphas):
        ev_ms = [events[k][3 * i].elapsed_time(events[k][3 * i + 1]) for k in range(steps)]
        de_ms = [events[k][3 * i + 1].elapsed_time(events[k][3 * i + 2]) for k in range(steps)]
        e_med, d_med = _pct(ev_ms, 0.5), _pct(de_ms, 0.5)
        nk = n_keep[a]
        tok_bytes = nl * sum(_decode_bytes(Hq, Hkv, d, nk + t + 1) for t in range(T)) / T
        tok_us = d_med * 1e3 / T
        streams_hbm = tok_bytes > LLC_BYTES
        rows.append({
            "alpha": a, "n_keep": nk,
            "evict_all_layers_us": round(e_med * 1e3, 1),
            "us_per_token": round(tok_us, 2),
            "us_per_token_p10_p90": [round(_pct(de_ms, 0.1) * 1e3 / T, 2),
                                     round(_pct(de_ms, 0.9) * 1e3 / T, 2)],
            "tokens_per_s": round(T / ((d_med + e_med) * 1e-3), 1),
            "decode_tokens_per_s": round(1e6 / tok_us, 1),
            "decode_bytes_per_token": round(tok_bytes),
            "decode_GBps": round(tok_bytes / (tok_us * 1e-6) / 1e9, 1),
            "decode_frac_of_8TBps": round(tok_bytes / (tok_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "working_set": "hbm" if streams_hbm else "fits the 256 MB last-level cache (warm)",
        })
        all_bytes += tok_bytes * T * steps
        all_ms += sum(de_ms)
        if streams_hbm:
            hbm_bytes += tok_bytes * T * steps
            hbm_ms += sum(de_ms)
            hbm_calls += T * nl * steps
    # eviction stages of one layer at ratio 0.5 (scores do not depend on the ratio)
    a = 0.5
    nk = n_keep[a]
    x = lay[0]
    c = _lib.KVCache(B, Hq, Hkv, nk + T, d, wl.dtype, device=dev)
    ev.evict(x["q_win"], x["k"], x["v"], [L], [a], c, stream)
    sc_t = _best_ms(torch, lambda: ev.score(x["q_win"], x["k"], [L], stream))
    se_t = _best_ms(torch, lambda: ev.select([L], [a], stream))
    co_t = _best_ms(torch, lambda: c.compact_from(x["k"], x["v"], ev.keep_idx, [nk], stream))
    cbytes = 2 * 2 * Hkv * nk * d * 2
    # the stack's compaction (all layers in one call, as evict_all runs it)
    evict_all(a)
    cs_t = _best_ms(torch, lambda: caches[a].compact_from(stack["k"], stack["v"], sev.keep_idx,
                                                          [nk] * (nl * B), stream))
    stack_compaction = {"alpha": a, "layers": nl, "us": round(cs_t * 1e3, 1),
                        "bytes": cbytes * nl,
                        "GBps": round(cbytes * nl / (cs_t * 1e-3) / 1e9, 1),
                        "frac_of_8TBps": round(cbytes * nl / (cs_t * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                        "timing": "best of 3, HIP events around one tb_compact_kv call over the "
                                  f"{nl}-layer stack"}
    stages = {"alpha": a, "score_us": round(sc_t * 1e3, 1), "select_us": round(se_t * 1e3, 1),
              "compact_us": round(co_t * 1e3, 1),
              "compaction_bytes": cbytes,
              "compact_GBps": round(cbytes / (co_t * 1e-3) / 1e9, 1),
              "compact_frac_of_8TBps": round(cbytes / (co_t * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
              "score_window_flops": 2 * Hq * w * L * d,
              "score_fp64_TFLOPs": round(2 * Hq * w * L * d / (sc_t * 1e-3) / 1e12, 2),
              "timing": "best of 3, HIP events around one call"}
    xs = [r["n_keep"] + (T + 1) / 2 for r in rows]
    ys = [r["us_per_token"] for r in rows]
    p, q = _lib.tb_ete_fit(xs, ys, 1)
    pred = [p * xx + q for xx in xs]
    my = sum(ys) / len(ys)
    ss_res = sum((y - f) ** 2 for y, f in zip(ys, pred))
    ss_tot = sum((y - my) ** 2 for y in ys)
    tokens = n_al * T * steps
    calls = hbm_calls
    achieved = hbm_bytes / (hbm_ms * 1e-3) / 1e9
    del graphs, caches, lay, stack, ev, sev, c, out
    torch.cuda.empty_cache()
    return {
        "value": round(tokens / (total_ms * 1e-3), 1),
        "ms_per_step": round(total_ms / steps, 3),
        "wall_s": round(wall, 3),
        "config": {
            "workload": f"{nl}-layer stack bf16 (28 q / 4 kv heads, d=128), B=1, prompt "
                        f"L={L}, w={w}, pool {wl.pool}, ratios alpha=k/20 (k=0..19), {T} "
                        f"decode tokens per ratio; one step = every ratio's eviction of all "
                        f"{nl} layers plus its {T} tokens",
            "B": B, "L": L, "layers": nl, "Hq": Hq, "Hkv": Hkv, "d": d, "w": w,
            "pool": wl.pool, "alphas": alphas, "decode_tokens_per_alpha": T,
            "parallelism": "none (1 GPU)",
        },
        "roofline": {
            "kernel": "tb_decode_attn: decode_mfma_kernel (split-K partials) + "
                      "decode_merge_split_kernel (log-sum-exp merge), one call per layer "
                      "and token",
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic(),
            "traffic_note": "HBM bytes per decode call (FETCH_SIZE and WRITE_SIZE scaled by a "
                            "512 MiB copy, profiles/pmc_decode_compact_28layer_L32768.md); null if the "
                            "decode kernels or their launch plan changed since",
            "avg_call_us": round(hbm_ms * 1e3 / calls, 3),
            "bytes_per_call": round(hbm_bytes / calls),
            "ratios": "alpha <= 0.85 (per-token working set above the 256 MB last-level "
                      "cache, streamed from HBM)",
            "all_ratios_GBps": round(all_bytes / (all_ms * 1e-3) / 1e9, 1),
            "timing": "HIP events on the replay stream around each ratio's graph of "
                      f"{T} x {nl} decode calls, divided by the call count (the gap between "
                      "the two kernels of a call included)",
        },
        "per_alpha": rows,
        "per_alpha_timing": "median over the timed steps (p10, p90 beside it) of HIP events "
                            "around each ratio's 28 evictions and its graph of decode calls",
        "evict_one_layer": stages,
        "stack_compaction": stack_compaction,
        "token_time_fit": {"p_us_per_kv_row": p, "q_us": q,
                           "r2": 1 - ss_res / ss_tot if ss_tot > 0 else 1.0,
                           "mape_pct": 100.0 * sum(abs(f - y) / y for y, f in zip(ys, pred)) / len(ys),
                           "note": "least squares of the per-token time (28 layer calls) against "
                                   "the mean retained length over the 20 ratios (tb_ete_fit): "
                                   "the decode-step form t = p N_kv + q of the execution-time "
                                   "model"},
    }


def counter_sweep(torch, _lib, synth, dev, tokens=8):
    """For HBM counter runs: the headline's compaction and decode calls at the
    ratios whose working set streams from HBM (alpha <= 0.85, the roofline's
    ratios) and at the headline's shapes and launch plans, launched one by one
    (no graph, no scoring).  Per ratio: every layer's cache is compacted from a
    fixed kept set (the first n_keep - w prefix positions and the window), then
    `tokens` decode tokens of all 28 layers.  Kernel traffic does not depend on
    which rows are kept.  Returns the dispatch order for attributing counters."""
    wl = synth.WORKLOADS[3]
    nl, B, Hq, Hkv, d, w, L = wl.layers, wl.B, wl.Hq, wl.Hkv, wl.d, wl.w, wl.L
    alphas = [a for a in wl.alphas
              if nl * _decode_bytes(Hq, Hkv, d, _lib.tb_keep_count(L, a, w) + 1) > LLC_BYTES]
    lay = []
    for layer in range(nl):
        pr = synth.make_prompt(wl, layer)
        dc = synth.make_decode(wl, layer, T=tokens)
        lay.append({x: pr[x].to(dev) for x in ("k", "v")})
        lay[-1].update({x: dc[x].to(dev) for x in ("q", "k_new", "v_new")})
        del pr, dc
    stream = torch.cuda.current_stream()
    order = []
    for a in alphas:
        nk = _lib.tb_keep_count(L, a, w)
        keep = torch.cat([torch.arange(nk - w), torch.arange(L - w, L)]).to(torch.int32)
        keep_idx = torch.zeros((B, Hkv, L), dtype=torch.int32)
        keep_idx[:, :, :nk] = keep
        keep_idx = keep_idx.to(dev)
        caches = [_lib.KVCache(B, Hq, Hkv, nk + wl.T, d, wl.dtype, device=dev) for _ in range(nl)]
        for layer in range(nl):
            caches[layer].compact_from(lay[layer]["k"], lay[layer]["v"], keep_idx, [nk], stream)
        out = torch.empty((B, Hq, d), dtype=wl.dtype, device=dev)
        for t in range(tokens):
            for layer in range(nl):
                x, c = lay[layer], caches[layer]
                _lib.tb_decode_attn(x["q"][t], x["k_new"][t], x["v_new"][t], c.k, c.v,
                                    c.kv_len, out, c.ws, stream=stream)
        torch.cuda.synchronize()
        order.append({"alpha": a, "n_keep": nk, "compactions": nl, "decode_calls": tokens * nl})
        del caches, keep_idx, out
    del lay
    torch.cuda.empty_cache()
    return {"workload": f"{nl}-layer L={L} shapes, ratios {alphas}: per ratio {nl} "
                        f"compactions then {tokens} x {nl} decode calls, eager",
            "tokens": tokens, "order": order}


def single_layer(torch, _lib, synth, Evictor, dev, reps=10, cold=True):
    """Supplementary: one bf16 layer with a prompt of L = 8192 tokens (28 q / 4
    kv heads, d = 128, w = 32, pool 7) at the ratios 0 (no eviction) and the
    paper's fixed-ratio arms 0.25 / 0.5 / 0.75 / 0.95, 256 decode steps each;
    reps passes of (eviction + a graph of the 256 steps) per ratio, medians.
    Its 17 MB cache sits in the last-level cache; the cold run rotates the
    ratio-0 step over >= 1 GiB of caches."""
    wl = synth.WORKLOADS[2]
    B, Hq, Hkv, d, w, L, T = wl.B, wl.Hq, wl.Hkv, wl.d, wl.w, wl.L, wl.T
    pr = synth.make_prompt(wl)
    dc = synth.make_decode(wl)
    q_win, k, v = (pr[x].to(dev) for x in ("q_win", "k", "v"))
    qd, knd, vnd = (dc[x].to(dev) for x in ("q", "k_new", "v_new"))
    del pr, dc
    ev = Evictor(B, L, Hq, Hkv, d, w, wl.pool, device=dev)
    stream = torch.cuda.current_stream()
    rows = []
    cap_stream = torch.cuda.Stream()
    for a in wl.alphas:
        nk = _lib.tb_keep_count(L, a, w)
        cache = _lib.KVCache(B, Hq, Hkv, nk + T, d, wl.dtype, device=dev)
        out = torch.empty((T, B, Hq, d), dtype=wl.dtype, device=dev)
        ev.evict(q_win, k, v, [L], [a], cache, stream)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cap_stream):
            for t in range(T):
                _lib.tb_decode_attn(qd[t], knd[t], vnd[t], cache.k, cache.v, cache.kv_len,
                                    out[t], cache.ws, stream=cap_stream)
        torch.cuda.synchronize()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        ev_ms, de_ms = [], []
        for r in range(reps + 1):
            e[0].record(stream)
            ev.evict(q_win, k, v, [L], [a], cache, stream)
            e[1].record(stream)
            g.replay()
            e[2].record(stream)
            torch.cuda.synchronize()
            if r:
                ev_ms.append(e[0].elapsed_time(e[1]))
                de_ms.append(e[1].elapsed_time(e[2]))
        e_med, d_med = _pct(ev_ms, 0.5), _pct(de_ms, 0.5)
        dbytes = sum(_decode_bytes(Hq, Hkv, d, nk + t + 1) for t in range(T))
        rows.append({"alpha": a, "n_keep": nk, "evict_us": round(e_med * 1e3, 2),
                     "decode_us_per_step": round(d_med * 1e3 / T, 3),
                     "decode_us_per_step_p10_p90": [round(_pct(de_ms, 0.1) * 1e3 / T, 3),
                                                    round(_pct(de_ms, 0.9) * 1e3 / T, 3)],
                     "decode_GBps": round(dbytes / (d_med * 1e-3) / 1e9, 1),
                     "tokens_per_s": round(T / ((d_med + e_med) * 1e-3), 1)})
        del g, cache, out
    xs = [r["n_keep"] + (T + 1) / 2 for r in rows]
    ys = [r["decode_us_per_step"] for r in rows]
    slope, icpt = _lib.tb_ete_fit(xs, ys, 1)
    res = {"workload": f"bf16, B=1, L={L}, 28 q / 4 kv heads, d=128, w=32, pool 7, ratios "
                       f"{list(wl.alphas)}, {T} decode steps each (cache in the last-level cache)",
           "per_alpha": rows,
           "decode_time_fit": {"p_us_per_kv_row": slope, "q_us": icpt},
           "timing": f"median of {reps} passes: HIP events around the eviction and around a "
                     f"graph of the {T} decode steps"}
    if cold:
        res["cold_decode"] = cold_decode(torch, _lib, Evictor, dev, wl, q_win, k, v, qd, knd, vnd)
    del q_win, k, v, qd, knd, vnd, ev
    torch.cuda.empty_cache()
    return res


def _paged_cold(torch, _lib, dev, k, v, keep_idx, n_keep, need, table, max_pages, qd, knd,
                vnd, B, Hq, Hkv, d, T, dtype, target_bytes=1 << 30):
    """The ragged batch's paged decode from HBM: R copies of the page pools
    (same table), step t on copy t % R, R chosen so the copies' attended rows
    total at least 1 GiB, so no step finds its pages in the last-level cache."""
    from paper_2512_21859_amd.serving import PAGE
    n_pages = sum(need)
    step_bytes = sum(_decode_bytes(Hq, Hkv, d, n + 1) for n in n_keep)
    R = max(2, -(-target_bytes // step_bytes))
    pools = [(torch.zeros((n_pages, Hkv, PAGE, d), dtype=dtype, device=dev),
              torch.zeros((n_pages, Hkv, PAGE, d), dtype=dtype, device=dev),
              torch.zeros((B,), dtype=torch.int32, device=dev),
              torch.zeros((_lib.tb_workspace_bytes(_lib.TB_OP_DECODE, B, 0, Hq, Hkv, d, 0,
                                                   max_pages * PAGE),),
                          dtype=torch.uint8, device=dev)) for _ in range(R)]
    out = torch.empty((T, B, Hq, d), dtype=dtype, device=dev)
    stream = torch.cuda.current_stream()

    def reset():
        for kp, vp, ln, _ in pools:
            _lib.tb_compact_kv_paged(k, v, keep_idx, n_keep, kp, vp, table, ln, stream)

    reset()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    cs = torch.cuda.Stream()
    with torch.cuda.graph(g, stream=cs):
        for t in range(T):
            kp, vp, ln, ws = pools[t % R]
            _lib.tb_decode_attn_paged(qd[t], knd[t], vnd[t], kp, vp, table, ln, out[t], ws,
                                      stream=cs)
    torch.cuda.synchronize()
    best = float("inf")
    for _ in range(3):
        reset()
        best = min(best, _best_ms(torch, g.replay, reps=1))
    dbytes = sum(_decode_bytes(Hq, Hkv, d, n + t // R + 1) for n in n_keep for t in range(T))
    us = best * 1e3 / T
    del pools, g, out
    torch.cuda.empty_cache()
    return {"how": f"step t on copy t % {R} of the page pools ({R * n_pages * Hkv * PAGE * d * 4 / 2**30:.2f} "
                   f"GiB), graph-replayed",
            "us_per_step": round(us, 2), "tokens_per_s": round(B / (us * 1e-6), 1),
            "GBps": round(dbytes / T / (us * 1e-6) / 1e9, 1),
            "frac_of_8TBps": round(dbytes / T / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}


def paged_serving(torch, _lib, synth, Evictor, dev, T=64, n_req=64, max_seqs=16,
                  max_admit=8):
    """Supplementary: paged caches.

    (1) The ragged 16-sequence batch (prompts of 1024..16384 tokens, a ratio
    in [0, 0.9] per sequence, 28 q / 4 kv heads, d = 128) decoded for T steps
    from contiguous caches and from pages scattered through a pool, with the
    same launch plan; both replayed from graphs.
    (2) A stream of n_req requests through the server (one layer, a library
    call per step): prompts of 1024..16384 tokens, ratios in [0, 0.9],
    64..256 new tokens each, all waiting at the start; up to max_admit are
    evicted per admission batch and up to max_seqs decode together; a
    finished request frees its pages at once.  Timed by the wall clock (host
    bookkeeping included) and by HIP events around each admission and decode
    step.  (3) The same with n_req / 2 requests through the 28-layer model
    shape, each decode step's 28 launches replayed from a captured graph."""
    from paper_2512_21859_amd.serving import PAGE, Server
    wl = synth.WORKLOADS[4]
    B, Hq, Hkv, d, w, pool = wl.B, wl.Hq, wl.Hkv, wl.d, wl.w, wl.pool
    L, alphas = synth.lengths_and_alphas(wl)
    Lmax = max(L)
    pr = synth.make_prompt(wl)
    dc = synth.make_decode(wl, T=T)
    q_win, k, v = (pr[x].to(dev) for x in ("q_win", "k", "v"))
    qd, knd, vnd = (dc[x].to(dev) for x in ("q", "k_new", "v_new"))
    del pr, dc
    stream = torch.cuda.current_stream()
    ev = Evictor(B, Lmax, Hq, Hkv, d, w, pool, device=dev)
    ev.score(q_win, k, L, stream)
    n_keep = ev.select(L, alphas, stream)
    cap = -(-(max(n_keep) + T) // PAGE) * PAGE
    cache = _lib.KVCache(B, Hq, Hkv, cap, d, wl.dtype, device=dev)
    max_pages = cap // PAGE
    need = [-(-(n + T) // PAGE) for n in n_keep]
    gen = torch.Generator().manual_seed(4242)
    perm = torch.randperm(sum(need), generator=gen).tolist()
    table = torch.empty((B, max_pages), dtype=torch.int32)
    at = 0
    for b in range(B):
        pg = perm[at:at + need[b]]
        at += need[b]
        table[b] = torch.tensor(pg + [pg[-1]] * (max_pages - need[b]), dtype=torch.int32)
    table = table.to(dev)
    k_pool = torch.zeros((sum(need), Hkv, PAGE, d), dtype=wl.dtype, device=dev)
    v_pool = torch.zeros((sum(need), Hkv, PAGE, d), dtype=wl.dtype, device=dev)
    len_p = torch.zeros((B,), dtype=torch.int32, device=dev)
    ws_p = torch.zeros_like(cache.ws)
    out_c = torch.empty((T, B, Hq, d), dtype=wl.dtype, device=dev)
    out_p = torch.empty_like(out_c)

    def reset():
        cache.compact_from(k, v, ev.keep_idx, n_keep, stream)
        _lib.tb_compact_kv_paged(k, v, ev.keep_idx, n_keep, k_pool, v_pool, table, len_p, stream)

    reset()
    torch.cuda.synchronize()
    cs = torch.cuda.Stream()
    g_c, g_p = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_c, stream=cs):
        for t in range(T):
            _lib.tb_decode_attn(qd[t], knd[t], vnd[t], cache.k, cache.v, cache.kv_len, out_c[t],
                                cache.ws, stream=cs)
    with torch.cuda.graph(g_p, stream=cs):
        for t in range(T):
            _lib.tb_decode_attn_paged(qd[t], knd[t], vnd[t], k_pool, v_pool, table, len_p,
                                      out_p[t], ws_p, stream=cs)
    torch.cuda.synchronize()
    best = {"contiguous": float("inf"), "paged": float("inf")}
    for _ in range(3):
        for name, g in (("contiguous", g_c), ("paged", g_p)):
            reset()
            best[name] = min(best[name], _best_ms(torch, g.replay, reps=1))
    same = bool(torch.equal(out_c, out_p))
    dbytes = sum(_decode_bytes(Hq, Hkv, d, n + t + 1) for n in n_keep for t in range(T)) / T
    batch = {"workload": f"bf16, B={B} ragged prompts {min(L)}..{max(L)}, ratios "
                         f"{min(alphas):.2f}..{max(alphas):.2f}, 28 q / 4 kv heads, d=128, "
                         f"{T} decode steps",
             "n_keep_total": sum(n_keep), "pages": sum(need), "bit_identical": same}
    for name in ("contiguous", "paged"):
        us = best[name] * 1e3 / T
        batch[name] = {"us_per_step": round(us, 2),
                       "GBps": round(dbytes / (us * 1e-6) / 1e9, 1)}
    for name in ("contiguous", "paged"):
        batch[name]["tokens_per_s"] = round(B / (best[name] * 1e-3 / T), 1)
    batch["paged_over_contiguous"] = round(best["paged"] / best["contiguous"], 4)
    batch["working_set"] = (f"{dbytes / 1e6:.0f} MB per step, in the 256 MB last-level cache "
                            "(warm: the caches were just written by the compaction)")
    del cache, g_c, g_p, out_c, out_p
    torch.cuda.empty_cache()
    batch["paged_cold"] = _paged_cold(torch, _lib, dev, k, v, ev.keep_idx, n_keep, need, table,
                                      max_pages, qd, knd, vnd, B, Hq, Hkv, d, T, wl.dtype)
    del k_pool, v_pool, q_win, k, v, qd, knd, vnd, ev
    torch.cuda.empty_cache()

    # (2) the streams: one layer with a library call per layer and step, and
    # the 28-layer model shape with each step's 28 launches replayed from a graph
    stream_res = _serving_stream(torch, _lib, Server, dev, wl, n_layers=1, n_req=n_req,
                                 max_seqs=max_seqs, max_admit=max_admit, graphed=False)
    stream28 = _serving_stream(torch, _lib, Server, dev, wl, n_layers=28, n_req=n_req // 2,
                               max_seqs=max_seqs, max_admit=max_admit, graphed=True)
    stream28o = _serving_stream(torch, _lib, Server, dev, wl, n_layers=28, n_req=n_req // 2,
                                max_seqs=max_seqs, max_admit=max_admit, graphed=True,
                                overlap=True)
    return {"batch": batch, "stream": stream_res, "stream_28_layers": stream28,
            "stream_28_layers_overlapped": stream28o}


def _serving_stream(torch, _lib, Server, dev, wl, n_layers, n_req, max_seqs, max_admit,
                    graphed, overlap=False):
    """n_req requests (prompts 1024..16384, ratios 0..0.9, 64..256 new tokens,
    all waiting at the start) through a server of n_layers layers; admission
    evicts every layer of up to max_admit requests; one decode step runs every
    layer of the running batch (graph-replayed when graphed).  With overlap the
    eviction runs on its own stream beside the decode steps and the batch joins
    at the first step after it has finished; otherwise it runs between two
    steps.  As a server that samples each step's tokens must, the host queues
    step t only once step t-2 has finished (one step in flight while the next
    is prepared).  The second of two passes is timed; GPU figures sum HIP
    events around admissions and steps, the token interval is the time between
    the ends of consecutive steps on the decode stream, and the join delay is
    the time from an admission's call to its requests' first step."""
    from paper_2512_21859_amd.serving import PAGE
    Hq, Hkv, d, w, pool = wl.Hq, wl.Hkv, wl.d, wl.w, wl.pool
    gen = torch.Generator().manual_seed(6464)
    rL = torch.randint(1024, 16385, (n_req,), generator=gen).tolist()
    ra = (0.9 * torch.rand(n_req, generator=gen, dtype=torch.float64)).tolist()
    rn = torch.randint(64, 257, (n_req,), generator=gen).tolist()
    Pmax = 16384
    max_pages = -(-(Pmax + 256) // PAGE)
    srv = Server(n_layers, n_pages=max_seqs * max_pages, max_seqs=max_seqs, max_pages=max_pages,
                 Hq=Hq, Hkv=Hkv, d=d, dtype=wl.dtype, w=w, pool=pool, max_admit=max_admit,
                 max_prompt=Pmax, device=dev)
    stream = srv.decode_stream                   # every step (and serial admission) goes here
    dg = torch.Generator(device=dev).manual_seed(77)
    kb = torch.randn((max_admit, Hkv, Pmax, d), generator=dg, device=dev).to(wl.dtype)
    vb = torch.randn((max_admit, Hkv, Pmax, d), generator=dg, device=dev).to(wl.dtype)
    qb = torch.randn((max_admit, Hq, w, d), generator=dg, device=dev).to(wl.dtype)
    for buf in (srv.q_in, srv.k_in, srv.v_in):         # decode inputs (any values)
        buf.copy_(torch.randn(buf.shape, generator=dg, device=dev).to(wl.dtype))
    prompts = [{"q_win": qb, "k": kb, "v": vb}] * n_layers   # every layer evicts the same data
    if graphed:
        for n in range(1, max_seqs + 1):         # capture synchronises: keep it out of the passes
            srv.capture(n)

    def run():
        queue = list(range(n_req))
        ev_pairs, de_pairs, waiting, just, joins = [], [], [], [], []
        steps = tokens = batch_sum = 0
        dec_bytes = 0.0
        while queue or srv.n_active or srv.slots.pending:
            fin = srv.slots.finished()
            if fin:
                srv.retire(fin)
            if overlap and srv.promote_ready(wait=srv.n_active == 0):
                just.append(waiting.pop(0))
            adm = []
            while (queue and not srv.slots.pending and len(adm) < max_admit and srv.slots.fits(
                    [_lib.tb_keep_count(rL[r], ra[r], w) + rn[r] for r in adm + [queue[0]]])):
                adm.append(queue.pop(0))
            if adm:
                b = len(adm)
                args = (adm, [rL[r] for r in adm], [ra[r] for r in adm], [rn[r] for r in adm],
                        [{k: x[:b] for k, x in p.items()} for p in prompts])
                if overlap:
                    e = torch.cuda.Event(enable_timing=True)
                    e.record(stream)
                    srv.admit_async(*args)
                    waiting.append(e)
                    if srv.n_active == 0:
                        srv.promote_ready(wait=True)
                        just.append(waiting.pop(0))
                    ev_pairs.append(None)
                else:
                    e = (torch.cuda.Event(enable_timing=True),
                         torch.cuda.Event(enable_timing=True))
                    e[0].record(stream)
                    srv.admit(*args, stream=stream)
                    e[1].record(stream)
                    ev_pairs.append(e)
                    just.append(e[0])
            n = srv.n_active
            if n == 0:
                continue                         # the last requests just retired
            lens = srv.slots.lengths()
            e = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            e[0].record(stream)
            if graphed:
                srv.step_graphed()
            else:
                srv.step(srv.q_in[:, :n], srv.k_in[:, :n], srv.v_in[:, :n], srv.o_out[:, :n],
                         stream=stream)
            e[1].record(stream)
            de_pairs.append(e)
            joins += [(x, e[0]) for x in just]
            just = []
            if len(de_pairs) >= 2:
                de_pairs[-2][1].synchronize()    # step t-1's tokens are read back
            steps += 1
            tokens += n
            batch_sum += n
            dec_bytes += n_layers * sum(_decode_bytes(Hq, Hkv, d, int(x) + 1) for x in lens)
        torch.cuda.synchronize()
        return ev_pairs, de_pairs, joins, steps, tokens, batch_sum, dec_bytes

    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        run()                                    # warm-up pass (and graph captures)
        t0 = time.perf_counter()
        ev_pairs, de_pairs, joins, steps, tokens, batch_sum, dec_bytes = run()
        wall = time.perf_counter() - t0
    de_ms = sum(a.elapsed_time(b) for a, b in de_pairs)
    gaps = sorted(de_pairs[i][1].elapsed_time(de_pairs[i + 1][1])
                  for i in range(len(de_pairs) - 1))
    jd = sorted(a.elapsed_time(b) for a, b in joins)
    res = {
        "workload": f"{n_req} requests, {n_layers} layer(s) bf16, prompts 1024..16384, ratios "
                    f"0..0.9, 64..256 new tokens, <= {max_seqs} decoding, <= {max_admit} per "
                    f"admission" + (", each step's launches replayed from a graph" if graphed else "")
                    + (", eviction overlapped with decode on a second stream" if overlap else ""),
        "tokens": tokens, "decode_steps": steps, "admissions": len(ev_pairs),
        "mean_batch": round(batch_sum / steps, 2),
        "wall_s": round(wall, 4), "tokens_per_s_wall": round(tokens / wall, 1),
        "gpu_decode_ms": round(de_ms, 3),
        "decode_tokens_per_s_gpu": round(tokens / (de_ms * 1e-3), 1),
        "decode_GBps": round(dec_bytes / (de_ms * 1e-3) / 1e9, 1),
        "token_interval_ms": {"p50": round(gaps[len(gaps) // 2], 4),
                              "p99": round(gaps[int(0.99 * (len(gaps) - 1))], 4),
                              "max": round(gaps[-1], 4)},
        "join_delay_ms": {"mean": round(sum(jd) / len(jd), 3), "max": round(jd[-1], 3)},
        "timing": "second pass over the stream (the first warms up); GPU figures sum HIP "
                  "events around each admission and each decode step"}
    if not overlap:
        ev_ms = sum(a.elapsed_time(b) for a, b in ev_pairs)
        res["gpu_evict_ms"] = round(ev_ms, 3)
        res["tokens_per_s_gpu"] = round(tokens / ((de_ms + ev_ms) * 1e-3), 1)
    del srv, kb, vb, qb
    torch.cuda.empty_cache()
    return res



def main():
    args = _parse()
    if args.gpus != 1:
        print(f"bench.py: the benchmark runs on exactly one GPU; --gpus {args.gpus} is not "
              f"supported (the path shards by sequence / KV head with no exchange).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2512_21859_amd import _lib, synth
    from paper_2512_21859_amd.pipeline import Evictor

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    _lib.load()
    if args.pmc_calibration:
        src = torch.ones((256 << 20,), dtype=torch.bfloat16, device=dev)   # 512 MiB
        dst = torch.empty_like(src)
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    sections = {
        "single": lambda: single_layer(torch, _lib, synth, Evictor, dev),
        "long": lambda: long_context(torch, _lib, synth, Evictor, dev),
        "ceiling": lambda: {"hbm": hbm_ceiling(torch, dev), "mfma": mfma_ceiling(torch, dev)},
        "scorers": lambda: scorer_variants(torch, _lib, synth, Evictor, dev),
        "prefill": lambda: prefill_sweep(torch, _lib, synth, dev),
        "paged": lambda: paged_serving(torch, _lib, synth, Evictor, dev),
        "counters": lambda: counter_sweep(torch, _lib, synth, dev),
    }
    if args.only and args.only != "headline":
        print(json.dumps({"section": args.only, **sections[args.only]()}), flush=True)
        return

    head = headline(torch, _lib, synth, Evictor, dev, args.steps, args.warmup, args.tokens)
    result = {
        "metric": "decode tokens/s and HBM GB/s (evict+decode attn) vs eviction ratio α, 1 GPU",
        "value": head.pop("value"),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head.pop("ms_per_step"),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) K/V/queries with planted heavy-hitter keys; "
                "random-init stand-in for LongBench on Qwen2.5-7B)",
        **head,
    }
    if args.only == "headline":
        print(json.dumps(result), flush=True)
        return
    if not args.no_single:
        result["single_layer"] = sections["single"]()
    if not args.no_long_context:
        result["long_context"] = sections["long"]()
    if not args.no_prefill:
        result["prefill"] = sections["prefill"]()
    if not args.no_paged:
        result["paged"] = sections["paged"]()
    if not args.no_scorers:
        result["scorers"] = sections["scorers"]()
    if not args.no_ceiling:
        ceil = sections["ceiling"]()
        result["hbm_ceiling"] = ceil["hbm"]
        result["mfma_ceiling"] = ceil["mfma"]
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
