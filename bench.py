"""Benchmark of the gauge-coded KV codec hot path on one MI355X.

A step is one full pass of the hot path over the Llama-3-8B-shaped KV cache (32 layers,
8 KV heads, head_dim 128, batch 1, 8192 tokens, bf16; Haar gauge with g = 128; block-uniform
4-bit, block 64): encode K, encode V (gauge -> block range -> quantise -> bit-pack), then
decode K, decode V (unpack -> dequantise -> inverse gauge -> bf16).  Inputs are seeded
synthetic tensors already resident in HBM.

Prints one JSON line.  `value` is the round-trip throughput in logical bf16 bytes
(2 bytes per K/V element) per second; `roofline` describes the dominant kernel against the
HBM peak, with its algorithmic bytes per launch and the average launch time measured with
HIP events on the stream the kernels run on, and (`ceiling`) the rate the library's streaming
probe reaches on the same read / write byte mix with no arithmetic; `cpu_baseline` times the
CPU oracle on a bounded sample of the same workload.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
WORKLOAD = "llama8b"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-layers", type=int, default=8)
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "traffic_llama8b.json"),
                    help="HBM traffic per launch measured with rocprofv3 counters (optional)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="after the timed region, run one plain 512 MiB device copy (counter calibration)")
    ap.add_argument("--workload", default=WORKLOAD, choices=sorted(["llama8b", "kivi", "rolling", "gemma27b", "tiles", "spectral", "grad", "attend", "attend_paged", "attend_tiles", "attend_kivi", "zfp"]),
                    help="llama8b (default) prints the headline line; the others print per-kernel timings of "
                         "the KIVI, rolling-step and 27B-sweep workloads")
    return ap.parse_args()


def algorithmic_bytes(w, s_count=1):
    """Bytes one launch must move: per element bf16 in (2) + codes (b/8) + side (4/n),
    plus the binary32 gauge blocks of the launch's cache type (4 g^2 per (l, h, r))."""
    per_elem = 2.0 + w.bits / 8.0 + 4.0 / w.block_c
    elems = w.L * w.B * w.H * w.T * w.d
    gauge = 4.0 * w.g * w.g * w.L * w.H * (w.d // w.g)
    return s_count * (elems * per_elem + gauge)


def kernel_source_hash():
    """First 16 hex digits of the SHA-256 of the matrix-core kernel sources (cg_mfma.hip followed by
    its shared header cg_mfma_util.h)."""
    import hashlib

    h = hashlib.sha256()
    for f in ("cg_mfma.hip", "cg_mfma_util.h"):
        h.update(open(os.path.join(ROOT, "paper_2607_20538_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(path, kernel):
    """HBM bytes per launch of `kernel` from the rocprofv3 FETCH_SIZE / WRITE_SIZE summary (scaled
    by the copy-kernel calibration), or None when there is none or the kernel source has changed
    since the counters were taken."""
    import hashlib

    try:
        tr = json.load(open(path))
        if kernel_source_hash() != tr.get("source_sha256_16"):
            return None
        return int(tr[kernel]["bytes"])
    except (OSError, ValueError, KeyError, TypeError):
        return None


def cpu_info():
    """Model, logical CPUs available to this process and the nominal clock of the host."""
    model, mhz = "unknown", None
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name") and model == "unknown":
                    model = ln.split(":", 1)[1].strip()
                elif ln.startswith("cpu MHz") and mhz is None:
                    mhz = float(ln.split(":", 1)[1])
    except OSError:
        pass
    return {"model": model, "logical_cpus": len(os.sched_getaffinity(0)), "mhz": mhz}


def oracle_threads():
    """Worker threads for the oracle: the CPUs this process may use, at most OMP_NUM_THREADS when set."""
    n = len(os.sched_getaffinity(0))
    cap = os.environ.get("OMP_NUM_THREADS")
    if cap and cap.isdigit() and int(cap) > 0:
        n = min(n, int(cap))
    return max(1, n)


def cpu_baseline(w, G_host, layers):
    """The oracle as written, timed two ways on the host: single-threaded on one layer of K and V,
    and with one thread per (layer, head) slice task over `layers` layers of K and V (the oracle's
    C calls release the interpreter lock, so the slices run in parallel; every slice is independent:
    the gauge never mixes heads or layers).  Encode + decode, GB/s of bf16 KV."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle as O
    from paper_2607_20538_amd import synth

    oc = O.Codec(backend=O.BLOCK_UNIFORM, bits=w.bits, block_c=w.block_c)

    def run_slice(s, X, G):
        cache, _ = O.kv_encode(oc, s, X, G, T_cap=w.T)
        O.kv_decode(oc, s, G, cache, 0, w.T, out_bf16=True)

    # single thread: layer 0 of K and V
    t1, e1 = 0.0, 0
    for s in (0, 1):
        X = synth.kv_tensor(w, s, L=1)
        t0 = time.perf_counter()
        run_slice(s, X, np.ascontiguousarray(G_host[:1]))
        t1 += time.perf_counter() - t0
        e1 += X.size
    # threads over (layer, head) slices of `layers` layers
    nth = oracle_threads()
    tasks = []
    for s in (0, 1):
        X = synth.kv_tensor(w, s, L=layers)
        for l in range(layers):
            for h in range(w.H):
                tasks.append((s, np.ascontiguousarray(X[l:l + 1, :, h:h + 1]),
                              np.ascontiguousarray(G_host[l:l + 1, :, h:h + 1])))
        del X
    em = sum(t[1].size for t in tasks)
    with ThreadPoolExecutor(max_workers=nth) as ex:
        t0 = time.perf_counter()
        list(ex.map(lambda t: run_slice(*t), tasks))
        tm = time.perf_counter() - t0
    info = cpu_info()
    return {"value": round(em * 2 / tm / 1e9, 4), "unit": "GB/s", "cores": nth, "kind": "oracle",
            "single_thread": {"value": round(e1 * 2 / t1 / 1e9, 4), "unit": "GB/s", "cores": 1,
                              "sample": f"layer 0 of K and V ({e1} elements), {t1:.1f} s"},
            "cpu": info,
            "sample": f"{layers} of {w.L} layers of K and V ({em} elements) in {len(tasks)} (layer, head) slice "
                      f"tasks on {nth} threads, encode+decode, {tm:.1f} s; host {info['model']}, "
                      f"{info['logical_cpus']} logical CPUs"}


def single_threaded(fn, *args):
    """fn(*args) with the numpy BLAS pool held to one thread (the oracle's numpy parts would
    otherwise use every host core while the baseline reports one)."""
    try:
        from threadpoolctl import threadpool_limits
    except ImportError:
        return fn(*args)
    with threadpool_limits(1):
        return fn(*args)


def workload_cpu_baseline(name, w, gpu):
    """The oracle (single thread, as written) on a bounded sample of workload `name`, in the unit of
    the workload's GPU figure: one layer and one batch row (every head) of K and V encoded and
    decoded (GB/s of bf16 KV, round trip) for the codec workloads; for the rolling and attention
    steps one (layer, batch row) of the step, extrapolated to the workload's L x B rows."""
    import numpy as np

    import oracle as O
    from paper_2607_20538_amd import synth

    if name in ("kivi", "gemma27b", "tiles", "zfp"):
        g, bits = {"tiles": (128, 4), "zfp": (128, 4)}.get(name, (w.g, w.bits))
        if name == "kivi":
            oc = O.Codec(backend=O.KIVI, bits=bits, block_c=64, key_tokens=w.key_tokens,
                         val_channels=w.val_channels, residual=w.residual)
        elif name == "tiles":
            oc = O.Codec(backend=O.BLOCK_UNIFORM, bits=bits, block_c=128, block_t=16)
        elif name == "zfp":
            oc = O.Codec(backend=O.ZFP, bits=bits)
        else:
            oc = O.Codec(backend=O.BLOCK_UNIFORM, bits=bits, block_c=w.block_c)
        G = O.gauge_make(O.GAUGE_HAAR, 1, w.H, w.d, g, seed=w.gauge_seed)
        t_total, elems = 0.0, 0
        for s in (0, 1):
            X = synth.kv_tensor(w, s, L=1, B=1)
            t0 = time.perf_counter()
            cache, _ = O.kv_encode(oc, s, X, G, T_cap=w.T)
            O.kv_decode(oc, s, G, cache, 0, w.T, lens=np.array([w.T], dtype=np.int32), out_bf16=True)
            t_total += time.perf_counter() - t0
            elems += X.size
        return {"value": round(elems * 2 / t_total / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
                "sample": f"layer 0, batch row 0 ({w.H} heads x {w.T} tokens) of K and V at g = {g}, "
                          f"{bits} bits ({elems} elements), encode + decode, {t_total:.1f} s single-threaded"}
    if name in ("rolling", "attend", "attend_tiles", "attend_paged", "attend_kivi"):
        # one (layer, batch row): its history encoded (untimed), then the step's work for it timed:
        # append one token to K and V and decode the history (rolling), or attention of its grp = 4
        # query heads per KV head over the history (attention steps; the oracle has no page table,
        # so paged caches are timed as the contiguous ones they are equivalent to)
        bt = 16 if name == "attend_tiles" else 1
        if name == "attend_kivi":
            oc = O.Codec(backend=O.KIVI, bits=w.bits, block_c=64, key_tokens=w.key_tokens,
                         val_channels=w.val_channels, residual=w.residual)
        else:
            oc = O.Codec(backend=O.BLOCK_UNIFORM, bits=w.bits, block_c=w.block_c, block_t=bt)
        G = O.gauge_make(O.GAUGE_HAAR, 1, w.H, w.d, w.g, seed=w.gauge_seed)
        T_cap = w.T + 32
        caches = []
        for s in (0, 1):
            X = synth.kv_tensor(w, s, L=1, B=1)
            caches.append(O.kv_encode(oc, s, X, G, T_cap=T_cap)[0])
            del X
        t0 = time.perf_counter()
        if name == "rolling":
            for s in (0, 1):
                xn = synth.kv_tensor(w, s, L=1, B=1, T=1, t_offset=w.T)[:, :, :, 0, :]
                O.kv_append(oc, s, xn, G, caches[s], np.array([w.T], dtype=np.int32))
                O.kv_decode(oc, s, G, caches[s], 0, w.T + 1, lens=np.array([w.T + 1], dtype=np.int32), out_bf16=True)
            held = w.T + 1
        else:
            held = w.T
            qv = synth.queries(w, 4 * w.H, L=1, B=1)
            q = (qv.astype(np.uint32) << 16).view(np.float32) if qv.dtype == np.uint16 else qv
            O.attend(oc, G, caches[0], caches[1], q, np.array([held], dtype=np.int32), 1.0 / np.sqrt(w.d))
        t_row = time.perf_counter() - t0
        rows = w.L * w.B
        ms = t_row * rows * 1e3
        out = {"value": round(ms, 1), "unit": "ms per step (extrapolated)", "cores": 1, "kind": "oracle",
               "sample": f"layer 0, batch row 0 ({w.H} KV heads, {held}-position history): "
                         + ("append one K / V token and decode the history" if name == "rolling"
                            else "attention of 4 query heads per KV head")
                         + f", {t_row:.1f} s single-threaded, x {rows} (layer, batch row) pairs"}
        return out
    if name == "grad":
        # the whole K tensor of batch row 0 (every layer, head and token), 16-channel gauges, scaled
        # by the batch rows
        g, nl = 16, w.L
        X = synth.kv_tensor(w, 0, L=nl, B=1)
        A = 0.05 * np.random.default_rng(w.gauge_seed).standard_normal((nl, 2, w.H, w.d // g, g, g))
        t0 = time.perf_counter()
        O.spectral_train_grad(X, A, 0, Tb=16)
        t1 = time.perf_counter() - t0
        scale = w.B
        return {"value": round(t1 * scale * 1e3, 1), "unit": "ms per tensor" + (" (extrapolated)" if scale > 1 else ""),
                "cores": 1, "kind": "oracle", "sample": f"K of batch row 0 ({nl} layers x {w.H} heads x {w.T} tokens), g = {g}: "
                                            f"{t1:.1f} s single-threaded, x {scale} batch row(s)"}
    if name == "spectral":
        G = O.gauge_make(O.GAUGE_HAAR, 1, w.H, w.d, w.g, seed=w.gauge_seed)
        t_total, elems = 0.0, 0
        for s in (0, 1):
            X = synth.kv_tensor(w, s, L=8)
            t0 = time.perf_counter()
            O.spectral_stats(X, np.repeat(G, 8, axis=0), s, 16, 0.04)
            t_total += time.perf_counter() - t0
            elems += X.size
        return {"value": round(elems * 2 / t_total / 1e9, 4), "unit": "GB/s bf16 in", "cores": 1, "kind": "oracle",
                "sample": f"layers 0-7 of K and V ({elems} elements), {t_total:.1f} s single-threaded"}
    return None


def _timed(fn, steps, warmup, stream):
    """Average milliseconds of fn() over `steps` launches (after `warmup`), HIP events on `stream`."""
    import torch

    for _ in range(warmup):
        fn()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(steps):
        fn()
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / steps


def copy_probe():
    """One plain 512 MiB device-to-device copy: the reference dispatch that rocprofv3's FETCH_SIZE /
    WRITE_SIZE counters are calibrated against."""
    import torch

    src = torch.empty(256 << 20, dtype=torch.int16, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def other_workload(name, steps, warmup, cpu=True, probe=False):
    """Per-kernel timings of the KIVI, rolling, 27B and token-channel tile workloads at their
    full shapes, from seeded synthetic K/V (synth.kv_tensor): eight distinct layers repeated to
    L layers for the KIVI, 27B and tile inputs (the tiles use the Llama-3-8B shape with one
    range per 16 tokens x 128 channels); for the rolling step the history is encoded from one
    layer viewed with layer stride 0 (each layer's own gauge makes its cache distinct), and the
    timed step appends one token per (layer, batch, head) and decodes the whole history into
    bf16."""
    import numpy as np
    import torch

    from paper_2607_20538_amd import codec as cg
    from paper_2607_20538_amd import synth

    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    w = synth.WORKLOADS["llama8b" if name in ("tiles", "spectral", "grad", "zfp") else
                        ("rolling" if name in ("attend", "attend_paged", "attend_tiles") else
                         ("kivi" if name == "attend_kivi" else name))]
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = {"workload": name, "shape": {"L": w.L, "B": w.B, "H": w.H, "T": w.T, "d": w.d}, "steps": steps,
           "kernels": os.environ.get("CG_KERNELS") or "default"}

    def layer_input(s):
        # the workload's first min(8, L) layers, repeated: 8 distinct layers of these shapes span
        # more than the chip's caches, so every layer is read from HBM
        nd = min(8, w.L)
        xs = synth.kv_tensor(w, s, L=nd)
        xs = torch.from_numpy(xs.view(np.int16)).view(torch.bfloat16).cuda()
        X = torch.empty((w.L, w.B, w.H, w.T, w.d), dtype=torch.bfloat16, device="cuda")
        for l0 in range(0, w.L, nd):
            X[l0:l0 + nd] = xs[: min(nd, w.L - l0)]
        return X

    def layer_view(s):
        # one layer viewed with layer stride 0 (history construction of the rolling workload)
        x1 = synth.kv_tensor(w, s, L=1)
        x1 = torch.from_numpy(x1.view(np.int16)).view(torch.bfloat16).cuda()
        return x1.expand(w.L, w.B, w.H, w.T, w.d)

    def bytes_per_elem(bits, n, kivi=False):
        return 2.0 + bits / 8.0 + (4.0 / n if not kivi else 0.0)

    if name == "spectral":
        # section 4.2 statistics of G X on the Llama-3-8B shape, 16-token blocks, tau = 0.04
        shp = cg.shape(w.L, w.H, w.d, w.g)
        Gd = cg.alloc_gauge(shp)
        cg.gauge_make(cg.GAUGE_HAAR, shp, seed=w.gauge_seed, G_host=None, G_dev=Gd)
        ws = torch.empty(cg.spectral_workspace_bytes(shp, 16), dtype=torch.uint8, device="cuda")
        stats = torch.empty((w.L, 4), dtype=torch.float64, device="cuda")
        rows = {}
        for s, tag in ((0, "K"), (1, "V")):
            X = layer_input(s)
            ms = _timed(lambda: cg.kv_spectral_stats(s, X, Gd, shp, 16, 0.04, ws, stats, stream=stream.cuda_stream),
                        steps, warmup, stream)
            st = stats.cpu().numpy()
            rows[tag] = {"ms": round(ms, 3), "GBps_bf16_in": round(X.numel() * 2 / ms / 1e6, 1),
                         "L_freq_mean": round(float(st[:, 0].mean()), 6), "L_rate_mean": round(float(st[:, 1].mean()), 6)}
            del X
            torch.cuda.empty_cache()
        out["runs"] = rows
    elif name == "grad":
        # gradient of the section 4.2 objective with respect to the generators A of G = exp(A - A^T)
        # (section 4.1) on the Llama-3-8B shape: full-head (g = 128) and 16-channel gauges,
        # 16-token blocks, tau = 0.04, lambda_f = 1, lambda_r = 0.02; generators drawn N(0, 0.05^2)
        rows = {}
        for g in (128, 16):
            shp = cg.shape(w.L, w.H, w.d, g)
            A = (0.05 * np.random.default_rng(w.gauge_seed).standard_normal((w.L, 2, w.H, w.d // g, g, g))).astype(np.float32)
            Gd = cg.alloc_gauge(shp)
            t0 = time.perf_counter()
            cg.gauge_make(cg.GAUGE_EXPM, shp, params=A, G_host=None, G_dev=Gd)
            t_make = time.perf_counter() - t0
            Ad = torch.from_numpy(A).cuda()
            ws = torch.empty(cg.gauge_grad_workspace_bytes(shp, w.B, w.T, 16), dtype=torch.uint8, device="cuda")
            stats = torch.empty((w.L, 4), dtype=torch.float64, device="cuda")
            grad = torch.empty((w.L, w.H, w.d // g, g, g), dtype=torch.float64, device="cuda")
            for s, tag in ((0, "K"), (1, "V")):
                X = layer_input(s)
                ms = _timed(lambda: cg.kv_gauge_grad(s, X, Ad, Gd, shp, 16, 0.04, 1.0, 0.02, ws, stats, grad,
                                                     stream=stream.cuda_stream), steps, warmup, stream)
                st = stats.cpu().numpy()
                rows[f"g{g}_{tag}"] = {"ms": round(ms, 3), "GBps_bf16_in": round(X.numel() * 2 / ms / 1e6, 1),
                                       "L_train_mean": round(float((st[:, 0] + 0.02 * st[:, 1]).mean()), 6),
                                       "grad_max": float(grad.abs().max().item())}
                del X
                torch.cuda.empty_cache()
            rows[f"g{g}_gauge_make_s"] = round(t_make, 2)
            del ws, grad, Gd
            torch.cuda.empty_cache()
        out["runs"] = rows
    elif name in ("kivi", "gemma27b", "tiles", "zfp"):
        combos = {"kivi": [(w.g, w.bits)], "tiles": [(128, 4), (128, 3), (32, 4)],
                  "zfp": [(128, r) for r in (2, 3, 4, 6, 8)]}.get(
            name, [(g, b) for g in (8, 16, 32, 128) for b in (3, 4, 6)])
        rows = []
        for g, bits in combos:
            shp = cg.shape(w.L, w.H, w.d, g)
            Gd = cg.alloc_gauge(shp)
            cg.gauge_make(cg.GAUGE_HAAR, shp, seed=w.gauge_seed, G_host=None, G_dev=Gd)
            if name == "kivi":
                codec = cg.Codec(cg.KIVI, bits, 64, w.key_tokens, w.val_channels, w.residual)
            elif name == "tiles":
                codec = cg.Codec(cg.BLOCK_UNIFORM, bits, 128, block_t=16)
            elif name == "zfp":
                codec = cg.Codec(cg.ZFP, bits)
            else:
                codec = cg.Codec(cg.BLOCK_UNIFORM, bits, w.block_c)
            row = {"g": g, "bits": bits}
            for s, tag in ((0, "K"), (1, "V")):
                X = layer_input(s)
                cache = cg.Cache(codec, s, w.L, w.B, w.H, w.T, w.d)
                Y = torch.empty((w.L, w.B, w.H, w.T, w.d), dtype=torch.bfloat16, device="cuda")
                enc = _timed(lambda: cg.kv_encode(s, X, Gd, shp, codec, cache, err_flag=err,
                                                  stream=stream.cuda_stream), steps, warmup, stream)
                if name in ("kivi", "tiles"):
                    cache.len = w.T
                dec = _timed(lambda: cg.kv_decode(s, cache, Gd, shp, codec, 0, Y, err_flag=err,
                                                  stream=stream.cuda_stream), steps, warmup, stream)
                nelem = w.L * w.B * w.H * w.T * w.d
                nc, ns, nr = cache.nbytes
                alg = nelem * 2 + nc + ns + nr
                row[tag] = {"encode_ms": round(enc, 3), "decode_ms": round(dec, 3),
                            "encode_GBps": round(alg / enc / 1e6, 1), "decode_GBps": round(alg / dec / 1e6, 1)}
                del X, Y, cache
                torch.cuda.empty_cache()
            rows.append(row)
        out["runs"] = rows
    elif name == "attend_paged":
        # the attention workload over page pools: 256-position pages in a seeded random order,
        # the history encoded through the page table, one paged append + paged attention per step
        grp, P = 4, 256
        shp = cg.shape(w.L, w.H, w.d, w.g)
        codec = cg.Codec(cg.BLOCK_UNIFORM, w.bits, w.block_c)
        Gd = cg.alloc_gauge(shp)
        cg.gauge_make(cg.GAUGE_HAAR, shp, seed=w.gauge_seed, G_host=None, G_dev=Gd)
        maxp = (w.T + warmup + 2 * steps + 1 + P - 1) // P
        perm = np.random.default_rng(w.data_seed).permutation(w.B * maxp).astype(np.int32)
        pages = torch.from_numpy(perm.reshape(w.B, maxp)).cuda()
        pt = cg.page_table(pages, P)
        pools, news = [], []
        for s in (0, 1):
            X = layer_view(s)
            c = cg.Cache(codec, s, w.L, w.B * maxp, w.H, P, w.d)
            cg.kv_encode_paged(s, X, pt, Gd, shp, codec, c, 0, err_flag=err, stream=stream.cuda_stream)
            torch.cuda.synchronize()
            del X
            pools.append(c)
            nt = synth.kv_tensor(w, s, L=1, T=1, t_offset=w.T)
            nt = torch.from_numpy(nt.view(np.int16)).view(torch.bfloat16).cuda()
            news.append(nt.expand(w.L, w.B, w.H, 1, w.d))
        q = torch.from_numpy(synth.queries(w, w.H * grp).view(np.int16)).view(torch.bfloat16).cuda()
        q = q.reshape(w.L, w.B, w.H * grp, 1, w.d)
        o = torch.empty((w.L, w.B, w.H * grp, 1, w.d), dtype=torch.bfloat16, device="cuda")
        ws = torch.empty(max(16, cg.attend_paged_workspace_bytes(shp, w.L, w.B, w.H * grp, maxp, P)),
                         dtype=torch.uint8, device="cuda")
        pos = torch.full((w.B,), w.T, dtype=torch.int32, device="cuda")
        lens = pos + 1
        scale = 1.0 / float(np.sqrt(w.d))

        def attend():
            cg.kv_attend_paged(0, w.L, q, pools[0], pools[1], pt, Gd, shp, codec, lens, scale, o, ws, err_flag=err,
                               stream=stream.cuda_stream)

        def step():
            cg.kv_append_paged(0, w.L, news[0], news[1], pos, pt, Gd, shp, codec, pools[0], pools[1], err_flag=err,
                               stream=stream.cuda_stream)
            attend()
            pos.add_(1)
            lens.add_(1)

        ms = _timed(step, steps, warmup, stream)
        ms_att = _timed(attend, steps, 0, stream)
        held = int(lens[0].item())
        per_pos = 2 * (w.d * w.bits // 8 + 4 * (w.d // w.block_c))     # K and V codes + side words
        out["step_ms"] = round(ms, 3)
        out["attend_ms"] = round(ms_att, 3)
        out["history_tokens"] = held
        out["page_size"] = P
        out["query_heads"] = w.H * grp
        out["attend_GBps"] = round(w.L * w.B * w.H * held * per_pos / ms_att / 1e6, 1)
    elif name in ("attend", "attend_tiles", "attend_kivi"):
        # the rolling step with the history consumed by fused decode-phase attention instead of
        # being decoded to bf16: append one token per (layer, b, h), then attention of the
        # grp = 4 query heads of every KV head (32 query heads over 8 KV heads) over the history;
        # attend_tiles: one range per 16 tokens x 64 channels (appends stage the unfinished tile);
        # attend_kivi: the KIVI-style cache of the KIVI workload (3 bits, g = 32, 128-token window)
        grp = 4
        bt = 16 if name == "attend_tiles" else 1
        shp = cg.shape(w.L, w.H, w.d, w.g)
        if name == "attend_kivi":
            codec = cg.Codec(cg.KIVI, w.bits, 64, w.key_tokens, w.val_channels, w.residual)
        else:
            codec = cg.Codec(cg.BLOCK_UNIFORM, w.bits, w.block_c, block_t=bt)
        Gd = cg.alloc_gauge(shp)
        cg.gauge_make(cg.GAUGE_HAAR, shp, seed=w.gauge_seed, G_host=None, G_dev=Gd)
        T_cap = (w.T + warmup + 2 * steps + 1 + 31) // 32 * 32
        caches, news = [], []
        for s in (0, 1):
            X = layer_view(s)
            c = cg.Cache(codec, s, w.L, w.B, w.H, T_cap, w.d)
            cg.kv_encode(s, X, Gd, shp, codec, c, err_flag=err, stream=stream.cuda_stream)
            torch.cuda.synchronize()
            del X
            caches.append(c)
            nt = synth.kv_tensor(w, s, L=1, T=1, t_offset=w.T)
            nt = torch.from_numpy(nt.view(np.int16)).view(torch.bfloat16).cuda()
            news.append(nt.expand(w.L, w.B, w.H, 1, w.d))
        q = torch.from_numpy(synth.queries(w, w.H * grp).view(np.int16)).view(torch.bfloat16).cuda()
        q = q.reshape(w.L, w.B, w.H * grp, 1, w.d)
        o = torch.empty((w.L, w.B, w.H * grp, 1, w.d), dtype=torch.bfloat16, device="cuda")
        ws = torch.empty(max(16, cg.attend_workspace_bytes(shp, w.L, w.B, w.H * grp, T_cap)), dtype=torch.uint8,
                         device="cuda")
        pos = torch.full((w.B,), w.T, dtype=torch.int32, device="cuda")
        lens = pos + 1
        scale = 1.0 / float(np.sqrt(w.d))

        def attend():
            cg.kv_attend(0, w.L, q, caches[0], caches[1], Gd, shp, codec, lens, scale, o, ws, err_flag=err,
                         stream=stream.cuda_stream)

        def step():
            cg.kv_append_step(0, w.L, news[0], news[1], pos, Gd, shp, codec, caches[0], caches[1], None, None,
                              err_flag=err, stream=stream.cuda_stream)
            attend()
            pos.add_(1)
            lens.add_(1)

        ms = _timed(step, steps, warmup, stream)
        # attention alone over the same history length (the positions the last step held)
        ms_att = _timed(attend, steps, 0, stream)
        nc, ns, _ = caches[0].nbytes
        held = int(lens[0].item())
        cache_bytes = 2 * (nc + ns) * held // T_cap          # K and V codes + side words read
        out["step_ms"] = round(ms, 3)
        out["attend_ms"] = round(ms_att, 3)
        out["history_tokens"] = held
        out["query_heads"] = w.H * grp
        out["attend_GBps"] = round(cache_bytes / ms_att / 1e6, 1)
        out["block_t"] = bt
    else:  # rolling decode step
        shp = cg.shape(w.L, w.H, w.d, w.g)
        codec = cg.Codec(cg.BLOCK_UNIFORM, w.bits, w.block_c)
        Gd = cg.alloc_gauge(shp)
        cg.gauge_make(cg.GAUGE_HAAR, shp, seed=w.gauge_seed, G_host=None, G_dev=Gd)
        T_cap = w.T + warmup + steps
        caches, news, hists = [], [], []
        for s in (0, 1):
            X = layer_view(s)
            c = cg.Cache(codec, s, w.L, w.B, w.H, T_cap, w.d)
            cg.kv_encode(s, X, Gd, shp, codec, c, err_flag=err, stream=stream.cuda_stream)
            torch.cuda.synchronize()
            del X
            caches.append(c)
            nt = synth.kv_tensor(w, s, L=1, T=1, t_offset=w.T)          # one new token per (b, h)
            nt = torch.from_numpy(nt.view(np.int16)).view(torch.bfloat16).cuda()
            news.append(nt.expand(w.L, w.B, w.H, 1, w.d))
            hists.append(torch.empty((w.L, w.B, w.H, T_cap, w.d), dtype=torch.bfloat16, device="cuda"))
        pos = torch.full((w.B,), w.T, dtype=torch.int32, device="cuda")

        def step():
            cg.kv_append_step(0, w.L, news[0], news[1], pos, Gd, shp, codec, caches[0], caches[1],
                              hists[0], hists[1], err_flag=err, stream=stream.cuda_stream)
            pos.add_(1)

        ms = _timed(step, steps, warmup, stream)
        hist_elems = 2 * w.L * w.B * w.H * (w.T + warmup + steps // 2) * w.d
        alg = hist_elems * bytes_per_elem(w.bits, w.block_c)
        out["step_ms"] = round(ms, 3)
        out["history_tokens"] = w.T
        out["decode_GBps"] = round(alg / ms / 1e6, 1)
    assert int(err.item()) == 0, f"device error flag {int(err.item())}"
    if probe:
        copy_probe()
    out["cpu_baseline"] = single_threaded(workload_cpu_baseline, name, w, out) if cpu else None
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.workload != WORKLOAD:
        if args.gpus != 1:
            print("bench.py measures one GPU", file=sys.stderr)
            sys.exit(2)
        other_workload(args.workload, args.steps, args.warmup, cpu=not args.no_cpu_baseline, probe=args.copy_probe)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported: the codec path has no "
              f"cross-GPU step (every (layer, head, batch) slice is independent).", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2607_20538_amd import codec as cg
    from paper_2607_20538_amd import synth

    torch.cuda.set_device(0)
    w = synth.WORKLOADS[WORKLOAD]
    shp = cg.shape(w.L, w.H, w.d, w.g)
    codec = cg.Codec(cg.BLOCK_UNIFORM, w.bits, w.block_c)
    Gd = cg.alloc_gauge(shp)
    G_host, _ = cg.gauge_make(cg.GAUGE_HAAR, shp, seed=w.gauge_seed, G_dev=Gd)

    X, Y, caches = [], [], []
    for s in (0, 1):
        bits = synth.kv_tensor(w, s)
        X.append(torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda())
        del bits
        Y.append(torch.empty_like(X[-1]))
        caches.append(cg.Cache(codec, s, w.L, w.B, w.H, w.T, w.d))
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()

    enc_ev, dec_ev = [], []

    def step(record):
        for s in (0, 1):
            if record:
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(stream)
            cg.kv_encode(s, X[s], Gd, shp, codec, caches[s], err_flag=err, stream=stream.cuda_stream)
            if record:
                b.record(stream)
                enc_ev.append((a, b))
        for s in (0, 1):
            if record:
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(stream)
            cg.kv_decode(s, caches[s], Gd, shp, codec, 0, Y[s], err_flag=err, stream=stream.cuda_stream)
            if record:
                b.record(stream)
                dec_ev.append((a, b))

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(True)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    assert int(err.item()) == 0, f"device error flag {int(err.item())}"

    enc_ms = float(np.mean([a.elapsed_time(b) for a, b in enc_ev]))
    dec_ms = float(np.mean([a.elapsed_time(b) for a, b in dec_ev]))
    ms_step = elapsed * 1e3 / args.steps
    n_elem = w.n_elements
    value = n_elem * 2 / (ms_step * 1e-3) / 1e9           # logical bf16 GB/s, encode+decode

    alg = algorithmic_bytes(w)                             # one launch = one of K or V
    dom_name, dom_ms = ("kv_encode", enc_ms) if enc_ms >= dec_ms else ("kv_decode", dec_ms)
    achieved = alg / (dom_ms * 1e-3) / 1e9
    traffic = measured_traffic(args.traffic, dom_name)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic, "kernel": dom_name,
                "kernel_ms": round(dom_ms, 4), "encode_ms": round(enc_ms, 4), "decode_ms": round(dec_ms, 4),
                "alg_bytes_per_launch": int(alg)}

    # HBM ceiling of each kernel's read / write mix: the library's streaming probe (LDS-direct
    # loads through the encoder's tile ring, no arithmetic) moving the same bf16 and code bytes
    elem_b, code_b = n_elem // 2 * 2, n_elem // 2 * w.bits // 8 + n_elem // 2 * 4 // w.block_c
    scratch = torch.empty(code_b, dtype=torch.uint8, device="cuda")

    def probe_gbps(src, rb, dst, wb, reps=20):
        for _ in range(3):
            cg.cg_stream_probe(src, rb, dst, wb, stream=stream.cuda_stream)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            cg.cg_stream_probe(src, rb, dst, wb, stream=stream.cuda_stream)
        b.record(stream)
        torch.cuda.synchronize()
        return (rb + wb) / (a.elapsed_time(b) / reps * 1e-3) / 1e9

    enc_ceil = probe_gbps(X[0], elem_b, scratch, code_b)
    dec_ceil = probe_gbps(scratch, code_b, Y[0], elem_b)
    dom_ceil = enc_ceil if dom_name == "kv_encode" else dec_ceil
    roofline["ceiling"] = {"GBps": round(dom_ceil, 1), "frac": round(achieved / dom_ceil, 4),
                           "kernel": "cg_stream_probe", "read_bytes": elem_b if dom_name == "kv_encode" else code_b,
                           "write_bytes": code_b if dom_name == "kv_encode" else elem_b,
                           "decode_GBps": round(alg / (dec_ms * 1e-3) / 1e9, 1), "decode_ceiling_GBps": round(dec_ceil, 1)}
    del scratch

    if args.copy_probe:
        copy_probe()

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, G_host, args.cpu_sample_layers)

    line = {
        "metric": "KV encode+decode GB/s (bf16 in) and % of MI355X HBM peak, 4-bit g=128",
        "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "llama3-8b-shaped KV: L=32 B=1 H=8 T=8192 d=128 bf16, Haar g=128, "
                               "block-uniform 4-bit n=64",
                   "elements": n_elem, "global_batch": w.B, "seq_len": w.T, "parallelism": "none"},
        "roofline": roofline,
        # per direction, from the HIP-event launch averages: logical bf16 GB/s of the tensor a launch
        # handles (K or V) and key / value vectors per second (one per (layer, batch, head, token))
        "rates": {
            "encode_logical_GBps": round(n_elem / (enc_ms * 1e-3) / 1e9, 1),
            "decode_logical_GBps": round(n_elem / (dec_ms * 1e-3) / 1e9, 1),
            "encode_token_heads_per_s": round(n_elem / 2 / w.d / (enc_ms * 1e-3), -6),
            "decode_token_heads_per_s": round(n_elem / 2 / w.d / (dec_ms * 1e-3), -6),
            "round_trip_token_heads_per_s": round(n_elem / w.d / (ms_step * 1e-3), -6),
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
