#!/usr/bin/env python3
"""Benchmark of the GRKV prefill-compression path on one MI355X.

One step = one grkv_compress call over the whole workload: window attention
over the full cache, pooled top-k retention, retained-cache attention and the
ridge value merge, for every (layer, KV head) unit.  Default workload: a
32-layer x 8-KV-head Llama-3-8B-shaped cache, 32 query heads (G = 4),
head_dim 128, n = 32768 tokens, window 32, budget 2048, pool kernel 7,
lambda 1e-2, bfloat16, synthetic seeded inputs resident in HBM.

Prints one JSON line: heads/s (value), ms per step and per layer, the
roofline of the dominant kernel (its duration measured with HIP events around
its launches inside the timed steps), and the float64 oracle's CPU throughput
on a bounded sample of the same workload.  Besides: the same workload as one
call per layer (`per_layer_calls`, not `value`) and the device copy bandwidth
(`copy_gbs`, the practical ceiling for streaming), and the key step of GRKV
run after the value step (`key_step`: grkv_compress_kv on the same workload,
its CG iterations and the time of one CG iteration against the MFMA peak), and
the carrier-concentration diagnostic (`carrier`: the key-cosine matcher and
the load metrics, against the MFMA peak).

  python bench.py [--steps K] [--warmup W] [--config 4] [--no-cpu-baseline] [--no-per-layer]
                  [--no-key-step] [--no-carrier]
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "compressed KV heads/sec (and ms per layer) at n=32k; % of HBM roofline"
HBM_PEAK_GBS = 8000.0   # MI355X HBM3E peak


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--budget", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-per-layer", dest="per_layer", action="store_false",
                    help="skip the one-call-per-layer measurement")
    ap.add_argument("--no-key-step", dest="key_step", action="store_false",
                    help="skip the key-step measurement (grkv_compress_kv)")
    ap.add_argument("--no-front-ends", dest="front_ends", action="store_false",
                    help="skip the ragged-budget front-end timings")
    ap.add_argument("--no-carrier", dest="carrier", action="store_false",
                    help="skip the carrier-concentration measurement")
    ap.add_argument("--no-h2o", dest="h2o", action="store_false",
                    help="skip the H2O front-end (accumulated-attention scores)")
    ap.add_argument("--no-configs", dest="configs", action="store_false",
                    help="skip the one-layer 32k and 4-layer 128k workloads")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a 1 GiB device copy (for counter calibration)")
    return ap.parse_args()


class Hip:
    """The few HIP runtime calls the benchmark needs for raw events."""

    def __init__(self):
        self.lib = ctypes.CDLL("libamdhip64.so")

    def event(self):
        ev = ctypes.c_void_p()
        if self.lib.hipEventCreate(ctypes.byref(ev)) != 0:
            raise RuntimeError("hipEventCreate failed")
        return ev

    def elapsed_ms(self, a, b):
        ms = ctypes.c_float()
        if self.lib.hipEventElapsedTime(ctypes.byref(ms), a, b) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def destroy(self, ev):
        self.lib.hipEventDestroy(ev)


def source_hash(files):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def copy_calibration():
    import torch
    x = torch.ones(2 ** 30 // 4, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(5):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": 2 ** 30, "launches": 5}), flush=True)


def blas_threads():
    """Threads the oracle's numpy linear algebra runs on (its matmuls are the
    only multi-threaded part of it)."""
    try:
        from threadpoolctl import threadpool_info
        return int(max([i.get("num_threads", 1) for i in threadpool_info()] or [1]))
    except Exception:
        return 1


def host_info():
    """The host the oracle is timed on: usable cores and the CPU model."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"host_cores": len(os.sched_getaffinity(0)), "cpu_model": model}


def oracle_record(done, total, el, what, unit="heads/s", per=1.0):
    rec = {"value": per * done / el, "unit": unit, "cores": blas_threads(), "kind": "oracle",
           "sample": "%d of %d %s, %.1f s" % (done, total, what, el),
           "label": "plain fp64 reference, not an optimized CPU implementation"}
    rec.update(host_info())
    return rec


def cpu_baseline(cfg, q, K, V, seconds, units=None):
    """The oracle as it stands, on a bounded sample of whole units."""
    import workloads as W
    from oracle import grkv_oracle as O
    units = list(range(cfg.units)) if units is None else list(units)
    done, t0 = 0, time.perf_counter()
    while done < len(units) and (done < 2 or time.perf_counter() - t0 < seconds):
        u = units[done]
        qd, Kd, Vd = (W.decode(a[u], cfg.dtype) for a in (q, K, V))
        O.compress_unit(qd, Kd, Vd, cfg.window, cfg.budget, cfg.pool_kernel, cfg.lam)
        done += 1
    el = time.perf_counter() - t0
    return oracle_record(done, cfg.units, el, "units (whole units, float64 numpy oracle)")


def cpu_baseline_key(cfg, q, K, V, seconds):
    """The oracle's value step followed by its key step (float64 CG to 1e-12),
    on a bounded sample of whole units."""
    import workloads as W
    from oracle import grkv_key_oracle as KO
    done, t0 = 0, time.perf_counter()
    while done < cfg.units and (done < 2 or time.perf_counter() - t0 < seconds):
        qd, Kd_, Vd_ = (W.decode(a[done], cfg.dtype) for a in (q, K, V))
        KO.grkv_unit(qd, Kd_, Vd_, cfg.window, cfg.budget, cfg.pool_kernel, cfg.lam, cfg.lam)
        done += 1
    el = time.perf_counter() - t0
    return oracle_record(done, cfg.units, el,
                         "units (whole units: value and key step, float64 numpy oracle)")


def carrier(args, cfg, G, hip, stream, Kd, res, host=None):
    """The carrier-concentration diagnostic on the same workload: the key-cosine
    matcher over every cache position against the retained keys of the
    compress call, then the per-unit load metrics.  Algorithmic flops per unit:
    2 (n - c) c d (the similarities of the evicted tokens)."""
    import numpy as np
    import torch

    U, n, c, d = cfg.units, cfg.n, cfg.budget, cfg.head_dim
    if cfg.dtype != "bf16":
        return None
    print("bench: carrier diagnostics", file=sys.stderr, flush=True)
    a, cnt, met, lc = G.carrier_stats(Kd, res.idx, cfg.group, res.stats)
    torch.cuda.synchronize()
    reps = max(1, min(args.steps, 5))
    c0, c1 = hip.event(), hip.event()
    hip.lib.hipEventRecord(c0, ctypes.c_void_p(stream.cuda_stream))
    for _ in range(reps):
        G.carrier_stats(Kd, res.idx, cfg.group, res.stats, assign=a, counts=cnt, metrics=met,
                        l_common=lc)
    hip.lib.hipEventRecord(c1, ctypes.c_void_p(stream.cuda_stream))
    torch.cuda.synchronize()
    ms = hip.elapsed_ms(c0, c1) / reps
    flops = U * 2.0 * (n - c) * c * d
    tflops = flops / (ms / 1e3) / 1e12
    m = met.cpu().numpy().astype(np.float64)
    summary = {k: float(np.nanmean(m[:, i])) for i, k in enumerate(G.CARRIER_METRICS)}
    summary["b_over_c"] = summary["b"] / c
    summary["b_eff_over_c"] = summary["b_eff"] / c
    cpu = None
    if host is not None:
        import workloads as W
        from oracle import grkv_carrier_oracle as CO
        idx = res.idx.cpu().numpy().astype(np.int64)
        done, t0 = 0, time.perf_counter()
        while done < U and (done < 1 or time.perf_counter() - t0 < min(args.cpu_seconds, 10.0)):
            CO.carrier_metrics(CO.carrier_assignment(W.decode(host[done], cfg.dtype), idx[done]),
                               idx[done])
            done += 1
        el = time.perf_counter() - t0
        cpu = oracle_record(done, U, el, "units (float64 numpy oracle)")
    return {
        "ms_per_call": ms,
        "heads_per_s": U / (ms / 1e3),
        "l_common": float(lc.cpu()[0]),
        "macro_metrics": summary,
        "roofline": {"bound": "mfma", "kernel": "match_kernel + stats_kernel",
                     "achieved": tflops, "peak": 2500.0, "unit": "TFLOP/s",
                     "frac": tflops / 2500.0, "traffic": None},
        "cpu_baseline": cpu,
    }


def front_ends(args, cfg, G, hip, stream, qd, Kd, Vd, res, host=None):
    """The budget front-ends on the same workload: ragged compression with the
    pyramid schedule (mean budget c, top layer c / 2, bottom 3c / 2) and with
    the adaptive per-head allocation computed on the GPU from the pooled scores
    of the uniform call (the allocation kernel timed on its own)."""
    import torch

    U, w, c = cfg.units, cfg.window, cfg.budget
    print("bench: budget front-ends", file=sys.stderr, flush=True)
    reps = max(1, min(args.steps, 5))

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        a, b = hip.event(), hip.event()
        hip.lib.hipEventRecord(a, ctypes.c_void_p(stream.cuda_stream))
        for _ in range(reps):
            fn()
        hip.lib.hipEventRecord(b, ctypes.c_void_p(stream.cuda_stream))
        torch.cuda.synchronize()
        return hip.elapsed_ms(a, b) / reps

    import numpy as np

    pooled = G.intermediates(res)["pooled"].contiguous().clone()
    budgets = G.adaptive_budgets(pooled, cfg.layers, cfg.kv_heads, c, w)
    ms_alloc = timed(lambda: G.adaptive_budgets(pooled, cfg.layers, cfg.kv_heads, c, w,
                                                out=budgets))
    # the allocation reads every pooled score once (algorithmic bytes)
    alloc_gbs = pooled.numel() * 4 / (ms_alloc / 1e3) / 1e9
    out = {"adaptive_allocation": {
        "ms_per_call": ms_alloc, "kernel": "adaptive_kernel",
        "roofline": {"bound": "hbm", "achieved": alloc_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": alloc_gbs / HBM_PEAK_GBS, "traffic": None}}}
    full_prob = G.STAGES.index("full_prob")
    esz = 2 if cfg.dtype == "bf16" else 4
    for name, b in (("pyramid", G.pyramid_budgets(cfg.layers, cfg.kv_heads, c, w, cfg.n)),
                    ("adaptive", budgets.cpu().numpy())):
        dt = G.GRKV_BF16 if cfg.dtype == "bf16" else G.GRKV_F32
        ws = torch.empty(max(256, G.workspace_bytes_ragged(U, cfg.group, cfg.head_dim, dt, cfg.n,
                                                           w, b)), dtype=torch.uint8, device="cuda")
        r = G.compress_ragged(qd, Kd, Vd, w, b, cfg.pool_kernel, cfg.lam, workspace=ws)
        ms = timed(lambda: G.compress_ragged(qd, Kd, Vd, w, b, cfg.pool_kernel, cfg.lam,
                                             workspace=ws, out=r))
        # the dominant stage (full-cache pass B), timed with events on the stream
        evs = (ctypes.c_void_p * (2 * G.NUM_STAGES))()
        e0, e1 = hip.event(), hip.event()
        evs[2 * full_prob], evs[2 * full_prob + 1] = e0.value, e1.value
        fp = []
        for _ in range(reps):
            G.compress_ragged(qd, Kd, Vd, w, b, cfg.pool_kernel, cfg.lam, workspace=ws, out=r,
                              stage_events=evs)
            torch.cuda.synchronize()
            fp.append(hip.elapsed_ms(e0, e1))
        fp_ms = float(np.mean(fp))
        gbs = U * (2 * cfg.n * cfg.head_dim * esz + cfg.group * w * cfg.head_dim * esz) / \
            (fp_ms / 1e3) / 1e9
        out[name] = {"ms_per_call": ms, "heads_per_s": U / (ms / 1e3),
                     "distinct_budgets": int(len(set(b.tolist()))),
                     "budget_min": int(b.min()), "budget_max": int(b.max()),
                     "roofline": {"bound": "hbm", "kernel": "full_prob", "achieved": gbs,
                                  "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                  "frac": gbs / HBM_PEAK_GBS, "traffic": None}}
    if host is not None:
        # the oracle's allocation (float64 joint top-k per layer) on a few layers
        from oracle import grkv_frontend_oracle as FO
        pl = pooled.cpu().numpy().astype(np.float64)
        H = cfg.kv_heads
        done, t0 = 0, time.perf_counter()
        while done < cfg.layers and (done < 1 or time.perf_counter() - t0 < 5.0):
            FO.adaptive_budgets(pl[done * H:(done + 1) * H], 1, H, c, w)
            done += 1
        el = time.perf_counter() - t0
        rec = oracle_record(done, cfg.layers, el, "layers (float64 numpy lexsort)",
                            unit="layers/s")
        rec["cores"] = 1   # a sort: numpy runs it on one thread
        out["adaptive_allocation"]["cpu_baseline"] = rec
        out["adaptive_allocation"]["layers_per_s"] = cfg.layers / (ms_alloc / 1e3)
    return out


def key_step(args, cfg, G, hip, stream, qd, Kd, Vd, host=None):
    """The key step after the value step (grkv_compress_kv) on the same
    workload: time per call and of its key stage (default CG settings), CG
    iterations per unit, and the time of one CG iteration (one operator pass
    plus one CG update), from the difference of two runs with a fixed
    iteration count.  Algorithmic flops of one operator application per unit:
    a V*^T and (X o W D) V* (2mcd each) and W D (2m^2 c)."""
    import numpy as np
    import torch

    U, w, c, d, m = cfg.units, cfg.window, cfg.budget, cfg.head_dim, cfg.group * cfg.window
    if G.workspace_bytes_kv(U, cfg.group, d, 0 if cfg.dtype == "bf16" else 1, cfg.n, w, c) == 0:
        return None
    print("bench: key step", file=sys.stderr, flush=True)
    res, kstar, info = G.compress_kv(qd, Kd, Vd, w, c, cfg.pool_kernel, cfg.lam)
    ks = G.STAGES.index("key")

    def run(reps, **kw):
        evs = []
        for _ in range(reps):
            arr = (ctypes.c_void_p * (2 * G.NUM_STAGES))()
            a, b = hip.event(), hip.event()
            arr[2 * ks], arr[2 * ks + 1] = a.value, b.value
            evs.append((arr, a, b))
        c0, c1 = hip.event(), hip.event()
        hip.lib.hipEventRecord(c0, ctypes.c_void_p(stream.cuda_stream))
        for arr, _, _ in evs:
            G.compress_kv(qd, Kd, Vd, w, c, cfg.pool_kernel, cfg.lam, workspace=res.workspace,
                          out=res, k_star=kstar, cg_info=info, stage_events=arr, **kw)
        hip.lib.hipEventRecord(c1, ctypes.c_void_p(stream.cuda_stream))
        torch.cuda.synchronize()
        return (float(np.mean([hip.elapsed_ms(a, b) for _, a, b in evs])),
                hip.elapsed_ms(c0, c1) / reps)

    for _ in range(args.warmup):
        run(1)
    reps = max(1, min(args.steps, 5))
    key_ms, call_ms = run(reps)
    it = info[:, 0].cpu().numpy()
    state = info[:, 2].cpu().numpy()
    # the first 10 iterations run with one block per unit (all units active)
    n1, n2 = 0, 8
    t1, _ = run(reps, max_iter=n1, tol=0.0)
    t2, _ = run(reps, max_iter=n2, tol=0.0)
    it_ms = (t2 - t1) / (n2 - n1)
    flops = U * (4.0 * m * c * d + 2.0 * m * m * c)
    tflops = flops / (it_ms / 1e3) / 1e12
    # Algorithm 1 with two alternating steps (the second value step on the
    # generic fp32 kernels at the moved keys, then a second key step)
    res2, k2, i2 = G.compress_kv(qd, Kd, Vd, w, c, cfg.pool_kernel, cfg.lam, steps=2)
    torch.cuda.synchronize()
    s0, s1 = hip.event(), hip.event()
    hip.lib.hipEventRecord(s0, ctypes.c_void_p(stream.cuda_stream))
    for _ in range(reps):
        G.compress_kv(qd, Kd, Vd, w, c, cfg.pool_kernel, cfg.lam, steps=2,
                      workspace=res2.workspace, out=res2, k_star=k2, cg_info=i2)
    hip.lib.hipEventRecord(s1, ctypes.c_void_p(stream.cuda_stream))
    torch.cuda.synchronize()
    steps2_ms = hip.elapsed_ms(s0, s1) / reps
    del res2, k2, i2
    cpu = None
    if host is not None:
        print("bench: timing the key-step oracle on the host", file=sys.stderr, flush=True)
        cpu = cpu_baseline_key(cfg, *host, min(args.cpu_seconds, 10.0))
    return {
        "ms_per_call": call_ms,
        "key_stage_ms": key_ms,
        "heads_per_s": U / (call_ms / 1e3),
        "cg_iterations_mean": float(it.mean()),
        "cg_iterations_max": int(it.max()),
        "units_converged": int((state == G.KEY_CONVERGED).sum()),
        "cg_tol": 1e-5,
        "iteration_ms": it_ms,
        "ms_per_call_steps2": steps2_ms,
        "roofline": {"bound": "mfma",
                     "kernel": "key_ring_kernel operator pass with the CG update (one iteration)",
                     "achieved": tflops, "peak": 2500.0, "unit": "TFLOP/s",
                     "frac": tflops / 2500.0, "traffic": None,
                     "note": "fp32-accurate products as three bf16 MFMAs each; X streamed from "
                             "HBM (written once per key step by key_x)"},
        "cpu_baseline": cpu,
    }


def h2o(args, G, hip, stream, want_cpu):
    """The H2O front-end on one layer of the 32-layer workload (8 KV heads,
    n = 32768): the accumulated-attention scores of every prefix token over all
    prompt queries (grkv_h2o_scores), then compression from those scores with
    no pooling (grkv_compress_scored).  Algorithmic flops of the scores: the
    causal Q K^T of both passes, 2 * G * n(n+1)/2 * d * 2 per unit."""
    import numpy as np
    import torch
    import workloads as W

    cfg = W.config(4, layers=1)
    print("bench: H2O front-end (%d units, n=%d)" % (cfg.units, cfg.n), file=sys.stderr, flush=True)
    q, K, V = W.make_batch(cfg)
    q_all = W.make_prompt_queries(cfg, q, K)
    dev = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    qd, Kd, Vd, qa = dev(q), dev(K), dev(V), dev(q_all)
    w, c, n, d, Gq, U = cfg.window, cfg.budget, cfg.n, cfg.head_dim, cfg.group, cfg.units
    ws = torch.empty(G.h2o_workspace_bytes(U, Gq, d, G.GRKV_BF16, n), dtype=torch.uint8, device="cuda")
    s = G.h2o_scores(qa, Kd, w, workspace=ws)
    res = G.compress_scored(qd, Kd, Vd, w, c, 1, cfg.lam, s)
    torch.cuda.synchronize()

    def timed(fn, reps):
        a, b = hip.event(), hip.event()
        hip.lib.hipEventRecord(a, ctypes.c_void_p(stream.cuda_stream))
        for _ in range(reps):
            fn()
        hip.lib.hipEventRecord(b, ctypes.c_void_p(stream.cuda_stream))
        torch.cuda.synchronize()
        return hip.elapsed_ms(a, b) / reps

    ms_scores = timed(lambda: G.h2o_scores(qa, Kd, w, workspace=ws, out=s), 3)
    # one layer's inputs fit in the last-level cache: a 512 MB read-modify-write
    # before each timed compression (outside its events) evicts them
    flush = torch.empty(2 ** 27, dtype=torch.float32, device="cuda")
    comp = []
    for _ in range(5):
        flush.add_(1.0)
        comp.append(timed(lambda: G.compress_scored(qd, Kd, Vd, w, c, 1, cfg.lam, s,
                                                    workspace=res.workspace, out=res), 1))
    del flush
    ms_comp = float(np.mean(comp))
    flops = U * 2 * Gq * (n * (n + 1) / 2) * d * 2
    tflops = flops / (ms_scores / 1e3) / 1e12
    out = {"workload": "llama3-8b-layer-n32k (layer 0 of the 32-layer workload)", "units": U,
           "ms_scores": ms_scores, "ms_compress_scored": ms_comp,
           "heads_per_s": U / ((ms_scores + ms_comp) / 1e3),
           "roofline": {"bound": "mfma", "kernel": "h2o_lse + h2o_colsum", "achieved": tflops,
                        "peak": 2500.0, "unit": "TFLOP/s", "frac": tflops / 2500.0,
                        "traffic": None}}
    if want_cpu:
        # the oracle forms each head's n x n attention: timed on the same
        # recipe at n = 4096 (one unit), the scores and the compression
        from oracle import grkv_frontend_oracle as FO
        cs = W.config(4, layers=1, n=4096, budget=256)
        q2, K2, V2 = W.make_batch(cs, units=[0])
        qa2 = W.make_prompt_queries(cs, q2, K2, units=[0])
        t0 = time.perf_counter()
        done = 0
        while done < 1 or time.perf_counter() - t0 < 3.0:
            FO.compress_h2o(W.decode(qa2[0], cs.dtype), W.decode(q2[0], cs.dtype),
                            W.decode(K2[0], cs.dtype), W.decode(V2[0], cs.dtype), cs.window,
                            cs.budget, cs.lam)
            done += 1
        el = time.perf_counter() - t0
        rec = oracle_record(done, done, el, "runs of one unit at n = 4096 (H2O scores and "
                                            "compression, float64 numpy oracle; the oracle "
                                            "forms n x n attention, so not at n = 32768)")
        out["cpu_baseline"] = rec
    del qd, Kd, Vd, qa, res, s, ws
    torch.cuda.empty_cache()
    return out


def path_bytes_per_unit(cfg):
    """Algorithmic bytes of one unit: read K, V and q_obs once, write idx,
    k_out (input dtype) and v_out (fp32) once."""
    esz = 2 if cfg.dtype == "bf16" else 4
    n, d, c, m = cfg.n, cfg.head_dim, cfg.budget, cfg.group * cfg.window
    return 2 * n * d * esz + m * d * esz + c * 4 + c * d * esz + c * d * 4


def other_configs(args, G, hip, stream, want_cpu):
    """The other workloads, each timed as one call over all of its units (the
    same measurement as the headline, at their sizes): the
    one-layer 32k cache at budgets 1024 and 2048, and the 4-layer 128k cache
    (window 64, so m = 256 stacked rows), with the oracle timed on a bounded
    sample of each."""
    import numpy as np
    import torch
    import workloads as W

    out = {}
    full_prob = G.STAGES.index("full_prob")
    for key, cfg in (("llama3-8b-layer-n32k-c1024", W.config(3, budget=1024)),
                     ("llama3-8b-layer-n32k-c2048", W.config(3, budget=2048)),
                     ("llama3-8b-4layer-n128k", W.config(5))):
        print("bench: %s (%d units, n=%d, c=%d)" % (key, cfg.units, cfg.n, cfg.budget),
              file=sys.stderr, flush=True)
        q, K, V = W.make_batch(cfg)
        qd, Kd, Vd = (torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
                      for a in (q, K, V))
        w, c = cfg.window, cfg.budget
        res = G.compress(qd, Kd, Vd, w, c, cfg.pool_kernel, cfg.lam)
        for _ in range(args.warmup):
            G.compress(qd, Kd, Vd, w, c, cfg.pool_kernel, cfg.lam, workspace=res.workspace, out=res)
        torch.cuda.synchronize()
        reps = max(3, min(args.steps, 10))
        evs = []
        for _ in range(reps):
            arr = (ctypes.c_void_p * (2 * G.NUM_STAGES))()
            a, b = hip.event(), hip.event()
            arr[2 * full_prob], arr[2 * full_prob + 1] = a.value, b.value
            evs.append((arr, a, b, hip.event(), hip.event()))
        # a one-layer cache (134 MB at n = 32k) fits in the 256 MB last-level
        # cache: each timed call is preceded, outside its events, by a 512 MB
        # read-modify-write that evicts the previous call's inputs
        flush = torch.empty(2 ** 27, dtype=torch.float32, device="cuda")
        for arr, _, _, c0, c1 in evs:
            flush.add_(1.0)
            hip.lib.hipEventRecord(c0, ctypes.c_void_p(stream.cuda_stream))
            G.compress(qd, Kd, Vd, w, c, cfg.pool_kernel, cfg.lam, workspace=res.workspace,
                       out=res, stage_events=arr)
            hip.lib.hipEventRecord(c1, ctypes.c_void_p(stream.cuda_stream))
        torch.cuda.synchronize()
        del flush
        ms = float(np.mean([hip.elapsed_ms(c0, c1) for _, _, _, c0, c1 in evs]))
        fp_ms = float(np.mean([hip.elapsed_ms(a, b) for _, a, b, _, _ in evs]))
        esz = 2
        fp_bytes = cfg.units * (2 * cfg.n * cfg.head_dim * esz + cfg.group * w * cfg.head_dim * esz)
        path = cfg.units * path_bytes_per_unit(cfg)
        rec = {"units": cfg.units, "n": cfg.n, "window": w, "budget": c, "m": cfg.group * w,
               "ms_per_call": ms, "ms_per_layer": ms / cfg.layers,
               "heads_per_s": cfg.units / (ms / 1e3),
               "roofline": {"bound": "hbm", "kernel": "full_prob",
                            "achieved": fp_bytes / (fp_ms / 1e3) / 1e9, "peak": HBM_PEAK_GBS,
                            "unit": "GB/s",
                            "frac": fp_bytes / (fp_ms / 1e3) / 1e9 / HBM_PEAK_GBS,
                            "path_frac": path / (ms / 1e3) / 1e9 / HBM_PEAK_GBS,
                            "traffic": None}}
        if want_cpu:
            rec["cpu_baseline"] = cpu_baseline(cfg, q, K, V, min(args.cpu_seconds, 6.0))
        out[key] = rec
        del res, qd, Kd, Vd, q, K, V
        torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path (units are "
              "independent, so a multi-GPU run would give each GPU its own units with no "
              "communication)", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration()
        return

    import numpy as np
    import torch

    import paper_2605_31105_amd as G
    import workloads as W

    cfg = W.config(args.config)
    if args.budget:
        cfg = W.config(args.config, budget=args.budget)
    U, Gq, w, d, n, c = cfg.units, cfg.group, cfg.window, cfg.head_dim, cfg.n, cfg.budget
    m = Gq * w
    print("bench: generating %s (%d units, n=%d)" % (cfg.name, U, n), file=sys.stderr, flush=True)
    t_gen = time.perf_counter()
    q, K, V = W.make_batch(cfg)
    print("bench: generated in %.1f s" % (time.perf_counter() - t_gen), file=sys.stderr, flush=True)

    def dev(a):
        if cfg.dtype == "bf16":
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(a).cuda()

    qd, Kd, Vd = dev(q), dev(K), dev(V)
    torch.cuda.synchronize()
    res = G.compress(qd, Kd, Vd, w, c, cfg.pool_kernel, cfg.lam)   # allocates outputs once
    ws, out = res.workspace, res
    for _ in range(args.warmup):
        G.compress(qd, Kd, Vd, w, c, cfg.pool_kernel, cfg.lam, workspace=ws, out=out)
    torch.cuda.synchronize()
    print("bench: warmup done", file=sys.stderr, flush=True)

    hip = Hip()
    timed = {"full_prob": G.STAGES.index("full_prob"), "full_lse": G.STAGES.index("full_lse")}
    slots = []
    for _ in range(args.steps):
        arr = (ctypes.c_void_p * (2 * G.NUM_STAGES))()
        evs = {}
        for name, s in timed.items():
            a, b = hip.event(), hip.event()
            arr[2 * s], arr[2 * s + 1] = a.value, b.value
            evs[name] = (a, b)
        slots.append((arr, evs))
    stream = torch.cuda.current_stream()
    e0, e1 = hip.event(), hip.event()

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    hip.lib.hipEventRecord(e0, ctypes.c_void_p(stream.cuda_stream))
    for k in range(args.steps):
        G.compress(qd, Kd, Vd, w, c, cfg.pool_kernel, cfg.lam, workspace=ws, out=out,
                   stage_events=slots[k][0])
    hip.lib.hipEventRecord(e1, ctypes.c_void_p(stream.cuda_stream))
    torch.cuda.synchronize()
    t1 = time.perf_counter()

    ms_wall = (t1 - t0) * 1e3 / args.steps
    ms_events = hip.elapsed_ms(e0, e1) / args.steps
    stage_ms = {name: float(np.mean([hip.elapsed_ms(*ev[name]) for _, ev in slots]))
                for name in timed}
    ms_step = ms_wall
    heads_s = U / (ms_step / 1e3)

    # algorithmic bytes (read once / written once), per unit
    esz = 2 if cfg.dtype == "bf16" else 4
    kv_bytes = 2 * n * d * esz
    q_bytes = m * d * esz
    path_bytes = path_bytes_per_unit(cfg)
    alg = {"full_prob": U * (kv_bytes + q_bytes), "full_lse": U * (n * d * esz + q_bytes)}
    dom = max(stage_ms, key=stage_ms.get)
    achieved = alg[dom] / (stage_ms[dom] / 1e3) / 1e9

    traffic = None
    tfile = os.path.join(ROOT, "profiles", "traffic_full_prob_llama3-8b-32layer-n32k.json")
    if os.path.exists(tfile) and dom == "full_prob" and args.config == 4:
        t = json.load(open(tfile))
        if t.get("source_hash") == source_hash(t.get("sources", [])):
            traffic = t.get("bytes_per_launch")

    # the same workload as one call per layer (the kv_heads units of a layer
    # per call, back to back on one stream): the pattern of a prefill that
    # compresses each layer as it finishes
    per_layer = None
    if args.per_layer and cfg.layers > 1:
        upl = cfg.kv_heads
        calls = []
        for l in range(cfg.layers):
            sl = slice(l * upl, (l + 1) * upl)
            a = (qd[sl], Kd[sl], Vd[sl])
            calls.append((a, G.compress(*a, w, c, cfg.pool_kernel, cfg.lam)))
        def layer_step():
            for a, r in calls:
                G.compress(*a, w, c, cfg.pool_kernel, cfg.lam, workspace=r.workspace, out=r)
        for _ in range(args.warmup):
            layer_step()
        torch.cuda.synchronize()
        p0, p1 = hip.event(), hip.event()
        hip.lib.hipEventRecord(p0, ctypes.c_void_p(stream.cuda_stream))
        for _ in range(args.steps):
            layer_step()
        hip.lib.hipEventRecord(p1, ctypes.c_void_p(stream.cuda_stream))
        torch.cuda.synchronize()
        ms_pl = hip.elapsed_ms(p0, p1) / args.steps
        per_layer = {"units_per_call": upl, "calls_per_step": cfg.layers,
                     "ms_per_step": ms_pl, "ms_per_layer": ms_pl / cfg.layers,
                     "heads_per_s": U / (ms_pl / 1e3)}

    # device copy bandwidth on this GPU (read + write of 1 GiB), the practical
    # ceiling for streaming kernels
    x = torch.empty(2 ** 28, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    y.copy_(x)
    torch.cuda.synchronize()
    c0, c1 = hip.event(), hip.event()
    hip.lib.hipEventRecord(c0, ctypes.c_void_p(stream.cuda_stream))
    for _ in range(5):
        y.copy_(x)
    hip.lib.hipEventRecord(c1, ctypes.c_void_p(stream.cuda_stream))
    torch.cuda.synchronize()
    copy_gbs = 5 * 2 * 2 ** 30 / (hip.elapsed_ms(c0, c1) / 1e3) / 1e9
    del x, y

    key = (key_step(args, cfg, G, hip, stream, qd, Kd, Vd,
                    host=None if args.no_cpu_baseline else (q, K, V))
           if args.key_step else None)
    car = (carrier(args, cfg, G, hip, stream, Kd, out, host=None if args.no_cpu_baseline else K)
           if args.carrier else None)

    fe = (front_ends(args, cfg, G, hip, stream, qd, Kd, Vd, out,
                     host=None if args.no_cpu_baseline else True) if args.front_ends else None)

    cpu = None
    if not args.no_cpu_baseline:
        print("bench: timing the oracle on the host", file=sys.stderr, flush=True)
        cpu = cpu_baseline(cfg, q, K, V, args.cpu_seconds)

    path_gbs = U * path_bytes / (ms_step / 1e3) / 1e9
    h2o_rec = None
    if args.h2o and args.config == 4:
        h2o_rec = h2o(args, G, hip, stream, not args.no_cpu_baseline)
    others = None
    if args.configs and args.config == 4:
        del q, K, V
        others = other_configs(args, G, hip, stream, not args.no_cpu_baseline)

    line = {
        "metric": METRIC,
        "value": heads_s,
        "unit": "heads/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "ms_per_layer": ms_step / cfg.layers,
        "ms_per_step_events": ms_events,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": cfg.name, "layers": cfg.layers, "kv_heads": cfg.kv_heads,
                   "query_heads": cfg.kv_heads * Gq, "head_dim": d, "n": n, "window": w,
                   "budget": c, "pool_kernel": cfg.pool_kernel, "lambda": cfg.lam,
                   "units": U},
        "path_hbm_frac": path_gbs / HBM_PEAK_GBS,
        "copy_gbs": copy_gbs,
        "per_layer_calls": per_layer,
        "stage_ms": stage_ms,
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "frac_of_copy": achieved / copy_gbs,
                     "traffic": traffic,
                     # the whole call: every unit's algorithmic bytes over the step time
                     "path_achieved": path_gbs, "path_frac": path_gbs / HBM_PEAK_GBS,
                     "path_bytes_per_unit": path_bytes},
        "key_step": key,
        "carrier": car,
        "front_ends": fe,
        "configs": others,
        "h2o": h2o_rec,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
