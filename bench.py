#!/usr/bin/env python3
"""Benchmark: one decoder layer with contextual sparsity per step, OPT-175B shape.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload opt175b_b1]

Batch 1 (default, --workload opt175b_b1): a step is one dv_sparse_block call: both
predictors (low-rank GEMVs and top-k), gathered QKV, KV append, split-KV attention,
gathered out-projection, residual, layer norms, gathered fc1/ReLU/fc2 and residual, for
one token. value = microseconds per layer per token.

Batch 32 (--workload opt175b_b32): a step is dv_sparse_attn (each sequence's own 32 of
96 heads, own KV length) followed by dv_sparse_mlp on the union of the 32 sequences'
Zipf-skewed neuron sets, on the matrix cores. value = step time / 32.

Inputs are seeded synthetic layers already resident in HBM; R independent layer
replicas are cycled so that nothing a step reads is served from the 256 MB Infinity
Cache (default R = 10 at batch 1, whose selected keys and values are 33.5 MB per
replica; 4 at batch 32, which reads 675 MB of keys and values per step). Prints ONE JSON line: the value, the roofline of the dominant kernel from HIP
events stamped by its launches' own dispatches on the library's stream, and the fp64
oracle timed on this host's cores on a bounded sample.
"""
import argparse
import collections
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "µs/layer/token sparse block at OPT-175B shape, batch 1; achieved HBM GB/s vs peak"
METRIC_B32 = ("µs/layer/token sparse attention + union MLP at OPT-175B shape, batch 32 (sets given); "
              "achieved HBM GB/s vs peak")
PEAK_HBM_GBPS = 8000.0
ROOFLINE_EVERY = 8   # timed steps per event-timed launch of the dominant kernel


def kernel_bytes(cfg, pos):
    """Algorithmic bytes per launch of each kernel of one block call (look-ahead mode)."""
    sw, skv = cfg.wbytes, cfg.kvbytes
    d, kh, km, dh, r = cfg.d, cfg.k_heads, cfg.k_mlp, cfg.dh, cfg.r
    return {
        "pred_hidden": 2 * r * d * sw,                     # AT_h and AT_m rows
        "pred_scores": (cfg.H + cfg.N) * r * sw,           # BT_h and BT_m rows
        "qkv": 3 * kh * dh * d * sw,                       # W^Q, W^K, W^V rows of S_A
        "attn": 2 * kh * (pos + 1) * dh * skv,             # keys and values of S_A
        "oproj": kh * dh * d * sw,                         # W^O rows of S_A
        "fc1": km * d * sw,                                # W1T rows of S_M
        "fc2": km * d * sw,                                # W2T rows of S_M
    }


def batch_kernel_bytes(cfg, heads, sets, pos):
    """Algorithmic bytes per launch of the batched attention + union MLP of one step."""
    sw, skv = cfg.wbytes, cfg.kvbytes
    nu_h = len(set(int(h) for row in heads for h in row))
    nu = len(set(int(i) for row in sets for i in row))
    d, dh = cfg.d, cfg.dh
    return {
        "qkv": 3 * nu_h * dh * d * sw,                                   # Q/K/V rows of the head union
        "attn": sum(len(heads[b]) * (int(pos[b]) + 1) * 2 * dh * skv for b in range(len(pos))),
        "oproj": nu_h * dh * d * sw,                                     # W^O rows of the head union
        "fc1": nu * d * sw,                                              # W1T rows of the neuron union
        "fc2": nu * d * sw,                                              # W2T rows of the neuron union
    }, nu, nu_h


# Sources each kernel is compiled from (with the build flags); the HBM counters committed
# under profiles/ are valid only for the sources they were taken with.
_CSRC = os.path.join(ROOT, "paper_2310_17157_amd", "csrc")
KERNEL_SOURCES = {
    "pred_hidden": ["dv_predict.hip", "dv_rowdot.hpp", "dv_internal.hpp", "dv_select.hpp"],
    "pred_scores": ["dv_predict.hip", "dv_rowdot.hpp", "dv_internal.hpp", "dv_select.hpp"],
    "qkv": ["dv_attn.hip", "dv_rowdot.hpp", "dv_internal.hpp", "dv_select.hpp"],
    "attn": ["dv_attn.hip", "dv_rowdot.hpp", "dv_internal.hpp", "dv_select.hpp"],
    "oproj": ["dv_axpy.hip", "dv_internal.hpp", "dv_select.hpp"],
    "fc2": ["dv_axpy.hip", "dv_internal.hpp", "dv_select.hpp"],
    "fc1": ["dv_mlp.hip", "dv_rowdot.hpp", "dv_internal.hpp"],
    "b32:qkv": ["dv_batch.hip", "dv_internal.hpp"],
    "b32:attn": ["dv_attn.hip", "dv_rowdot.hpp", "dv_internal.hpp", "dv_select.hpp"],
    "b32:oproj": ["dv_batch.hip", "dv_internal.hpp"],
    "b32:fc1": ["dv_batch.hip", "dv_internal.hpp"],
    "b32:fc2": ["dv_batch.hip", "dv_internal.hpp"],
}


def kernel_sources_digest(label):
    import hashlib
    h = hashlib.sha256()
    files = [os.path.join(_CSRC, f) for f in KERNEL_SOURCES[label]]
    files.append(os.path.join(ROOT, "paper_2310_17157_amd", "build.py"))
    for f in files:
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode() + b"\0" + fh.read())
    return h.hexdigest()


def counter_traffic(workload, label):
    """HBM bytes per launch of `label` from the committed rocprofv3 FETCH_SIZE/WRITE_SIZE
    summary, or None if there is none or the kernel's sources changed since."""
    kind = "sparse_attn_mlp" if workload.endswith("_b32") else "sparse_block"
    p = os.path.join(ROOT, "profiles", f"{kind}_{workload}_hbm_counters.txt")
    try:
        with open(p) as fh:
            line = next(l for l in fh if l.startswith("json: "))
        rec = json.loads(line[len("json: "):])
        key = f"b32:{label}" if workload.endswith("_b32") else label
        if rec["sources_sha256"].get(label) != kernel_sources_digest(key):
            return None
        return rec["traffic_bytes"].get(label)
    except (OSError, StopIteration, ValueError, KeyError):
        return None


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        return 1


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_sparse_step(O, cfg, h, pos):
    """One token through the oracle: both predictors, top-k and the sparse layer."""
    import numpy as np
    lno = dict(g1=h["g1"], be1=h["be1"], g2=h["g2"], be2=h["be2"], eps=1e-5)
    attn = {k: h[k] for k in ("Wq", "Wk", "Wv", "WoT", "bq", "bk", "bv", "bo")}
    mlp = {k: h[k] for k in ("W1T", "W2T", "b1", "b2")}
    return O.sparse_block(h["x"][0], attn, mlp, h["K"][0], h["V"][0], pos, 1.0 / np.sqrt(cfg.dh),
                          pred_h=dict(AT=h["AT_h"], BT=h["BT_h"]), pred_m=dict(AT=h["AT_m"], BT=h["BT_m"]),
                          k_heads=cfg.k_heads, k_mlp=cfg.k_mlp, ln=lno, mode="lookahead")


def _oracle_dense_step(O, cfg, h, pos):
    import numpy as np
    lno = dict(g1=h["g1"], be1=h["be1"], g2=h["g2"], be2=h["be2"], eps=1e-5)
    attn = {k: h[k] for k in ("Wq", "Wk", "Wv", "WoT", "bq", "bk", "bv", "bo")}
    mlp = {k: h[k] for k in ("W1T", "W2T", "b1", "b2")}
    return O.dense_block(h["x"][0], attn, mlp, h["K"][0], h["V"][0], pos, 1.0 / np.sqrt(cfg.dh), ln=lno)


def _timed(fn, runs):
    ts = []
    for _ in range(runs):
        t0 = time.perf_counter()
        fn()
        ts.append(time.perf_counter() - t0)
    return statistics.median(ts) * 1e6


def cpu_baseline(cfg, t_host, pos, small_configs=("opt125m_b1", "opt6.7b_b1", "opt66b_b1")):
    """The fp64 oracle on this host: the predict + sparse layer for one token of the
    benchmark's own workload (median of 3, all BLAS threads, and once on 1 thread), and
    the sparse and dense layers of the smaller OPT shapes (median of 3 / 1 run)."""
    from oracle import dejavu as O
    from synth import get_config, make_layer
    threads = _blas_threads()
    value = _timed(lambda: _oracle_sparse_step(O, cfg, t_host, pos), 3)
    one = None
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            one = round(_timed(lambda: _oracle_sparse_step(O, cfg, t_host, pos), 1), 1)
    except Exception:  # pragma: no cover
        pass
    by_cfg = {}
    for name in small_configs:
        c = get_config(name)
        h = _host_copy(make_layer(c, 0, device="cuda", biases=False, ln_random=False))
        p = c.L - 1
        by_cfg[name] = {"sparse_us": round(_timed(lambda: _oracle_sparse_step(O, c, h, p), 3), 1),
                        "dense_us": round(_timed(lambda: _oracle_dense_step(O, c, h, p), 1 if c.d > 4096 else 3), 1)}
        del h
    return {"value": value, "unit": "us/layer/token", "cores": threads, "kind": "oracle",
            "sample": f"the fp64 oracle's predict + sparse layer for one token of {cfg.name} (the same seeded "
                      f"layer as replica 0), median of 3 runs on {threads} BLAS threads; host cores visible: "
                      f"{len(os.sched_getaffinity(0))}",
            "cpu_model": _cpu_model(), "one_thread_us": one, "by_config": by_cfg}


class StepEvents:
    """Timing-only HIP events (no system fence) recorded around whole steps on a stream."""

    def __init__(self, n):
        import ctypes
        from ctypes import POINTER, c_float, c_void_p
        self._ct = ctypes
        self._hip = ctypes.CDLL("libamdhip64.so")
        self._hip.hipEventCreateWithFlags.argtypes = [POINTER(c_void_p), ctypes.c_uint]
        self._hip.hipEventRecord.argtypes = [c_void_p, c_void_p]
        self._hip.hipEventElapsedTime.argtypes = [POINTER(c_float), c_void_p, c_void_p]
        self._hip.hipEventSynchronize.argtypes = [c_void_p]
        self._hip.hipEventDestroy.argtypes = [c_void_p]
        self.ev = []
        for _ in range(2 * n):
            e = c_void_p()
            if self._hip.hipEventCreateWithFlags(ctypes.byref(e), 0x20000000) != 0:
                raise RuntimeError("hipEventCreateWithFlags failed")
            self.ev.append(e)

    def record(self, i, stream):
        self._hip.hipEventRecord(self.ev[i], stream.cuda_stream)

    def ms(self, i):
        a, b = self.ev[2 * i], self.ev[2 * i + 1]
        self._hip.hipEventSynchronize(b)
        out = self._ct.c_float(0.0)
        self._hip.hipEventElapsedTime(self._ct.byref(out), a, b)
        return out.value

    def close(self):
        for e in self.ev:
            self._hip.hipEventDestroy(e)


def step_spread(stream, step, n):
    """p10 / p50 / p90 of single steps, each bracketed by its own pair of timing-only
    events (the events leave the GPU idle for a few microseconds each, so this pass is
    reported beside the unbracketed window mean, not instead of it)."""
    import torch
    ev = StepEvents(n)
    torch.cuda.synchronize()
    for i in range(n):
        ev.record(2 * i, stream)
        step(i)
        ev.record(2 * i + 1, stream)
    torch.cuda.synchronize()
    v = sorted(ev.ms(i) * 1e3 for i in range(n))
    ev.close()
    q = lambda f: round(v[min(n - 1, int(f * (n - 1) + 0.5))], 2)
    return {"steps": n, "p10_us": q(0.1), "p50_us": q(0.5), "p90_us": q(0.9), "min_us": round(v[0], 2),
            "max_us": round(v[-1], 2)}


def stream_ceiling(nbytes_list, steps, replicas=4):
    """The plain streaming read (dv_stream_read) of each byte count, rotating over
    `replicas` buffers (beyond the 256 MB Infinity Cache); launch averages from events
    on the stream."""
    import torch
    from paper_2310_17157_amd import binding as Bd
    top = max(nbytes_list)
    bufs = [torch.empty(top, dtype=torch.uint8, device="cuda") for _ in range(replicas)]
    sink = torch.zeros(1, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    out = {}
    for nb in nbytes_list:
        nb16 = nb // 16 * 16

        def step(i, timers=None):
            if timers:
                timers[0].arm()
            Bd.dv_stream_read(bufs[i % replicas], sink, nb16, stream=stream)
            if timers:
                timers[0].disarm()

        for i in range(5):
            step(i)
        _, _, per = _measure(stream, step, steps, 1)
        us = statistics.mean(per["stream_read"]) * 1e3
        out[str(nb)] = {"bytes": nb16, "avg_launch_us": round(us, 2), "GBps": round(nb16 / us / 1e3, 1),
                        "frac": round(nb16 / us / 1e3 / PEAK_HBM_GBPS, 4)}
    del bufs
    torch.cuda.empty_cache()
    return out


def _measure(stream, step, n, calls_per_step, only=None, every=1, pairs=16):
    """Run n steps; per-call LaunchTimers (all launches, or only label `only`) on the
    steps i with i % every == 0. Returns (ms per step from events on `stream`, wall
    seconds, {label: [ms, ...]})."""
    import torch
    from paper_2310_17157_amd import binding as Bd
    timers = [[Bd.LaunchTimer(pairs, only=only) for _ in range(calls_per_step)] if i % every == 0 else None
              for i in range(n)]
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    w0 = time.perf_counter()
    ev0.record(stream)
    for i in range(n):
        step(i, timers[i])
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    per = {}
    for ts in timers:
        for tm in ts or ():
            for lab, ms in tm.times_ms():
                per.setdefault(lab, []).append(ms)
            tm.close()
    return ev0.elapsed_time(ev1) / n, wall, per


def _kernel_table(per_kernel, kb_of):
    """Per-label averages; kb_of(label) -> algorithmic bytes per launch (or None)."""
    kernels = {}
    for lab, v in per_kernel.items():
        avg = statistics.mean(v)
        k = {"avg_us": round(avg * 1e3, 2), "p50_us": round(statistics.median(v) * 1e3, 2), "launches": len(v)}
        nb = kb_of(lab)
        if nb is not None:
            k["bytes"] = nb
            k["GBps"] = round(nb / (avg * 1e-3) / 1e9, 1)
            k["frac"] = round(k["GBps"] / PEAK_HBM_GBPS, 4)
        kernels[lab] = k
    return kernels


def _host_copy(t, keys=None):
    import torch
    out = {}
    for k, v in t.items():
        if k == "pos" or (keys is not None and k not in keys):
            continue
        a = v.detach().cpu()
        out[k] = a.numpy() if a.dtype == torch.float16 else a.to(torch.float64).numpy()
    return out


BLOCK_KERNELS = ("qkv", "attn", "oproj", "fc1", "fc2")   # the sparse layer itself (not the predictors)
TARGET_FRAC = 0.70                                        # of peak HBM bandwidth, over the block's bytes


def bench_b1(args, cfg):
    import numpy as np
    import torch

    from paper_2310_17157_amd import binding as Bd
    from paper_2310_17157_amd import accounting
    from paper_2310_17157_amd.workload import layer_objects
    from synth import make_layer

    mode = Bd.DV_LOOKAHEAD if args.mode == "lookahead" else Bd.DV_SEQUENTIAL
    scale = 1.0 / float(np.sqrt(cfg.dh))
    print(f"[bench] generating {args.replicas} replica(s) of {cfg.name} on the GPU", file=sys.stderr, flush=True)
    layers = []
    for r in range(args.replicas):
        t = make_layer(cfg, seed=r, device="cuda", biases=False, ln_random=False)
        objs = layer_objects(t, cfg.H)
        ws = torch.empty(Bd.block_workspace_bytes(*objs[:4], objs[4], 1, cfg.k_heads, cfg.k_mlp),
                         dtype=torch.uint8, device="cuda")
        out = torch.empty_like(t["x"])
        hs = torch.empty((1, cfg.k_heads), dtype=torch.int32, device="cuda")
        ms = torch.empty((1, cfg.k_mlp), dtype=torch.int32, device="cuda")
        layers.append((t, objs, ws, out, hs, ms))
    torch.cuda.synchronize()
    pos = cfg.L - 1

    stream = torch.cuda.Stream()
    torch.cuda.set_stream(stream)

    def step(i, timers=None):
        t, (attn, mlp, ph, pm, kv, ln), ws, out, hs, ms = layers[i % len(layers)]
        if timers:
            timers[0].arm()
        Bd.dv_sparse_block(attn, mlp, ph, pm, ln, kv, t["x"], cfg.k_heads, cfg.k_mlp, scale, mode=mode,
                           out=out, heads_out=hs, idx_out=ms, ws=ws, stream=stream)
        if timers:
            timers[0].disarm()

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # Diagnostic pass: every launch timed with events (each timed launch leaves the
    # GPU idle for a few microseconds, so this pass is not the reported step time).
    ms_all_events, _, per_kernel = _measure(stream, step, args.steps, 1)
    kb = kernel_bytes(cfg, pos)
    dom = max((l for l in per_kernel if l in kb), key=lambda l: statistics.mean(per_kernel[l]))
    # Timed region: events on the dominant kernel's launch on every
    # ROOFLINE_EVERY-th step (each timed launch idles the GPU for a few microseconds).
    ms_per_step, wall, per_dom = _measure(stream, step, args.steps, 1, only=dom, every=ROOFLINE_EVERY)
    # Each block kernel timed the same way in a pass of its own (launch averages for
    # the block roofline).
    per_one = {dom: per_dom[dom]}
    for lab in BLOCK_KERNELS:
        if lab != dom and lab in per_kernel:
            per_one[lab] = _measure(stream, step, args.steps, 1, only=lab, every=4)[2][lab]
    kernels = _kernel_table(per_kernel, kb.get)
    for lab, v in per_one.items():
        kernels[lab]["avg_us_alone"] = round(statistics.mean(v) * 1e3, 2)
    dom_avg_s = statistics.mean(per_dom[dom]) * 1e-3
    achieved = kb[dom] / dom_avg_s / 1e9
    b = accounting.layer_bytes(cfg)
    spread = step_spread(stream, step, args.steps)

    # measured ceiling: a plain contiguous read of the block's bytes and of the step's bytes,
    # and of each block kernel's own bytes (what one launch of that size can do at best)
    torch.cuda.set_stream(torch.cuda.default_stream())
    sizes = [b.block, b.total, kb[dom]] + [kb[k] for k in BLOCK_KERNELS if k in kb]
    ceil = stream_ceiling(list(dict.fromkeys(sizes)), args.steps)
    torch.cuda.set_stream(stream)
    blk_us = sum(statistics.mean(per_one[k]) * 1e3 for k in BLOCK_KERNELS if k in per_one)
    blk_gbps = b.block / (blk_us * 1e-6) / 1e9
    floors_us = sum(ceil[str(kb[k])]["avg_launch_us"] for k in BLOCK_KERNELS if k in kb)
    block = {"kernels": list(BLOCK_KERNELS), "bytes": b.block, "us": round(blk_us, 2),
             "achieved": round(blk_gbps, 1), "frac": round(blk_gbps / PEAK_HBM_GBPS, 4),
             "target_frac": TARGET_FRAC, "met": bool(blk_gbps / PEAK_HBM_GBPS >= TARGET_FRAC),
             "stream_same_bytes_GBps": ceil[str(b.block)]["GBps"],
             "frac_vs_measured_stream": round(blk_gbps / ceil[str(b.block)]["GBps"], 4),
             # five plain reads, each of one block kernel's bytes: the best five launches can do
             "per_kernel_stream_floors_us": round(floors_us, 2),
             "per_kernel_floors_frac": round(b.block / (floors_us * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4),
             "us_over_per_kernel_floors": round(blk_us / floors_us, 4)}
    roofline = {"bound": "hbm", "kernel": dom, "scope": "dominant kernel", "achieved": round(achieved, 1),
                "peak": PEAK_HBM_GBPS, "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBPS, 4),
                "traffic": counter_traffic(cfg.name, dom),
                "bytes_per_launch": kb[dom], "avg_launch_us": round(dom_avg_s * 1e6, 2),
                "frac_vs_measured_stream": round(achieved / ceil[str(kb[dom])]["GBps"], 4),
                "block": block}
    step_gbps = b.total / (ms_per_step * 1e-3) / 1e9
    hbm = {"block_bytes": b.block, "predictor_bytes": b.pred, "total_bytes": b.total,
           "step_GBps": round(step_gbps, 1), "step_frac": round(step_gbps / PEAK_HBM_GBPS, 4),
           "step_frac_vs_measured_stream": round(step_gbps / ceil[str(b.total)]["GBps"], 4),
           "sparse_block_kernels_us": block["us"], "sparse_block_kernels_frac": block["frac"],
           "stream_ceiling": ceil}

    loop = lookahead_loop(args, cfg, layers, stream, scale, b.total)
    kvfill = kvfill_steps(cfg, layers[0][0], stream, scale)
    q4 = q4_mlp(args, cfg, layers, stream)

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the fp64 oracle on the host", file=sys.stderr, flush=True)
        cpu = cpu_baseline(cfg, _host_copy(layers[0][0]), pos)
    del layers
    torch.cuda.synchronize()
    torch.cuda.empty_cache()

    return {
        "metric": METRIC, "value": round(ms_per_step * 1e3, 2), "unit": "us/layer/token", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "f16 weights, f32 accumulate",
        "data": "synthetic",
        "config": {"workload": cfg.name, "d_model": cfg.d, "ffn": cfg.N, "heads": cfg.H, "head_dim": cfg.dh,
                   "kv_len": cfg.L, "rank": cfg.r, "k_mlp": cfg.k_mlp, "k_heads": cfg.k_heads, "batch": 1,
                   "weights": cfg.wdtype, "kv": cfg.kvdtype, "mode": args.mode, "replicas": args.replicas,
                   "parallelism": "none (1 GPU)"},
        "roofline": roofline, "cpu_baseline": cpu, "hbm": hbm, "step_spread": spread, "lookahead_loop": loop,
        "kvfill": kvfill, "w4a16_mlp": q4, "kernels": kernels,
        "wall_s_timed": round(wall, 4), "ms_per_step_all_launch_events": round(ms_all_events, 5),
    }


def lookahead_loop(args, cfg, layers, stream, scale, layer_bytes):
    """The replicas as consecutive layers of one token (dv_sparse_decode): the sets of
    layer l+1 predicted from layer l's input inside layer l's launches (Section 4.3),
    per layer and token, beside the single-layer calls timed above."""
    import torch
    from paper_2310_17157_amd import binding as Bd
    objs = [L[1] for L in layers]
    n = len(objs)
    arr = Bd._layers_c(objs)
    x = layers[0][0]["x"]
    ws = torch.empty(Bd.decode_workspace_bytes(objs, cfg.k_heads, cfg.k_mlp), dtype=torch.uint8, device="cuda")
    out = torch.empty_like(x)
    hs = torch.empty((n, cfg.k_heads), dtype=torch.int32, device="cuda")
    ms = torch.empty((n, cfg.k_mlp), dtype=torch.int32, device="cuda")

    def step(i, timers=None):
        if timers:
            timers[0].arm()
        Bd.dv_sparse_decode(objs, x, cfg.k_heads, cfg.k_mlp, scale, out=out, heads_out=hs, idx_out=ms, ws=ws,
                            stream=stream, _arr=arr)
        if timers:
            timers[0].disarm()

    for i in range(args.warmup):
        step(i)
    ms_call, _, _ = _measure(stream, step, args.steps, 1, every=10 ** 9)
    _, _, per = _measure(stream, step, max(4, args.steps // 4), 1, pairs=64)
    us = ms_call * 1e3 / n
    gbps = layer_bytes / (us * 1e-6) / 1e9
    return {"layers_per_call": n, "calls": args.steps, "us_per_layer_token": round(us, 2),
            "GBps": round(gbps, 1), "frac": round(gbps / PEAK_HBM_GBPS, 4),
            "launch_avg_us": {k: round(statistics.mean(v) * 1e3, 2) for k, v in per.items()}}


PAPER_KERNEL_CLAIMS = ("context, not a target (A100, Triton, 8-way tensor parallel): the fused sparse MLP up to "
                       "4.5x and sparse attention up to 5x faster than index-then-multiply in PyTorch, both faster "
                       "than dense up to density 0.8 (Appendix E); the unfused gather moves 3x the bytes (Section 4.4)")


def density_sweep(args, cfg, densities=(0.05, 0.1, 0.2, 0.3, 0.4, 0.5, 0.6, 0.7, 0.8, 0.9, 1.0), reps=20):
    """Appendix E's kernel benchmark on this GPU: the sparse MLP and the sparse attention
    at a range of densities, three ways each: the fused gathered kernels of this library
    (dv_sparse_mlp, dv_sparse_attn), the dense layer with torch's library GEMVs, and the
    unfused form (index_select of the selected rows into a new tensor, then the same
    GEMVs on it). Weights are cycled over replicas beyond the 256 MB last-level cache;
    each point is the median of `reps` calls timed with events on the stream."""
    import numpy as np
    import torch
    import torch.nn.functional as F
    from paper_2310_17157_amd import binding as Bd
    from synth import make_layer

    R = 2
    reps_ = [make_layer(cfg, seed=r, device="cuda", with_predictors=False) for r in range(R)]
    scale = 1.0 / float(np.sqrt(cfg.dh))
    d, N, H, dh = cfg.d, cfg.N, cfg.H, cfg.dh
    x = reps_[0]["x"]
    x16 = x.half()
    stream = torch.cuda.current_stream()

    def med_us(fn):
        for i in range(3):
            fn(i)
        ts = []
        for i in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn(i)
            b.record(stream)
            b.synchronize()
            ts.append(a.elapsed_time(b) * 1e3)
        return round(statistics.median(ts), 2)

    rng = np.random.default_rng(5)
    mlp_objs = [Bd.MLP(t["W1T"], t["W2T"], t["b1"], t["b2"]) for t in reps_]
    attn_objs = [Bd.Attn(t["Wq"], t["Wk"], t["Wv"], t["WoT"], H, t["bq"], t["bk"], t["bv"], t["bo"]) for t in reps_]
    kvs = [Bd.KVCache(t["K"], t["V"], [cfg.L - 1]) for t in reps_]
    pos = cfg.L - 1

    def dense_mlp(i):
        t = reps_[i % R]
        h = torch.relu(F.linear(x16, t["W1T"], t["b1"].half()))
        return torch.matmul(h, t["W2T"]) + t["b2"]

    def dense_attn(i):
        t = reps_[i % R]
        q, k, v = (F.linear(x16, t[w], t[b].half()).view(H, 1, dh) for w, b in (("Wq", "bq"), ("Wk", "bk"),
                                                                                   ("Wv", "bv")))
        Kc, Vc = t["K"][0], t["V"][0]
        Kc[:, pos] = k[:, 0]
        Vc[:, pos] = v[:, 0]
        sc = torch.matmul(Kc[:, :pos + 1], q.transpose(1, 2).contiguous()).float() * scale      # [H, L, 1]
        p = torch.softmax(sc, dim=1).half()
        o = torch.matmul(p.transpose(1, 2).contiguous(), Vc[:, :pos + 1])                       # [H, 1, dh]
        return torch.matmul(o.reshape(1, H * dh), t["WoT"]) + t["bo"]

    t_dense_mlp = med_us(dense_mlp)
    t_dense_attn = med_us(dense_attn)
    mlp_bytes_dense = 2 * N * d * cfg.wbytes
    attn_bytes_dense = 4 * H * dh * d * cfg.wbytes + 2 * H * (pos + 1) * dh * cfg.kvbytes
    out = {"mlp": [], "attn": []}
    for p in densities:
        k = max(1, int(round(p * N)))
        S = [torch.tensor(np.sort(rng.choice(N, k, replace=False)).astype(np.int32), device="cuda") for _ in range(R)]
        o_m = torch.empty_like(x)
        ws_m = torch.empty(Bd.mlp_workspace_bytes(mlp_objs[0], 1, k), dtype=torch.uint8, device="cuda")
        fused = med_us(lambda i: Bd.dv_sparse_mlp(mlp_objs[i % R], x, S[i % R], out=o_m, ws=ws_m))

        def unfused_mlp(i):
            t, idx = reps_[i % R], S[i % R].long()
            W1s = t["W1T"].index_select(0, idx)
            W2s = t["W2T"].index_select(0, idx)
            h = torch.relu(F.linear(x16, W1s, t["b1"].half().index_select(0, idx)))
            return torch.matmul(h, W2s) + t["b2"]

        unfused = med_us(unfused_mlp)
        b = 2 * k * d * cfg.wbytes
        out["mlp"].append({"density": p, "k": k, "fused_us": fused, "unfused_us": unfused, "dense_us": t_dense_mlp,
                           "fused_GBps": round(b / fused / 1e3, 1),
                           "unfused_over_fused": round(unfused / fused, 2), "dense_over_fused": round(t_dense_mlp / fused, 2)})
        kh = max(1, int(round(p * H)))
        Hs = [torch.tensor(np.sort(rng.choice(H, kh, replace=False)).astype(np.int32), device="cuda").view(1, -1)
              for _ in range(R)]
        o_a = torch.empty_like(x)
        ws_a = torch.empty(Bd.attn_workspace_bytes(attn_objs[0], kvs[0], 1, kh), dtype=torch.uint8, device="cuda")
        fused_a = med_us(lambda i: Bd.dv_sparse_attn(attn_objs[i % R], x, kvs[i % R], Hs[i % R], scale, out=o_a,
                                                     ws=ws_a))

        def unfused_attn(i):
            t, hs = reps_[i % R], Hs[i % R].view(-1).long()
            rows = (hs[:, None] * dh + torch.arange(dh, device="cuda")[None, :]).reshape(-1)
            q, k_, v = (F.linear(x16, t[w].index_select(0, rows), t[b].half().index_select(0, rows)).view(kh, 1, dh)
                        for w, b in (("Wq", "bq"), ("Wk", "bk"), ("Wv", "bv")))
            t["K"][0][hs, pos] = k_[:, 0]
            t["V"][0][hs, pos] = v[:, 0]
            Kc = t["K"][0].index_select(0, hs)
            Vc = t["V"][0].index_select(0, hs)
            sc = torch.matmul(Kc[:, :pos + 1], q.transpose(1, 2).contiguous()).float() * scale
            pr = torch.softmax(sc, dim=1).half()
            o = torch.matmul(pr.transpose(1, 2).contiguous(), Vc[:, :pos + 1])
            return torch.matmul(o.reshape(1, kh * dh), t["WoT"].index_select(0, rows)) + t["bo"]

        unfused_a = med_us(unfused_attn)
        ba = 4 * kh * dh * d * cfg.wbytes + 2 * kh * (pos + 1) * dh * cfg.kvbytes
        out["attn"].append({"density": round(kh / H, 4), "k_heads": kh, "fused_us": fused_a, "unfused_us": unfused_a,
                            "dense_us": t_dense_attn, "fused_GBps": round(ba / fused_a / 1e3, 1),
                            "unfused_over_fused": round(unfused_a / fused_a, 2),
                            "dense_over_fused": round(t_dense_attn / fused_a, 2)})
    cross = {}
    for part in ("mlp", "attn"):
        faster = [r["density"] for r in out[part] if r["fused_us"] < r["dense_us"]]
        cross[part] = {"fused_faster_than_dense_up_to_density": max(faster) if faster else None,
                       "max_unfused_over_fused": max(r["unfused_over_fused"] for r in out[part])}
    return {"sweep": "density", "workload": cfg.name, "reps": reps, "replicas": R,
            "dense_mlp_us": t_dense_mlp, "dense_mlp_GBps": round(mlp_bytes_dense / t_dense_mlp / 1e3, 1),
            "dense_attn_us": t_dense_attn, "dense_attn_GBps": round(attn_bytes_dense / t_dense_attn / 1e3, 1),
            "summary": cross, "paper": PAPER_KERNEL_CLAIMS, **out}


def q4_mlp(args, cfg, layers, stream):
    """Section 5.2's W4A16 setting: the sparse MLP of each replica with its W1T and W2T
    rows stored as 4-bit codes in blocks of 32 with an fp16 scale (dv_sparse_mlp_q4,
    same neuron sets as the block's), per call and per launch, against the fp16 rows."""
    import torch
    from paper_2310_17157_amd import binding as Bd
    from synth import quantize_q4
    objs = []
    for t, *_ in layers:
        P1, S1 = quantize_q4(t["W1T"])
        P2, S2 = quantize_q4(t["W2T"])
        objs.append(Bd.MLPQ4(P1, S1, P2, S2, t["b1"], t["b2"]))
    sets = [L[5].view(-1) for L in layers]          # each replica's neuron set from the timed steps
    x = layers[0][0]["x"]
    out = torch.empty_like(x)
    ws = torch.empty(Bd.load().dv_sparse_mlp_q4_workspace_bytes(__import__("ctypes").byref(objs[0].c()), cfg.k_mlp),
                     dtype=torch.uint8, device="cuda")
    n = len(objs)

    def step(i, timers=None):
        if timers:
            timers[0].arm()
        Bd.dv_sparse_mlp_q4(objs[i % n], x, sets[i % n], out=out, ws=ws, stream=stream)
        if timers:
            timers[0].disarm()

    for i in range(args.warmup):
        step(i)
    ms_call, _, _ = _measure(stream, step, args.steps, 1, every=10 ** 9)
    _, _, per = _measure(stream, step, args.steps, 1)
    row = cfg.d // 2 + cfg.d // 16
    nb = 2 * cfg.k_mlp * row
    us = {k: statistics.mean(v) * 1e3 for k, v in per.items()}
    return {"bytes": nb, "fp16_bytes": 2 * cfg.k_mlp * cfg.d * cfg.wbytes, "us_per_call": round(ms_call * 1e3, 2),
            "launch_avg_us": {k: round(v, 2) for k, v in us.items()},
            "GBps_launches": round(nb / (sum(us.values()) * 1e-6) / 1e9, 1),
            "frac_launches": round(nb / (sum(us.values()) * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4)}


def kvfill_steps(cfg, t, stream, scale, T=32):
    """Section 4.2's missing-KV rule over T consecutive tokens with independent uniform
    head sets (k_heads of H per token): dv_sparse_attn_kvfill per token against
    dv_sparse_attn on the same sets (which leaves the missing rows missing), and the
    fill launch alone; missing rows filled per token, counted on the host."""
    import numpy as np
    import torch
    from paper_2310_17157_amd import binding as Bd
    H, cap, d = cfg.H, cfg.kv_cap, cfg.d
    attn = Bd.Attn(t["Wq"], t["Wk"], t["Wv"], t["WoT"], H)
    p0 = cap - T
    kv = Bd.KVCache(t["K"], t["V"], [p0])
    Y = torch.randn((cap, d), device="cuda").to(t["K"].dtype)   # kept inputs, in the cache's type
    valid = torch.zeros((H, cap), dtype=torch.uint8, device="cuda")
    valid[:, :p0] = 1
    rng = np.random.default_rng(17)
    sets = [torch.tensor(np.sort(rng.choice(H, cfg.k_heads, replace=False)).astype(np.int32), device="cuda")
            for _ in range(T)]
    last = np.full(H, p0 - 1)
    filled = []
    for s_ in range(T):
        S = sets[s_].cpu().numpy()
        filled.append(int(sum(p0 + s_ - 1 - last[h] for h in S)))
        last[S] = p0 + s_
    ws = torch.empty(Bd.attn_workspace_bytes(attn, kv, 1, cfg.k_heads), dtype=torch.uint8, device="cuda")
    out = torch.empty((1, d), dtype=torch.float32, device="cuda")
    x = torch.randn((1, d), device="cuda")
    res = {}
    # the per-token times come from passes without launch events (each timed launch
    # leaves the GPU idle for a few microseconds); a third pass times the fill's launches
    for key in ("kvfill", "plain", "launches"):
        valid[:, p0:] = 0
        valid[:, :p0] = 1
        tm = [Bd.LaunchTimer(8) for _ in range(T)] if key == "launches" else None
        torch.cuda.synchronize()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record(stream)
        for s_ in range(T):
            kv.set_pos([p0 + s_])
            if key == "plain":
                Bd.dv_sparse_attn(attn, x, kv, sets[s_].view(1, -1), scale, out=out, ws=ws, stream=stream)
                continue
            if tm:
                tm[s_].arm()
            Bd.dv_sparse_attn_kvfill(attn, x, kv, Y, valid, sets[s_], scale, out=out, ws=ws, stream=stream)
            if tm:
                tm[s_].disarm()
        ev1.record(stream)
        torch.cuda.synchronize()
        res[key] = ev0.elapsed_time(ev1) * 1e3 / T
        if tm:
            per = collections.defaultdict(list)
            for tmr in tm:
                for lab, ms in tmr.times_ms():
                    per[lab].append(ms * 1e3)
                tmr.close()
            res["fill_launch_us"] = round(statistics.mean(per["kv_fill"]), 2)
            res["qkv_launch_us"] = round(statistics.mean(per["qkv"]), 2)
    kv.set_pos([cap - 1])
    return {"tokens": T, "k_heads": cfg.k_heads, "heads": H, "missing_rows_filled_per_token": round(statistics.mean(
            filled[1:]), 2), "us_per_token_kvfill": round(res["kvfill"], 2),
            "us_per_token_without_fill": round(res["plain"], 2), "fill_launch_us": res["fill_launch_us"],
            "qkv_launch_us": res["qkv_launch_us"]}


def cpu_baseline_b32(cfg, th, heads, sets, pos):
    """The fp64 oracle's attention (own heads and cache) + union MLP for one sequence."""
    import numpy as np
    from oracle import dejavu as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    U = O.union_of_sets([list(s) for s in sets])
    attn = {k: th[k] for k in ("Wq", "Wk", "Wv", "WoT")}
    t0 = time.perf_counter()
    a_out, _, _, _ = O.mha_sparse(th["x"][0], attn, th["K0"], th["V0"], int(pos[0]), heads[0], 1.0 / np.sqrt(cfg.dh))
    O.mlp_sparse(a_out, th["W1T"], None, th["W2T"], None, U)
    dt = time.perf_counter() - t0
    return {"value": dt * 1e6, "unit": "us/layer/token", "cores": threads, "kind": "oracle",
            "sample": f"one sequence (b = 0, kv length {int(pos[0]) + 1}) of {cfg.name}: its sparse attention "
                      f"over 32 heads and the MLP over the union of the batch's sets (|U| = {len(U)}); "
                      f"host cores visible: {len(os.sched_getaffinity(0))}"}


def bench_batch(args, cfg):
    import numpy as np
    import torch

    from paper_2310_17157_amd import binding as Bd
    from synth import make_layer, uniform_head_sets, zipf_mlp_sets

    B = cfg.B
    scale = 1.0 / float(np.sqrt(cfg.dh))
    print(f"[bench] generating {args.replicas} replica(s) of {cfg.name} on the GPU", file=sys.stderr, flush=True)
    layers = []
    for r in range(args.replicas):
        t = make_layer(cfg, seed=r, device="cuda", biases=False, with_predictors=False)
        heads = uniform_head_sets(cfg, r)
        sets = zipf_mlp_sets(cfg, r)
        pos = [int(p) for p in t["pos"]]
        attn = Bd.Attn(t["Wq"], t["Wk"], t["Wv"], t["WoT"], cfg.H)
        mlp = Bd.MLP(t["W1T"], t["W2T"])
        kv = Bd.KVCache(t["K"], t["V"], pos)
        ht = torch.tensor(heads, dtype=torch.int32, device="cuda")
        st = torch.tensor(sets, dtype=torch.int32, device="cuda")
        ws_a = torch.empty(Bd.attn_workspace_bytes(attn, kv, B, cfg.k_heads), dtype=torch.uint8, device="cuda")
        ws_m = torch.empty(Bd.mlp_workspace_bytes(mlp, B, cfg.k_mlp, 1), dtype=torch.uint8, device="cuda")
        a_out = torch.empty_like(t["x"])
        m_out = torch.empty_like(t["x"])
        kb, nu, nu_h = batch_kernel_bytes(cfg, heads, sets, pos)
        layers.append(dict(t=t, attn=attn, mlp=mlp, kv=kv, ht=ht, st=st, ws_a=ws_a, ws_m=ws_m, a_out=a_out,
                           m_out=m_out, kb=kb, nu=nu, nu_h=nu_h, heads=heads, sets=sets, pos=pos))
    torch.cuda.synchronize()
    stream = torch.cuda.Stream()
    torch.cuda.set_stream(stream)

    def step(i, timers=None):
        L = layers[i % len(layers)]
        if timers:
            timers[0].arm()
        Bd.dv_sparse_attn(L["attn"], L["t"]["x"], L["kv"], L["ht"], scale, out=L["a_out"], ws=L["ws_a"],
                          stream=stream)
        if timers:
            timers[0].disarm()
            timers[1].arm()
        Bd.dv_sparse_mlp(L["mlp"], L["a_out"], L["st"], idx_per_seq=1, batch_mode=Bd.DV_MLP_UNION,
                         out=L["m_out"], ws=L["ws_m"], stream=stream)
        if timers:
            timers[1].disarm()

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    ms_all_events, _, per_kernel = _measure(stream, step, args.steps, 2)
    # bytes per launch averaged over the replicas the steps cycled through
    kb = {lab: statistics.mean(L["kb"][lab] for L in layers) for lab in layers[0]["kb"]}
    dom = max((l for l in per_kernel if l in kb), key=lambda l: statistics.mean(per_kernel[l]))
    ms_per_step, wall, per_dom = _measure(stream, step, args.steps, 2, only=dom, every=ROOFLINE_EVERY)
    kernels = _kernel_table(per_kernel, lambda l: round(kb[l]) if l in kb else None)
    dom_avg_s = statistics.mean(per_dom[dom]) * 1e-3
    achieved = kb[dom] / dom_avg_s / 1e9
    step_bytes = sum(kb.values())
    roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBPS, 4),
                "traffic": counter_traffic(cfg.name, dom),
                "bytes_per_launch": round(kb[dom]), "avg_launch_us": round(dom_avg_s * 1e6, 2)}
    hbm = {"step_bytes": round(step_bytes), "step_GBps": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 1),
           "step_frac": round(step_bytes / (ms_per_step * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
           "union_neurons": [L["nu"] for L in layers], "union_heads": [L["nu_h"] for L in layers]}
    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the fp64 oracle on the host", file=sys.stderr, flush=True)
        L = layers[0]
        th = _host_copy(L["t"], keys=("x", "Wq", "Wk", "Wv", "WoT", "W1T", "W2T"))
        th["K0"] = L["t"]["K"][0].cpu().numpy()
        th["V0"] = L["t"]["V"][0].cpu().numpy()
        cpu = cpu_baseline_b32(cfg, th, L["heads"], L["sets"], L["pos"])
    return {
        "metric": METRIC_B32, "value": round(ms_per_step * 1e3 / B, 3), "unit": "us/layer/token", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "f16 MFMA, f32 accumulate",
        "data": "synthetic",
        "config": {"workload": cfg.name, "d_model": cfg.d, "ffn": cfg.N, "heads": cfg.H, "head_dim": cfg.dh,
                   "kv_len": f"U[{cfg.L_range[0]},{cfg.L_range[1]}] per sequence", "k_mlp": cfg.k_mlp,
                   "k_heads": cfg.k_heads, "batch": B, "zipf_s": cfg.zipf_s, "weights": cfg.wdtype,
                   "kv": cfg.kvdtype, "mlp": "union", "replicas": args.replicas,
                   "parallelism": "none (1 GPU)"},
        "roofline": roofline, "cpu_baseline": cpu, "hbm": hbm, "kernels": kernels,
        "wall_s_timed": round(wall, 4), "ms_per_step_all_launch_events": round(ms_all_events, 5),
    }


def default_replicas(cfg):
    """Layer copies the steps cycle through: enough that what one step reads is not still
    in the 256 MB Infinity Cache when the same copy comes round again. At batch 1 the
    selected keys and values of a copy (33.5 MB at the OPT-175B shape) would otherwise
    stay in the cache across calls: 10 copies hold 335 MB of them (with 4, the attention
    launch measured 8.4 us against 9.5 us)."""
    return 10 if cfg.B == 1 else 4


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="opt175b_b1")
    ap.add_argument("--replicas", type=int, default=None,
                    help="independent layer copies cycled by the steps (default 10 at batch 1, 4 at batch 32)")
    ap.add_argument("--mode", choices=["lookahead", "sequential"], default="lookahead")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sweep", choices=["density"], default=None,
                    help="instead of the step: the sparse MLP and attention at densities 0.05-1.0, fused vs dense "
                         "vs index-then-multiply (Appendix E)")
    ap.add_argument("--no-b32", dest="b32", action="store_false",
                    help="skip the batch-32 sub-record of the default batch-1 run")
    ap.add_argument("--copy-calib-gib", type=float, default=0.0,
                    help="only run a plain device-to-device copy of this many GiB (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build runs on one GPU only (the single-GPU share of the layer); "
              "--gpus must be 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from synth import get_config

    torch.cuda.set_device(0)
    if args.copy_calib_gib > 0:
        n = int(args.copy_calib_gib * 2 ** 30)
        a = torch.empty(n, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n, "launches": 3}))
        return

    cfg = get_config(args.workload)
    explicit_replicas = args.replicas is not None
    if not explicit_replicas:
        args.replicas = default_replicas(cfg)
    if args.sweep == "density":
        print(json.dumps(density_sweep(args, cfg)))
        return
    rec = bench_b1(args, cfg) if cfg.B == 1 else bench_batch(args, cfg)
    if cfg.B == 1 and args.b32 and cfg.name == "opt175b_b1":
        # the batch-32 workload of the same layer shape, as a sub-record of the line
        print("[bench] batch-32 sub-record", file=sys.stderr, flush=True)
        a32 = argparse.Namespace(**vars(args))
        a32.no_cpu_baseline = True
        c32 = get_config("opt175b_b32")
        if not explicit_replicas:
            a32.replicas = default_replicas(c32)
        r32 = bench_batch(a32, c32)
        rec["b32"] = {k: r32[k] for k in ("metric", "value", "unit", "ms_per_step", "dtype", "config", "roofline",
                                          "hbm", "kernels")}
    print(json.dumps(rec))


if __name__ == "__main__":
    main()
