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
replicas (default 4) are cycled so that no weight is served from the 256 MB Infinity
Cache. Prints ONE JSON line: the value, the roofline of the dominant kernel from HIP
events recorded around each of its launches on the library's stream, and the fp64
oracle timed on this host's cores on a bounded sample.
"""
import argparse
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
ROOFLINE_EVERY = 8   # timed steps per event-bracketed launch of the dominant kernel


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


def cpu_baseline(cfg, t_host, pos, seconds=10.0):
    """The fp64 oracle's predict + sparse block for one token of this workload."""
    import numpy as np
    from oracle import dejavu as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    h = t_host
    lno = dict(g1=h["g1"], be1=h["be1"], g2=h["g2"], be2=h["be2"], eps=1e-5)
    attn = {k: h[k] for k in ("Wq", "Wk", "Wv", "WoT", "bq", "bk", "bv", "bo")}
    mlp = {k: h[k] for k in ("W1T", "W2T", "b1", "b2")}
    runs = []
    t_end = time.perf_counter() + seconds
    while True:
        t0 = time.perf_counter()
        O.sparse_block(h["x"][0], attn, mlp, h["K"][0], h["V"][0], pos, 1.0 / np.sqrt(cfg.dh),
                       pred_h=dict(AT=h["AT_h"], BT=h["BT_h"]), pred_m=dict(AT=h["AT_m"], BT=h["BT_m"]),
                       k_heads=cfg.k_heads, k_mlp=cfg.k_mlp, ln=lno, mode="lookahead")
        runs.append(time.perf_counter() - t0)
        if time.perf_counter() > t_end or len(runs) >= 3:
            break
    med = statistics.median(runs)
    return {"value": med * 1e6, "unit": "us/layer/token", "cores": threads, "kind": "oracle",
            "sample": f"{len(runs)} run(s) of the full predict + sparse block for one token of "
                      f"{cfg.name} (same seeded layer), median; host cores visible: "
                      f"{len(os.sched_getaffinity(0))}"}


def _measure(stream, step, n, calls_per_step, only=None, every=1):
    """Run n steps; per-call LaunchTimers (all launches, or only label `only`) on the
    steps i with i % every == 0. Returns (ms per step from events on `stream`, wall
    seconds, {label: [ms, ...]})."""
    import torch
    from paper_2310_17157_amd import binding as Bd
    timers = [[Bd.LaunchTimer(16, only=only) for _ in range(calls_per_step)] if i % every == 0 else None
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

    # Diagnostic pass: every launch bracketed by events (the events themselves add
    # a few microseconds per launch, so this pass is not the reported step time).
    ms_all_events, _, per_kernel = _measure(stream, step, args.steps, 1)
    kb = kernel_bytes(cfg, pos)
    dom = max((l for l in per_kernel if l in kb), key=lambda l: statistics.mean(per_kernel[l]))
    # Timed region: events around the dominant kernel's launch on every
    # ROOFLINE_EVERY-th step (each event record idles the GPU for a few microseconds).
    ms_per_step, wall, per_dom = _measure(stream, step, args.steps, 1, only=dom, every=ROOFLINE_EVERY)
    kernels = _kernel_table(per_kernel, kb.get)
    dom_avg_s = statistics.mean(per_dom[dom]) * 1e-3
    achieved = kb[dom] / dom_avg_s / 1e9
    b = accounting.layer_bytes(cfg)
    roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBPS, 4),
                "traffic": counter_traffic(cfg.name, dom),
                "bytes_per_launch": kb[dom], "avg_launch_us": round(dom_avg_s * 1e6, 2)}
    blk_us = round(sum(kernels[k]["avg_us"] for k in ("qkv", "attn", "oproj", "fc1", "fc2") if k in kernels), 2)
    hbm = {"block_bytes": b.block, "predictor_bytes": b.pred, "total_bytes": b.total,
           "step_GBps": round(b.total / (ms_per_step * 1e-3) / 1e9, 1),
           "step_frac": round(b.total / (ms_per_step * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4),
           "sparse_block_kernels_us": blk_us,
           "sparse_block_kernels_frac": round(b.block / (blk_us * 1e-6) / 1e9 / PEAK_HBM_GBPS, 4) if blk_us else None}

    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the fp64 oracle on the host", file=sys.stderr, flush=True)
        cpu = cpu_baseline(cfg, _host_copy(layers[0][0]), pos)

    return {
        "metric": METRIC, "value": round(ms_per_step * 1e3, 2), "unit": "us/layer/token", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": cfg.name, "d_model": cfg.d, "ffn": cfg.N, "heads": cfg.H, "head_dim": cfg.dh,
                   "kv_len": cfg.L, "rank": cfg.r, "k_mlp": cfg.k_mlp, "k_heads": cfg.k_heads, "batch": 1,
                   "weights": cfg.wdtype, "kv": cfg.kvdtype, "mode": args.mode, "replicas": args.replicas,
                   "parallelism": "none (1 GPU)"},
        "roofline": roofline, "cpu_baseline": cpu, "hbm": hbm, "kernels": kernels,
        "wall_s_timed": round(wall, 4), "ms_per_step_all_launch_events": round(ms_all_events, 5),
    }


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


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="opt175b_b1")
    ap.add_argument("--replicas", type=int, default=4)
    ap.add_argument("--mode", choices=["lookahead", "sequential"], default="lookahead")
    ap.add_argument("--no-cpu-baseline", action="store_true")
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
    rec = bench_b1(args, cfg) if cfg.B == 1 else bench_batch(args, cfg)
    print(json.dumps(rec))


if __name__ == "__main__":
    main()
