#!/usr/bin/env python3
"""Benchmark of the fused SeKV decode step on one MI355X.

Workload: one attention layer of a Llama-3-8B-shaped model (32 query heads over 8 KV
heads, head_dim 128) at 131,072 tokens of context, batch 4, rank-32 span factors,
top-16 spans per KV head, bfloat16 storage, all factors device-resident.  A step is one
call of sekv_decode_step (routing, selection, zoom-in, mixed-resolution attention).

Inputs are synthetic and already resident in HBM when the timed region starts.  Steps
rotate over several copies of the cache so that the 256 MB Infinity Cache cannot serve
a step from the previous use of the same data (each step reads ~66 MB).  The timed
steps are replayed from a HIP graph with one decode-step node per cache copy, so the
host's launch cost stays out of the device's way; the same steps launched one by one on
the stream are timed afterwards for context.

Prints ONE JSON line on stdout; progress goes to stderr.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "decode-step latency (µs) and achieved HBM GB/s, 128K context, batch 4"
HBM_PEAK_GBS = 8000.0
FP32_PEAK_TFLOPS = 157.3          # MI355X dense fp32 vector
KERNEL_NAME = "sekv_step_kernel"
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2606_31145_amd", "csrc", f) for f in
                  ("sekv_internal.h", "sekv_step.h", "sekv_step_inst.hip", "sekv_kernels.hip")]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    """Hash of the kernel sources' code: comments and blank space removed, so that an
    edit to comments alone does not orphan the committed counter figures."""
    import re
    src = ""
    for path in KERNEL_SOURCES:
        with open(path) as f:
            src += f.read() + "\n"
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    src = " ".join(src.split())
    return hashlib.sha256(src.encode()).hexdigest()[:16]


def load_traffic(workload: str):
    """HBM traffic per launch from a committed rocprofv3 counter summary, if it was taken
    on the current kernel source; otherwise None."""
    path = os.path.join(ROOT, "profiles", "sekv_step_kernel_counters.json")
    if not os.path.exists(path):
        return None
    try:
        with open(path) as f:
            rec = json.load(f)
    except Exception:
        return None
    entry = rec.get(workload)
    if not entry or entry.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    return entry.get("hbm_bytes_per_launch")


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--variant", choices=["L", "N"], default="L",
                    help="L: literal synthetic values; N: planted needle spans")
    ap.add_argument("--rotate", type=int, default=8, help="cache copies cycled through")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-other-variant", action="store_true",
                    help="headline workload: skip timing the other value variant (planted "
                         "needles when --variant L)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="approximate CPU time spent timing the oracle")
    ap.add_argument("--no-adaptive", action="store_true",
                    help="skip the per-span adaptive-rank timing of the same layer")
    ap.add_argument("--no-gated", action="store_true",
                    help="skip the learned-routing (gated) step timing")
    ap.add_argument("--gated-budget", type=int, default=4096,
                    help="expanded-token budget per (sequence, KV head) of the gated step")
    ap.add_argument("--calibration-copy-mib", type=int, default=0,
                    help="also run one plain device copy of this size (counter calibration)")
    ap.add_argument("--workload", choices=["layer128k", "layers32", "hosttier", "hosttier_layers",
                                           "prefill128k"],
                    default="layer128k",
                    help="layer128k: one 128K x 4 layer (the headline); layers32: the 32-layer, "
                         "batch-32, 32K-context step replayed as one HIP graph; hosttier: the "
                         "128K x 4 layer with its factors in pinned host memory; prefill128k: "
                         "the prefill-side builder of one 128K x 4 layer (segmentation, "
                         "summaries, randomized SVD); hosttier_layers: --layers layers of the "
                         "128K x 4 host-tier workload in one step, with and without the "
                         "cross-layer prefetch")
    ap.add_argument("--layers", type=int, default=4, help="hosttier_layers: layers per step")
    ap.add_argument("--power", type=int, default=1, help="prefill128k: subspace iterations")
    ap.add_argument("--phase-trace", metavar="OUT_MD", default=None,
                    help="diagnostic: load the phase-trace build (libsekv_trace.so), trace the "
                         "work items of a few steps of the workload (of one build for "
                         "prefill128k) and write a per-phase percentile table to OUT_MD; prints "
                         "no benchmark line")
    ap.add_argument("--trace-reps", type=int, default=3)
    ap.add_argument("--distinct-layers", type=int, default=32,
                    help="layers32: independently seeded layers generated on the host; the "
                         "32 device-resident layers cycle through them, each in its own memory")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the decode step "
              f"is not sharded across GPUs in this build.", file=sys.stderr)
        sys.exit(2)

    if args.phase_trace:
        os.environ["SEKV_LIB"] = "trace"
    import numpy as np
    import torch

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    if args.workload == "layers32":
        return bench_layers32(args, dev)
    if args.workload == "hosttier":
        return bench_hosttier(args, dev)
    if args.workload == "prefill128k":
        return bench_prefill(args, dev)
    if args.workload == "hosttier_layers":
        return bench_hosttier_layers(args, dev)

    main_run = time_layer128k(args, dev, args.variant)
    if main_run is None:                     # phase-trace mode
        return
    adaptive = None
    if not args.no_adaptive:
        adaptive = time_layer128k(args, dev, args.variant, rank_mode="adaptive")
    gated = None
    if not args.no_gated:
        gated = time_gated(args, dev, main_run["case"])
    other = None
    if not args.no_other_variant:
        other = time_layer128k(args, dev, "N" if args.variant == "L" else "L")
    ceiling = copy_ceiling(dev)
    torch.cuda.empty_cache()

    bytes_step = main_run["bytes"]["total"]
    workload = "sekv-decode-step-128k-b4-r32-k16-bf16-" + args.variant
    traffic = load_traffic(workload)
    achieved = main_run["achieved"]
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": traffic, "kernel": KERNEL_NAME,
                "kernel_us_mean": main_run["kern_us"],
                "frac_of_measured_ceiling": {k: round(achieved / v, 4) for k, v in ceiling.items()
                                             if k.endswith("GB_s")},
                "algorithmic_bytes_per_launch": bytes_step,
                **{k: main_run[k] for k in ("stream_launch_us_mean", "stream_launch_us_p50",
                                            "stream_launch_us_p90")}}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(main_run["case"], bytes_step, args.cpu_seconds)

    line = {
        "metric": METRIC, "value": round(main_run["gbs"], 1), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(main_run["wall_us"] / 1e3, 5),
        "us_per_step": round(main_run["wall_us"], 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": workload, "batch": 4, "context": 131072,
                   "n_q_heads": 32, "n_kv_heads": 8, "head_dim": 128, "rank": 32,
                   "top_k": 16, "storage_dtype": "bf16", "routing_dtype": "f64",
                   "arith": "bf16 storage, f32 accumulate, f64 routing keys",
                   "variant": args.variant, "cache_copies": main_run["copies"],
                   "parallelism": "single-gpu"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "bytes": main_run["bytes"],
        "warm_same_cache_kernel_us": main_run["warm_us"],
        "measured_ceiling": ceiling,
    }
    if other is not None:
        line["other_variant"] = {
            "variant": other["variant"], "us_per_step": round(other["wall_us"], 3),
            "kernel_us_mean": other["kern_us"], "achieved_GB_s": round(other["achieved"], 1),
            "frac": round(other["achieved"] / HBM_PEAK_GBS, 4),
            "algorithmic_bytes_per_launch": other["bytes"]["total"],
            "factor_bytes": other["bytes"]["factors"],
            "mean_selected_len": other["bytes"]["mean_selected_len"]}
    if adaptive is not None:
        br = adaptive["case"].block_rank
        live = br[br != 0]
        line["adaptive_rank"] = {
            "rule": "per-span retained ranks r_K, r_V in {8, 16, 24, 32} (uniform draw)",
            "mean_rank_k": round(float(np.mean(live & 0xFFFF)), 2),
            "mean_rank_v": round(float(np.mean(live >> 16)), 2),
            "us_per_step": round(adaptive["wall_us"], 3), "kernel_us_mean": adaptive["kern_us"],
            "achieved_GB_s": round(adaptive["achieved"], 1),
            "frac": round(adaptive["achieved"] / HBM_PEAK_GBS, 4),
            "algorithmic_bytes_per_launch": adaptive["bytes"]["total"],
            "factor_bytes": adaptive["bytes"]["factors"]}
    if gated is not None:
        line["gated"] = gated
    print(json.dumps(line), flush=True)


def time_gated(args, dev, case, route_dim=32):
    """The same layer under the learned selection rule (random projections, tau = 0.05 for
    every head, a token budget per pair): the selection kernel alone and the whole gated
    step (selection, then attention over the chosen spans), K back-to-back calls over
    rotating cache copies, one event pair around each batch."""
    import numpy as np
    import torch

    from paper_2606_31145_amd import accounting
    from paper_2606_31145_amd import sekv
    from synth import make_gate

    spec = case.spec
    budget = args.gated_budget
    gate = make_gate(case, route_dim=route_dim, tau="permissive", budget_tokens=budget)
    arrays = dict(q=case.q, anchor_k=case.anchor_k, anchor_v=case.anchor_v,
                  n_anchors=case.n_anchors, sum_k=case.sum_k, sum_v=case.sum_v,
                  n_spans=case.n_spans, span_len=case.span_len, span_logsize=case.span_logsize,
                  factors=case.factors, block_off=case.block_off)
    base = sekv.DeviceCache.from_arrays(arrays, spec.dtype, dev)
    gbase = sekv.DeviceGate.from_arrays(route_dim, gate.proj, gate.sum_route, gate.thresholds,
                                        budget, spec.dtype, dev)
    R = max(1, args.rotate)
    caches, gates = [base], [gbase]
    for _ in range(R - 1):
        caches.append(sekv.DeviceCache({k: v.clone() for k, v in base.t.items()}, spec.dtype))
        gates.append(sekv.DeviceGate(route_dim, gbase.proj.clone(), gbase.sum_route.clone(),
                                     gbase.thresholds.clone(), budget))
    dims = sekv.make_dims(batch=spec.batch, n_q_heads=spec.n_q_heads, n_kv_heads=spec.n_kv_heads,
                          head_dim=spec.head_dim, rank=spec.rank, top_k=spec.top_k,
                          max_anchors=case.max_anchors, max_spans=case.max_spans,
                          max_span_len=case.max_span_len, dtype=spec.dtype,
                          softmax_scale=spec.softmax_scale)
    ws = sekv.Workspace(dims, dev)
    stream = torch.cuda.current_stream()
    B, Hq, Hkv, d = spec.batch, spec.n_q_heads, spec.n_kv_heads, spec.head_dim
    sel = torch.empty((B, Hkv, spec.top_k), dtype=torch.int32, device=dev)
    out = torch.empty((B, Hq, d), dtype=torch.bfloat16, device=dev)
    K = args.steps

    def timed(fn):
        """Warm up eagerly, capture one call per cache copy into a HIP graph, and time
        ceil(K / R) replays with one event pair (host launch cost out of the figure)."""
        for i in range(args.warmup):
            fn(i, stream)
        torch.cuda.synchronize()
        assert ws.status() == 0, "device error word set in the gated warmup"
        cap = torch.cuda.Stream()
        cap.wait_stream(stream)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=cap):
            for j in range(R):
                fn(j, cap)
        stream.wait_stream(cap)
        graph.replay()
        torch.cuda.synchronize()
        n = max(1, -(-K // R))
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(n):
            graph.replay()
        b.record(stream)
        torch.cuda.synchronize()
        assert ws.status() == 0, "device error word set in the gated timing"
        del graph
        return a.elapsed_time(b) * 1e3 / (n * R)

    log(f"[bench] gated: timing {K} selections and {K} steps over {R} copies (graph replays)")
    route_us = timed(lambda i, st: sekv.route_gated(dims, caches[i % R], gates[i % R], ws, sel=sel,
                                                    stream=st))
    sel_np = sel.cpu().numpy()
    step_us = timed(lambda i, st: sekv.decode_step_gated(dims, caches[i % R], gates[i % R], ws,
                                                         sel=sel, out=out, stream=st))
    if not np.array_equal(sel.cpu().numpy(), sel_np):
        raise RuntimeError("gated step selected other spans than the selection kernel")
    gb = accounting.gate_bytes(n_q_heads=Hq, head_dim=d, route_dim=route_dim, elem=2,
                               n_spans=case.n_spans, top_k=spec.top_k, n_kv_heads=Hkv)
    sb = accounting.step_bytes(n_q_heads=Hq, n_kv_heads=Hkv, head_dim=d, rank=spec.rank, elem=2,
                               out_elem=2, n_anchors=case.n_anchors, n_spans=case.n_spans,
                               span_len=case.span_len, sel=sel_np)
    total = gb["total"] + sb["total"]
    res = {"rule": "learned routing: W q, sigmoid gate, per-head threshold, token budget",
           "route_dim": route_dim, "tau": 0.05, "budget_tokens": budget, "cache_copies": R,
           "selection_kernel_us": round(route_us, 3),
           "selection_bytes": gb["total"],
           "selection_GB_s": round(gb["total"] / (route_us * 1e-6) / 1e9, 1),
           "selection_frac": round(gb["total"] / (route_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
           "step_us": round(step_us, 3), "step_bytes": total,
           "step_GB_s": round(total / (step_us * 1e-6) / 1e9, 1),
           "n_selected": sb["n_selected"], "mean_selected_len": round(sb["mean_selected_len"], 1)}
    del caches, gates, base, gbase, ws
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    log(f"[bench] gated: selection {route_us:.2f} us, step {step_us:.2f} us")
    return res


def time_layer128k(args, dev, variant, rank_mode="fixed"):
    """Generate the 128K x 4 cache (one variant), time K graph-replayed steps over rotating
    device copies, then the same steps launched one by one; returns the figures.
    rank_mode "adaptive": every span block keeps its own ranks (r_K, r_V) <= 32."""
    import numpy as np
    import torch

    from paper_2606_31145_amd import accounting
    from paper_2606_31145_amd import sekv
    from synth import WORKLOADS, make_case

    from dataclasses import replace as _replace
    spec = _replace(WORKLOADS["llama3-8b-layer-128k-b4"], rank_mode=rank_mode)
    log(f"[bench] generating the 128K x 4 cache (variant {variant}, {rank_mode} ranks)")
    t0 = time.time()
    case = make_case(spec, variant=variant)
    log(f"[bench] generated in {time.time() - t0:.1f}s; factors {case.factors.nbytes / 1e6:.1f} MB")
    arrays = dict(q=case.q, anchor_k=case.anchor_k, anchor_v=case.anchor_v,
                  n_anchors=case.n_anchors, sum_k=case.sum_k, sum_v=case.sum_v,
                  n_spans=case.n_spans, span_len=case.span_len, span_logsize=case.span_logsize,
                  factors=case.factors, block_off=case.block_off, block_rank=case.block_rank)
    base = sekv.DeviceCache.from_arrays(arrays, spec.dtype, dev)
    caches = [base]
    for _ in range(max(1, args.rotate) - 1):
        caches.append(sekv.DeviceCache({k: v.clone() for k, v in base.t.items()}, spec.dtype))
    dims = sekv.make_dims(batch=spec.batch, n_q_heads=spec.n_q_heads, n_kv_heads=spec.n_kv_heads,
                          head_dim=spec.head_dim, rank=spec.rank, top_k=spec.top_k,
                          max_anchors=case.max_anchors, max_spans=case.max_spans,
                          max_span_len=case.max_span_len, dtype=spec.dtype,
                          softmax_scale=spec.softmax_scale)
    ws = sekv.Workspace(dims, dev)
    B, Hq, Hkv, d = spec.batch, spec.n_q_heads, spec.n_kv_heads, spec.head_dim
    sels = [torch.empty((B, Hkv, spec.top_k), dtype=torch.int32, device=dev) for _ in caches]
    outs = [torch.empty((B, Hq, d), dtype=torch.bfloat16, device=dev) for _ in caches]
    stream = torch.cuda.current_stream()

    def step(i):
        j = i % len(caches)
        sekv.decode_step(dims, caches[j], ws, sel=sels[j], out=outs[j], stream=stream)

    log(f"[bench] warmup {args.warmup}")
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    assert ws.status() == 0, "device error word set during warmup"
    sel_np = sels[0].cpu().numpy()
    acct = accounting.step_bytes(n_q_heads=Hq, n_kv_heads=Hkv, head_dim=d, rank=spec.rank,
                                 elem=2, out_elem=2, n_anchors=case.n_anchors,
                                 n_spans=case.n_spans, span_len=case.span_len, sel=sel_np,
                                 block_rank=case.block_rank)
    bytes_step = acct["total"]
    if args.phase_trace:
        phase_trace(args, step, len(caches), dev,
                    f"128K x 4 layer (batch 4, rank 32, top-16), variant {variant}")
        return None

    # timed region: K steps, replayed from HIP graphs with one kernel node per cache copy
    # (a full graph over every copy, then one over the first K mod copies), one event
    # pair around the whole region on the launch stream
    K = args.steps
    R = len(caches)
    graph = sekv.LayerGraph(dims, caches, ws)
    tail = sekv.LayerGraph(dims, caches[:K % R], ws) if K % R else None
    graph.launch(stream)
    if tail is not None:
        tail.launch(stream)
    torch.cuda.synchronize()
    assert ws.status() == 0, "device error word set during the graph warmup"
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    log(f"[bench] timing {K} steps over {R} cache copies (graph replays), variant {variant}")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(K // R):
        graph.launch(stream)
    if tail is not None:
        tail.launch(stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    assert ws.status() == 0, "device error word set during the timed steps"
    if not torch.equal(graph.sel[0], sels[0]):
        raise RuntimeError("graph replay selected other spans than the stream launch")
    kern_us = ev0.elapsed_time(ev1) * 1e3 / K
    graph.destroy()
    if tail is not None:
        tail.destroy()

    # the same steps launched one by one on the stream, an event pair around each launch
    # (includes each launch's dispatch), for context
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(K)]
    torch.cuda.synchronize()
    for i in range(K):
        ev[i][0].record(stream)
        step(args.warmup + i)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    kern_ms = np.array([a.elapsed_time(b) for a, b in ev])
    assert ws.status() == 0, "device error word set during the stream launches"

    # same cache every step (Infinity-Cache warm), for context only
    for _ in range(5):
        sekv.decode_step(dims, caches[0], ws, sel=sels[0], out=outs[0], stream=stream)
    torch.cuda.synchronize()
    warm = []
    for _ in range(50):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        sekv.decode_step(dims, caches[0], ws, sel=sels[0], out=outs[0], stream=stream)
        b.record(stream)
        warm.append((a, b))
    torch.cuda.synchronize()
    warm_us = float(np.mean([a.elapsed_time(b) for a, b in warm]) * 1e3)

    if args.calibration_copy_mib > 0:
        n = args.calibration_copy_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        src.fill_(1)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {n} bytes done")
        del src, dst

    res = {"variant": variant, "case": case, "bytes": dict(acct), "copies": R,
           "wall_us": wall / K * 1e6, "kern_us": round(kern_us, 3),
           "gbs": bytes_step * K / wall / 1e9, "achieved": bytes_step / (kern_us * 1e-6) / 1e9,
           "stream_launch_us_mean": round(float(kern_ms.mean() * 1e3), 3),
           "stream_launch_us_p50": round(float(np.median(kern_ms) * 1e3), 3),
           "stream_launch_us_p90": round(float(np.percentile(kern_ms, 90) * 1e3), 3),
           "warm_us": round(warm_us, 3)}
    del caches, base, graph, tail, ws, sels, outs
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    log(f"[bench] variant {variant}: {res['kern_us']:.2f} us per step (events), "
        f"{res['achieved']:.0f} GB/s")
    return res


def copy_ceiling(dev, nbytes=1 << 30, reps=20):
    """Streaming ceilings on this device, same run: a 1 GiB device-to-device copy (read +
    write bytes per second) and a 1 GiB read-only reduction (bytes read per second)."""
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    out = {}
    for name, fn, mult in (("copy", lambda: dst.copy_(src), 2), ("read", lambda: src.sum(), 1)):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        sec = a.elapsed_time(b) * 1e-3 / reps
        out[f"{name}_GB_s"] = round(mult * nbytes / sec / 1e9, 1)
    out["bytes"] = nbytes
    out["how"] = ("torch copy_ of 1 GiB (2 x bytes per second) and torch sum over 1 GiB of "
                  "float32 (bytes read per second), event-timed, 20 repetitions each")
    del src, dst
    torch.cuda.synchronize()
    log(f"[bench] measured ceilings: {out}")
    return out


def bench_layers32(args, dev):
    """32 layers x (batch 32, 32K context, rank 16, top-8), one HIP graph per step."""
    import numpy as np
    import torch

    from paper_2606_31145_amd import accounting
    from paper_2606_31145_amd import sekv
    from synth import WORKLOADS, make_case

    spec = WORKLOADS["llama3-8b-32layer-32k-b32"]
    L = spec.n_layers
    D = max(1, min(args.distinct_layers, L))
    t0 = time.time()
    cases = []
    for l in range(D):
        cases.append(make_case(spec, layer=l, variant=args.variant))
        log(f"[bench] layer {l} generated ({time.time() - t0:.1f}s)")
    base = [sekv.DeviceCache.from_arrays(dict(
        q=c.q, anchor_k=c.anchor_k, anchor_v=c.anchor_v, n_anchors=c.n_anchors, sum_k=c.sum_k,
        sum_v=c.sum_v, n_spans=c.n_spans, span_len=c.span_len, span_logsize=c.span_logsize,
        factors=c.factors, block_off=c.block_off), spec.dtype, dev) for c in cases]
    caches = []
    for l in range(L):
        src = base[l % D]
        caches.append(src if l < D else
                      sekv.DeviceCache({k: v.clone() for k, v in src.t.items()}, spec.dtype))
    torch.cuda.synchronize()
    c0 = cases[0]
    dims = sekv.make_dims(batch=spec.batch, n_q_heads=spec.n_q_heads, n_kv_heads=spec.n_kv_heads,
                          head_dim=spec.head_dim, rank=spec.rank, top_k=spec.top_k,
                          max_anchors=c0.max_anchors, max_spans=c0.max_spans,
                          max_span_len=max(c.max_span_len for c in cases), dtype=spec.dtype,
                          softmax_scale=spec.softmax_scale)
    ws = sekv.Workspace(dims, dev)
    stream = torch.cuda.current_stream()
    if args.phase_trace:
        B, Hq, Hkv, d = spec.batch, spec.n_q_heads, spec.n_kv_heads, spec.head_dim
        sel = torch.empty((B, Hkv, spec.top_k), dtype=torch.int32, device=dev)
        out = torch.empty((B, Hq, d), dtype=torch.bfloat16, device=dev)

        def step(i):
            sekv.decode_step(dims, caches[i % L], ws, sel=sel, out=out, stream=stream)

        for i in range(args.warmup):
            step(i)
        torch.cuda.synchronize()
        assert ws.status() == 0, "device error word set during warmup"
        phase_trace(args, step, L, dev, "one layer of the 32-layer step (batch 32, 32K context, "
                    f"rank 16, top-8), variant {args.variant}, launched alone",
                    extra=f" --workload layers32 --distinct-layers {D} --warmup {args.warmup}")
        return None
    graph = sekv.LayerGraph(dims, caches, ws)
    log(f"[bench] 32-layer graph built; warmup {args.warmup}")
    for _ in range(args.warmup):
        graph.launch(stream)
    torch.cuda.synchronize()
    assert ws.status() == 0, "device error word set during warmup"
    sel_np = graph.sel.cpu().numpy()
    per_layer = [accounting.step_bytes(n_q_heads=spec.n_q_heads, n_kv_heads=spec.n_kv_heads,
                                       head_dim=spec.head_dim, rank=spec.rank, elem=2,
                                       out_elem=2, n_anchors=cases[l % D].n_anchors,
                                       n_spans=cases[l % D].n_spans,
                                       span_len=cases[l % D].span_len, sel=sel_np[l])
                 for l in range(L)]
    bytes_step = int(sum(a["total"] for a in per_layer))
    K = args.steps
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        ev[i][0].record(stream)
        graph.launch(stream)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    assert ws.status() == 0, "device error word set during the timed steps"
    step_ms = np.array([a.elapsed_time(b) for a, b in ev])
    step_us = float(step_ms.mean() * 1e3)
    achieved = bytes_step / (step_us * 1e-6) / 1e9
    graph.destroy()
    workload = f"sekv-decode-step-32layer-32k-b32-r16-k8-bf16-{args.variant}"
    line = {
        "metric": "decode-step latency (µs) and achieved HBM GB/s, 32 layers, 32K context, batch 32",
        "value": round(bytes_step * K / wall / 1e9, 1), "unit": "GB/s", "n_gpus": 1,
        "steps": K, "warmup": args.warmup, "ms_per_step": round(wall / K * 1e3, 5),
        "us_per_step": round(wall / K * 1e6, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": workload, "layers": L, "distinct_layer_seeds": D,
                   "batch": spec.batch, "context": spec.context, "n_q_heads": spec.n_q_heads,
                   "n_kv_heads": spec.n_kv_heads, "head_dim": spec.head_dim, "rank": spec.rank,
                   "top_k": spec.top_k, "storage_dtype": "bf16", "routing_dtype": "f64",
                   "variant": args.variant, "graph": "hipGraph, one kernel node per layer",
                   "parallelism": "single-gpu"},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": KERNEL_NAME, "graph_us_mean": round(step_us, 3),
                     "graph_us_p50": round(float(np.median(step_ms) * 1e3), 3),
                     "graph_us_p90": round(float(np.percentile(step_ms, 90) * 1e3), 3),
                     "algorithmic_bytes_per_step": bytes_step},
        "cpu_baseline": None,
        "bytes_per_layer_mean": {k: float(np.mean([a[k] for a in per_layer])) for k in per_layer[0]},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(cases[0], per_layer[0]["total"], args.cpu_seconds,
                                            what="full decode steps of one layer of the 32-layer "
                                                 "workload (batch 32, 32K)")
    print(json.dumps(line), flush=True)


def bench_hosttier(args, dev):
    """128K x 4 layer; factors in pinned host memory, selected blocks moved per step, in
    both copy modes of the tier (device-planned gather kernel; host-planned hipMemcpyAsync
    per run of neighbouring blocks)."""
    import numpy as np
    import torch

    from paper_2606_31145_amd import accounting
    from paper_2606_31145_amd import sekv
    from synth import WORKLOADS, make_case

    spec = WORKLOADS["llama3-8b-layer-128k-b4-hosttier"]
    t0 = time.time()
    case = make_case(spec, variant=args.variant)
    log(f"[bench] generated in {time.time() - t0:.1f}s")
    dummy = np.zeros(256, dtype=np.uint8)       # the device cache carries no factors
    arrays = dict(q=case.q, anchor_k=case.anchor_k, anchor_v=case.anchor_v,
                  n_anchors=case.n_anchors, sum_k=case.sum_k, sum_v=case.sum_v,
                  n_spans=case.n_spans, span_len=case.span_len, span_logsize=case.span_logsize,
                  factors=dummy, block_off=case.block_off)
    dc = sekv.DeviceCache.from_arrays(arrays, spec.dtype, dev)
    host = sekv.HostFactors(case.factors, case.block_off, case.span_len)
    dims = sekv.make_dims(batch=spec.batch, n_q_heads=spec.n_q_heads, n_kv_heads=spec.n_kv_heads,
                          head_dim=spec.head_dim, rank=spec.rank, top_k=spec.top_k,
                          max_anchors=case.max_anchors, max_spans=case.max_spans,
                          max_span_len=case.max_span_len, dtype=spec.dtype,
                          softmax_scale=spec.softmax_scale)
    ws = sekv.Workspace(dims, dev)
    side = torch.cuda.Stream()
    stream = torch.cuda.current_stream()
    B, Hq, Hkv, d = spec.batch, spec.n_q_heads, spec.n_kv_heads, spec.head_dim
    sel = torch.empty((B, Hkv, spec.top_k), dtype=torch.int32, device=dev)
    out = torch.empty((B, Hq, d), dtype=torch.bfloat16, device=dev)
    # pinned H2D hipMemcpyAsync bandwidth of one large copy, for context
    probe = torch.empty(256 << 20, dtype=torch.uint8, pin_memory=True)
    probe_d = torch.empty(probe.numel(), dtype=torch.uint8, device=dev)
    probe_d.copy_(probe, non_blocking=True)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(5):
        probe_d.copy_(probe, non_blocking=True)
    b.record()
    torch.cuda.synchronize()
    h2d_gbs = 5 * probe.numel() / (a.elapsed_time(b) * 1e-3) / 1e9
    del probe, probe_d
    modes = {}
    for mode in ("gather", "memcpy"):
        tier = sekv.Tier(dims, mode)
        for _ in range(args.warmup):
            sekv.decode_step_tiered(dims, dc, host, tier, ws, sel=sel, out=out, stream=stream, side=side)
        torch.cuda.synchronize()
        assert ws.status() == 0
        K = args.steps
        walls, copy_ms, copy_bytes, n_copies = [], [], [], []
        for _ in range(K):
            t1 = time.perf_counter()
            sekv.decode_step_tiered(dims, dc, host, tier, ws, sel=sel, out=out, stream=stream, side=side)
            torch.cuda.synchronize()
            walls.append(time.perf_counter() - t1)
            nb, nc, ms = tier.last_copy()
            copy_ms.append(ms)
            copy_bytes.append(nb)
            n_copies.append(nc)
        assert ws.status() == 0
        staging = tier.staging_bytes
        tier.destroy()
        step_s = float(np.median(walls))
        modes[mode] = {"us_per_step": round(step_s * 1e6, 1),
                       "us_per_step_p90": round(float(np.percentile(walls, 90)) * 1e6, 1),
                       "bytes_per_step": int(np.mean(copy_bytes)),
                       "copies_per_step": float(np.mean(n_copies)),
                       "copy_ms_per_step": round(float(np.mean(copy_ms)), 4),
                       "host_link_GB_s": round(float(np.mean(copy_bytes)) /
                                               (float(np.mean(copy_ms)) * 1e-3) / 1e9, 2)}
        log(f"[bench] hosttier {mode}: {modes[mode]}")
    sel_np = sel.cpu().numpy()
    acct = accounting.step_bytes(n_q_heads=Hq, n_kv_heads=Hkv, head_dim=d, rank=spec.rank,
                                 elem=2, out_elem=2, n_anchors=case.n_anchors,
                                 n_spans=case.n_spans, span_len=case.span_len, sel=sel_np)
    # HBM held by the tiered step vs a dense bf16 cache of the same tokens
    resident = int(sum(t.numel() * t.element_size() for k, t in dc.t.items() if k != "factors")
                   + staging)
    full = accounting.full_kv_bytes_same_shapes(n_kv_heads=Hkv, head_dim=d, elem=2,
                                                n_anchors=case.n_anchors, span_len=case.span_len)
    g = modes["gather"]
    line = {
        "metric": "decode-step latency (µs), host-link GB/s and HBM saved, 128K context, batch 4, "
                  "factors in pinned host memory",
        "value": g["us_per_step"], "unit": "us", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(g["us_per_step"] / 1e3, 4),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"sekv-decode-step-128k-b4-r32-k16-bf16-hosttier-{args.variant}",
                   "batch": B, "context": spec.context, "rank": spec.rank, "top_k": spec.top_k,
                   "variant": args.variant, "tier_mode": "gather", "parallelism": "single-gpu"},
        "host_link": g,
        "modes": modes,
        "pinned_h2d_memcpy_GB_s": round(h2d_gbs, 2),
        "hbm": {"resident_bytes": resident, "full_bf16_kv_bytes": full,
                "saved_frac": round(1.0 - resident / full, 4),
                "algorithmic_bytes_per_step": acct["total"]},
    }
    print(json.dumps(line), flush=True)


def bench_prefill(args, dev):
    """The prefill-side builder for one 128K x 4 layer of the headline shape (Hkv 8, d 128,
    bfloat16, R_max 32, sketch 40): segmentation, then anchors, summaries and the
    randomized SVD of every span.  Kernel times from HIP events on the launch stream; the
    whole call (with the span-table read-back and the host layout) by wall clock."""
    import numpy as np
    import torch

    from paper_2606_31145_amd import sekv
    from synth import make_prefill

    B, Hkv, d, N = 4, 8, 128, 131072
    R, l = 32, 40
    t0 = time.time()
    # one generated key/value stream per sequence; KV head g holds it with its feature columns
    # rotated by 8 g (a permutation: the same spans, ranks and spectra, distinct memory)
    p = make_prefill(B, 1, d, N, dtype="bf16", spike_every=170, true_rank=24, noise=0.02,
                     sketch=l, seed=5)
    log(f"[bench] prefill generated in {time.time() - t0:.1f}s")

    def to_dev(a, bf16=False):
        a = np.ascontiguousarray(a)
        t = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16) if bf16 else torch.from_numpy(a)
        return t.to(dev)

    def heads(a):
        t = to_dev(a, True)                                          # [B][1][N][d]
        return torch.cat([torch.roll(t, 8 * g, dims=3) for g in range(Hkv)], dim=1).contiguous()

    keys, values = heads(p.keys), heads(p.values)
    del p.keys, p.values
    H, n_tok, omega = to_dev(p.surprisal), to_dev(p.n_tokens), to_dev(p.omega)
    bd = sekv.make_build_dims(batch=B, n_kv_heads=Hkv, head_dim=d, max_tokens=N, rank=R, sketch=l,
                              min_span=16, window=512, dtype="bf16", alpha=1.0, sweeps=8,
                              power=args.power)
    wdims = sekv.make_dims(batch=1, n_q_heads=1, n_kv_heads=1, head_dim=64, rank=8, top_k=1,
                           max_anchors=1, max_spans=1, max_span_len=1, dtype="f32",
                           softmax_scale=1.0)
    ws = sekv.Workspace(wdims, dev)
    stream = torch.cuda.current_stream()
    cache, seg, lay = sekv.build_layer(bd, keys, values, H, n_tok, omega, ws)
    torch.cuda.synchronize()
    assert ws.status() == 0
    block_off = cache["block_off"]
    walls = []
    for _ in range(max(1, min(args.warmup, 3))):
        sekv.build_layer(bd, keys, values, H, n_tok, omega, ws)
    torch.cuda.synchronize()
    K = max(1, min(args.steps, 10))
    for _ in range(K):
        t1 = time.perf_counter()
        sekv.build_layer(bd, keys, values, H, n_tok, omega, ws)
        torch.cuda.synchronize()
        walls.append(time.perf_counter() - t1)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    seg_ms, build_ms = [], []
    for _ in range(K):
        ev[0].record(stream)
        seg2 = sekv.segment(bd, H, n_tok, stream)
        ev[1].record(stream)
        sekv.build_cache(bd, keys, values, H, n_tok, seg2, omega, lay["max_anchors"], lay["max_spans"],
                         block_off, lay["factors_bytes"], ws, out=cache, stream=stream)
        ev[2].record(stream)
        torch.cuda.synchronize()
        seg_ms.append(ev[0].elapsed_time(ev[1]))
        build_ms.append(ev[1].elapsed_time(ev[2]))
    assert ws.status() == 0
    if args.phase_trace:
        builder_phase_trace(args, bd, keys, values, H, n_tok, seg2, omega, lay, cache, block_off, ws, dev)
        return
    tokens = B * N
    kern_ms = float(np.mean(seg_ms)) + float(np.mean(build_ms))
    span_tokens = int(sum(int(cache["span_len"][b, :int(lay["n_spans"][b])].sum().item()) for b in range(B)))
    kv_bytes = 2 * B * Hkv * N * d * 2
    out_bytes = int(sum(cache[k].numel() * cache[k].element_size()
                        for k in ("anchor_k", "anchor_v", "sum_k", "sum_v", "factors")))
    wall_ms = float(np.median(walls)) * 1e3
    # algorithmic work of the SVD (the dominant kernel): per span side of |S| tokens, each of
    # the power + 1 sketch passes forms Y = X Omega (2 |S| d l), Y^T X (2 l |S| d) and Y^T Y
    # (2 l^2 |S|); the last pass forms Y again and U = Y T (2 |S| l r).  The small dense
    # algebra (Cholesky, Jacobi) is not counted.
    flops = 0.0
    for b in range(B):
        for Ls in cache["span_len"][b, :int(lay["n_spans"][b])].cpu().numpy().astype(np.float64):
            r_ = min(Ls, d, R)
            per = (args.power + 1) * (2 * Ls * d * l * 2 + 2 * l * l * Ls) + 2 * Ls * d * l + 2 * Ls * l * r_
            flops += 2 * Hkv * per                                   # both sides, every KV head
    build_s = float(np.mean(build_ms)) * 1e-3
    line = {
        "metric": "prefill-side build throughput (tokens per second per layer), 128K context, batch 4",
        "value": round(tokens / (kern_ms * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(kern_ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "sekv-prefill-build-128k-b4-hkv8-d128-r32-l40-bf16", "batch": B,
                   "context": N, "n_kv_heads": Hkv, "head_dim": d, "rank": R, "sketch": l,
                   "power": args.power, "min_span": 16, "window": 512, "alpha": 1.0,
                   "heads": "one generated stream per sequence, head g with columns rotated by 8 g",
                   "parallelism": "single-gpu"},
        "roofline": {"bound": "alu", "achieved": round(flops / build_s / 1e12, 3),
                     "peak": FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(flops / build_s / 1e12 / FP32_PEAK_TFLOPS, 5), "traffic": None,
                     "kernel": "svd_kernel (+ gather_kernel in the timed launch pair)",
                     "algorithmic_flops_per_launch": flops,
                     "note": "latency-bound: per span side, 40-step Cholesky factorisations and "
                             "Jacobi rounds with a workgroup barrier each"},
        "segment_ms": round(float(np.mean(seg_ms)), 4),
        "build_ms": round(float(np.mean(build_ms)), 4),
        "call_wall_ms_with_layout": round(wall_ms, 3),
        "spans": [int(x) for x in lay["n_spans"]], "anchors": [int(x) for x in lay["n_anchors"]],
        "span_tokens": span_tokens,
        "hbm": {"kv_read_bytes": kv_bytes, "written_bytes": out_bytes,
                "GB_s_kv_once": round((kv_bytes + out_bytes) / (kern_ms * 1e-3) / 1e9, 1)},
    }
    print(json.dumps(line), flush=True)


BUILD_PHASES = [("sketch pass", 2), ("Cholesky", 3), ("R^-1, B", 4), ("B B^T", 5),
                ("iteration (Cholesky + R2^-1 + basis)", 6), ("last pass", 7), ("Cholesky", 8),
                ("R^-1, B", 9), ("B B^T", 10), ("Jacobi", 11), ("V rows", 12), ("T", 13), ("U pass", 14)]


def builder_phase_trace(args, bd, keys, values, H, n_tok, seg, omega, lay, cache, block_off, ws, dev):
    """One build_cache of the trace build with a phase-trace buffer: per span side, the time
    of each phase of the randomized SVD (percentiles over the span sides of the layer)."""
    import numpy as np
    import torch

    from paper_2606_31145_amd import sekv
    slots = 16
    items = 2 * bd.batch * bd.n_kv_heads * int(lay["max_spans"])
    buf = torch.zeros(items * slots, dtype=torch.int64, device=dev)
    sekv.phase_trace(buf)
    sekv.build_cache(bd, keys, values, H, n_tok, seg, omega, lay["max_anchors"], lay["max_spans"], block_off,
                     lay["factors_bytes"], ws, out=cache)
    torch.cuda.synchronize()
    sekv.phase_trace(None)
    assert ws.status() == 0
    t = buf.cpu().numpy().reshape(items, slots)
    t = t[t[:, 1] > 0]
    L = t[:, 0].astype(np.float64)

    def pct(x):
        return "".join(f"| {v:.1f} " for v in np.percentile(x, [10, 50, 90]))

    lines = ["# Phase trace of the SVD kernel (trace build), one 128K x 4 layer", "",
             "Per span side, microseconds between the phase marks (the device's 100 MHz real-time "
             "counter, stamped by thread 0 of the span side's workgroup; trace build "
             "`libsekv_trace.so`, same sources compiled with `SEKV_PHASE_TRACE`).  Columns: "
             "percentiles 10 / 50 / 90 over the span sides.", "",
             f"Command: `python bench.py --workload prefill128k --phase-trace OUT.md`"
             + (f" `--power {args.power}`" if args.power != 1 else ""), "",
             f"{len(t)} span sides; |S| p10 / p50 / p90: {np.percentile(L, 10):.0f} / "
             f"{np.percentile(L, 50):.0f} / {np.percentile(L, 90):.0f} tokens.", "",
             "| phase | p10 | p50 | p90 |", "|---|---|---|---|"]
    prev = t[:, 1]
    for label, slot in BUILD_PHASES:
        cur = t[:, slot]
        ok = cur > 0
        lines.append(f"| {label} " + pct((cur[ok] - prev[ok]) * 0.01) + "|")
        prev = np.where(ok, cur, prev)
    lines.append("| whole span side " + pct((t[:, 14] - t[:, 1]) * 0.01) + "|")
    lines.append("")
    lines.append(f"First start to last end: {(t[:, 14].max() - t[:, 1].min()) * 0.01:.0f} us.")
    text = "\n".join(lines) + "\n"
    with open(args.phase_trace, "w") as f:
        f.write(text)
    log(text)
    print(json.dumps({"phase_trace": args.phase_trace, "span_sides": int(len(t))}), flush=True)


def bench_hosttier_layers(args, dev):
    """--layers layers of the 128K x 4 host-tier workload (planted variant, the planted spans
    shared by the layers) as one layered tiered step: with the cross-layer prefetch and
    without.  Wall time per step, copies after each selection (the critical path) and
    prefetched copies."""
    import numpy as np
    import torch

    from paper_2606_31145_amd import sekv
    from synth import WORKLOADS, make_case

    spec = WORKLOADS["llama3-8b-layer-128k-b4-hosttier"]
    L = max(1, args.layers)
    t0 = time.time()
    cases = [make_case(spec, layer=l, variant="N", needle_layer=0) for l in range(L)]
    log(f"[bench] {L} layers generated in {time.time() - t0:.1f}s")
    dummy = np.zeros(256, dtype=np.uint8)
    dcs, hosts = [], []
    for c in cases:
        arrays = dict(q=c.q, anchor_k=c.anchor_k, anchor_v=c.anchor_v, n_anchors=c.n_anchors,
                      sum_k=c.sum_k, sum_v=c.sum_v, n_spans=c.n_spans, span_len=c.span_len,
                      span_logsize=c.span_logsize, factors=dummy, block_off=c.block_off)
        dcs.append(sekv.DeviceCache.from_arrays(arrays, spec.dtype, dev))
        hosts.append(sekv.HostFactors(c.factors, c.block_off, c.span_len))
    c0 = cases[0]
    dims = sekv.make_dims(batch=spec.batch, n_q_heads=spec.n_q_heads, n_kv_heads=spec.n_kv_heads,
                          head_dim=spec.head_dim, rank=spec.rank, top_k=spec.top_k,
                          max_anchors=max(c.max_anchors for c in cases),
                          max_spans=max(c.max_spans for c in cases),
                          max_span_len=max(c.max_span_len for c in cases), dtype=spec.dtype,
                          softmax_scale=spec.softmax_scale)
    ws = sekv.Workspace(dims, dev)
    tier = sekv.Tier(dims, "gather")
    side = torch.cuda.Stream()
    modes = {}
    for prefetch in (False, True):
        for _ in range(max(1, args.warmup)):
            sekv.decode_layers_tiered(dims, dcs, hosts, tier, ws, prefetch=prefetch, side=side)
        torch.cuda.synchronize()
        assert ws.status() == 0
        walls = []
        for _ in range(max(1, args.steps)):
            t1 = time.perf_counter()
            sel, out = sekv.decode_layers_tiered(dims, dcs, hosts, tier, ws, prefetch=prefetch, side=side)
            torch.cuda.synchronize()
            walls.append(time.perf_counter() - t1)
        assert ws.status() == 0
        cb, cn, pb, pn = tier.layer_stats()
        key = "prefetch" if prefetch else "no_prefetch"
        modes[key] = {"us_per_step": round(float(np.median(walls)) * 1e6, 1),
                      "us_per_layer": round(float(np.median(walls)) * 1e6 / L, 1),
                      "critical_bytes_per_step": cb, "critical_blocks_per_step": cn,
                      "prefetched_bytes_per_step": pb, "prefetched_blocks_per_step": pn}
        log(f"[bench] layered tier {key}: {modes[key]}")
    sel_np = sel.cpu().numpy()
    hits = tot = 0
    for l in range(1, L):
        for b in range(spec.batch):
            for g in range(spec.n_kv_heads):
                prev = set(int(x) for x in sel_np[l - 1, b, g] if x >= 0)
                cur = [int(x) for x in sel_np[l, b, g] if x >= 0]
                tot += len(cur)
                hits += sum(1 for x in cur if x in prev)
    tier.destroy()
    p_, n_ = modes["prefetch"], modes["no_prefetch"]
    line = {
        "metric": "layered decode-step latency (µs), factors in pinned host memory, cross-layer prefetch",
        "value": p_["us_per_step"], "unit": "us", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(p_["us_per_step"] / 1e3, 4), "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"sekv-decode-{L}-layers-128k-b4-r32-k16-bf16-hosttier-N-shared",
                   "layers": L, "batch": spec.batch, "context": spec.context, "rank": spec.rank,
                   "top_k": spec.top_k, "variant": "N, planted spans shared by the layers",
                   "parallelism": "single-gpu"},
        "modes": modes,
        "prefetch_hit_rate": round(hits / tot, 4) if tot else None,
        "speedup": round(n_["us_per_step"] / p_["us_per_step"], 3),
        "note": "copies serialise on the side stream: prefetch hides them behind the attention "
                "and routing between two selections, so it gains at most that compute time per "
                "layer while the step is bound by the host link",
    }
    print(json.dumps(line), flush=True)


TRACE_ROUTE = [("start", 1), ("k rows loaded", 3), ("scored", 4), ("chunk sorted", 5),
               ("candidates published", 6), ("end", 2)]
TRACE_SHARE = [("start", 1), ("anchors folded", 3), ("first candidate poll answered", 13),
               ("selection known", 4),
               ("zoom: first factor loads issued", 5), ("zoom: mid fold done", 6),
               ("zoom: Vt_K q done", 7), ("zoom: token blocks done", 8), ("zoom: done", 9),
               ("summary share done", 10), ("partial written", 11), ("merged", 12), ("end", 2)]


def phase_trace(args, step, n_rot, dev, what, extra=""):
    """Trace the work items of single steps (trace build) and write a percentile table."""
    import numpy as np
    import torch

    from paper_2606_31145_amd import sekv
    slots = 16
    buf = torch.zeros(1 << 20, dtype=torch.int64, device=dev)     # up to 65 536 items
    sekv.phase_trace(buf)
    reps = []
    for r in range(args.trace_reps):
        for i in range(n_rot):                                     # touch every copy
            step(i)
        torch.cuda.synchronize()
        buf.zero_()
        torch.cuda.synchronize()
        step(r)                                                    # the traced step
        torch.cuda.synchronize()
        tr = buf.cpu().numpy().reshape(-1, slots)
        tr = tr[tr[:, 1] != 0]
        reps.append(tr)
    sekv.phase_trace(None)

    def pct(x):
        x = x[np.isfinite(x)]
        if len(x) == 0:
            return "| – " * 5
        return "".join(f"| {v:.2f} " for v in np.percentile(x, [0, 10, 50, 90, 100]))

    lines = [f"# Phase trace: {what}", "",
             "Per work item, microseconds from the first item's start (the device's 100 MHz "
             "real-time counter, stamped by thread 0 of the item's workgroup; trace build "
             "`libsekv_trace.so`, same sources compiled with `SEKV_PHASE_TRACE`).  Columns: "
             "percentiles 0 / 10 / 50 / 90 / 100 over the items of one step.", "",
             "Command: `python bench.py --phase-trace OUT.md" + extra +
             (f" --variant {args.variant}" if args.variant != "L" else "") + "`", ""]
    for r, tr in enumerate(reps):
        kind = tr[:, 0] >> 60
        xcc = (tr[:, 0] >> 48) & 0xF
        t0 = tr[:, 1].min()
        rel = (tr[:, 1:].astype(np.float64) - t0) * 0.01
        rel[tr[:, 1:] == 0] = np.nan
        span = np.nanmax(rel)
        lines += [f"## step {r}: {int((kind == 0).sum())} routing items, "
                  f"{int((kind == 1).sum())} share items, first start to last end "
                  f"{span:.2f} us, workgroups on {len(set(xcc.tolist()))} XCDs", "",
                  "| item | phase mark | p0 | p10 | p50 | p90 | p100 |", "|---|---|---|---|---|---|---|"]
        for nm, table in (("routing", TRACE_ROUTE), ("share", TRACE_SHARE)):
            sel = kind == (0 if nm == "routing" else 1)
            for label, slot in table:
                lines.append(f"| {nm} | {label} " + pct(rel[sel, slot - 1]) + "|")
        polls = tr[kind == 1, 14].astype(np.float64)
        polls = polls[polls > 0]
        if len(polls):
            lines.append("| share | candidate polls (count, not us) " + pct(polls) + "|")
        lines.append("")
    text = "\n".join(lines) + "\n"
    with open(args.phase_trace, "w") as f:
        f.write(text)
    log(text)
    print(json.dumps({"phase_trace": args.phase_trace, "steps": len(reps)}), flush=True)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(case, bytes_step, seconds, what="full decode steps of the same 128K x 4 layer"):
    """The oracle, as it stands, timed on the host on the same workload: BLAS limited to all
    usable cores, then to one thread (about seconds/2 of CPU time each)."""
    import numpy as np

    import oracle
    try:
        from threadpoolctl import threadpool_limits
    except Exception:  # pragma: no cover
        threadpool_limits = None
    s = case.spec
    kw = dict(q=case.q, anchor_k=case.anchor_k, anchor_v=case.anchor_v, n_anchors=case.n_anchors,
              sum_k=case.sum_k, sum_v=case.sum_v, n_spans=case.n_spans, span_len=case.span_len,
              span_logsize=case.span_logsize, factors=case.factors, block_off=case.block_off,
              rank=s.rank, top_k=s.top_k, softmax_scale=s.softmax_scale, dtype=s.dtype)
    cores = len(os.sched_getaffinity(0))
    runs = {}
    for label, threads in (("all", cores), ("one", 1)):
        ctx = threadpool_limits(limits=threads) if threadpool_limits else None
        if ctx:
            ctx.__enter__()
        try:
            times = []
            t_end = time.perf_counter() + seconds / 2
            while True:
                t0 = time.perf_counter()
                oracle.decode_step(**kw)
                times.append(time.perf_counter() - t0)
                if time.perf_counter() > t_end or len(times) >= 100:
                    break
        finally:
            if ctx:
                ctx.__exit__(None, None, None)
        runs[label] = (float(np.median(times)), len(times), threads)
        log(f"[bench] oracle, BLAS threads {threads}: {len(times)} steps, median {runs[label][0]:.3f}s")
    per, n, threads = runs["all"]
    per1, n1, _ = runs["one"]
    return {"value": round(bytes_step / per / 1e9, 4), "unit": "GB/s", "cores": threads,
            "kind": "oracle", "us_per_step": round(per * 1e6, 1),
            "sample": f"{n} {what}, median, numpy float64, BLAS threads limited to the "
                      f"{threads} usable cores (the oracle's own loops run on one)",
            "cpu_model": cpu_model(), "usable_cores": cores,
            "one_thread": {"value": round(bytes_step / per1 / 1e9, 4), "unit": "GB/s", "cores": 1,
                           "us_per_step": round(per1 * 1e6, 1), "steps": n1}}


if __name__ == "__main__":
    main()
