#!/usr/bin/env python3
"""Benchmark of the convolution hot path on one MI355X.

A step is one forward pass over every convolution layer of a workload (by
default the 53 convolutions of ResNet-50 at batch 32, bf16 data, fp32
accumulation), each layer running the algorithm chosen for it by measured
per-layer selection (every supported algorithm timed on that layer before
the timed region; the fastest goes into the algorithm table).  Inputs,
weights and outputs are resident in HBM before timing starts.

Prints one JSON line: throughput (TFLOP/s, 2*N*K*(C/G)*R*S*P*Q per layer),
the roofline of the dominant kernel measured with HIP events inside the
timed region, and the CPU oracle timed on a bounded sample on the host.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload resnet50]
                    [--select measured|default|<algo>] [--graph] [--sweep FILE]
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAKS_TFLOPS = {"bf16": 2500.0, "f32": 157.3}   # dense MFMA peaks of MI355X
HBM_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def build_plan(layers, wl_index, device, select, algos_allowed=None):
    """Resident tensors, descriptors and the chosen algorithm of every layer."""
    import torch
    import paper_2410_08300_amd as cs
    from paper_2410_08300_amd import _lib, workloads as W

    plan = []
    cache = {}   # selection is per unique shape
    for li, L in enumerate(layers):
        x, w, b = W.make_tensors(L, (wl_index, li, 3), device=device)
        y = torch.empty((L.n, L.k, L.p, L.q), device=device, dtype=x.dtype)
        desc = _lib.make_desc(L.n, L.c, L.h, L.w, L.k, L.r, L.s, L.stride, L.pad, L.dilation, L.groups,
                              L.dtype, b is not None, L.relu)
        key = L.shape_key()
        if key not in cache:
            if select == "measured":
                best, timings = cs.select_fastest(x, w, b, L.stride, L.pad, L.dilation, L.groups, L.relu,
                                                  algos=algos_allowed)
                cache[key] = (best, timings)
            elif select == "default":
                cache[key] = (_lib.default_algo(desc), {})
            else:
                cache[key] = (select, {})
        algo, timings = cache[key]
        pk = cs.pack_filters(w, tuple(x.shape), L.stride, L.pad, L.dilation, L.groups, algo, b is not None, L.relu)
        plan.append(dict(layer=L, x=x, w=w, b=b, y=y, desc=desc, algo=algo, algo_id=_lib.algo_id(algo),
                         ws_bytes=_lib.workspace_bytes(desc, algo), package=pk,
                         pk_ws_bytes=_lib.prepacked_workspace_bytes(desc, algo), timings=timings,
                         describe=_lib.describe(desc, algo)))
    ws_max = max(max(p["ws_bytes"], p["pk_ws_bytes"]) for p in plan)
    ws = torch.empty(max(ws_max, 1), dtype=torch.uint8, device=device)
    return plan, ws


def make_step(plan, ws, stream_ptr, prepacked=False):
    """A closure that enqueues every layer through the C ABI with prebuilt
    arguments (no allocation, no Python-side shape work per call).  With
    prepacked=True each layer uses its filter package (conv2d_prepacked);
    otherwise conv2d() rebuilds the package from the filters every call."""
    import ctypes
    from paper_2410_08300_amd import _lib

    L = _lib.lib()
    fn = L.conv2d_prepacked if prepacked else L.conv2d
    calls = []
    for p in plan:
        wsrc = p["package"] if prepacked else p["w"]
        calls.append((ctypes.c_void_p(p["x"].data_ptr()), ctypes.c_void_p(wsrc.data_ptr()),
                      ctypes.c_void_p(p["b"].data_ptr() if p["b"] is not None else 0),
                      ctypes.c_void_p(p["y"].data_ptr()), ctypes.byref(p["desc"]), p["algo_id"],
                      ctypes.c_void_p(ws.data_ptr()),
                      ctypes.c_size_t(p["pk_ws_bytes"] if prepacked else p["ws_bytes"]),
                      ctypes.c_void_p(stream_ptr)))

    def step(events=None):
        for i, args in enumerate(calls):
            if events is not None:
                events[i][0].record()
            st = fn(*args)
            if events is not None:
                events[i][1].record()
            if st:
                raise _lib.Conv2dError(st, "layer %d" % i)
    return step


def cpu_baseline(workload, budget_s=20.0):
    """The fp64 CPU oracle on a bounded sample of the same layers: all layers
    of the workload at batch 1 (one image), repeated while the time budget
    lasts.  Returns TFLOP/s of the sample."""
    import numpy as np
    import oracle
    from paper_2410_08300_amd import workloads as W

    layers = W.layers(workload, n=1)
    flops = 0
    t_total = 0.0
    images = 0
    rng = np.random.default_rng(0)
    while images == 0 or (t_total < budget_s and images < 64):
        for L in layers:
            x = rng.standard_normal((L.n, L.c, L.h, L.w))
            w = rng.standard_normal((L.k, L.c // L.groups, L.r, L.s))
            t0 = time.perf_counter()
            oracle.conv2d(x, w, None, L.stride, L.pad, L.dilation, L.groups, L.relu)
            t_total += time.perf_counter() - t0
            flops += L.flops
        images += 1
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": flops / t_total / 1e12, "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "sample": "all %d conv layers of %s at batch 1, %d image(s) (%.1f GFLOP, %.1f s), fp64 C loops "
                      "with OpenMP" % (len(layers), workload, images, flops / 1e9, t_total)}


def sweep(path, steps):
    """Every algorithm on every unique layer of all five workloads: JSONL rows."""
    import torch
    import paper_2410_08300_amd as cs
    from paper_2410_08300_amd import workloads as W

    dev = torch.device("cuda:0")
    with open(path, "w") as f:
        for wi, wl in enumerate(W.WORKLOADS):
            for li, (L, count) in enumerate(W.unique_layers(W.layers(wl))):
                x, w, b = W.make_tensors(L, (wi, li, 4), device=dev)
                for algo in cs.supported_algos(x, w, b, L.stride, L.pad, L.dilation, L.groups, L.relu):
                    ms = cs.time_conv(x, w, b, L.stride, L.pad, L.dilation, L.groups, algo, L.relu,
                                      warmup=2, reps=steps)
                    tf = L.flops / (ms * 1e-3) / 1e12
                    gbs = L.compulsory_bytes() / (ms * 1e-3) / 1e9
                    row = dict(workload=wl, layer=L.name, count=count, shape=L.asdict(), algo=algo, ms=ms,
                               tflops=tf, frac_mfma_peak=tf / PEAKS_TFLOPS[L.dtype], gbs=gbs,
                               frac_hbm=gbs / HBM_GBS, flops=L.flops, bytes=L.compulsory_bytes())
                    f.write(json.dumps(row) + "\n")
                    f.flush()
                    log("sweep %-12s %-22s %-14s %9.4f ms %8.2f TFLOP/s %8.1f GB/s"
                        % (wl, L.name, algo, ms, tf, gbs))
                del x, w, b
                torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="resnet50")
    ap.add_argument("--select", default="measured")
    ap.add_argument("--graph", action="store_true", help="replay the step as a captured HIP graph")
    ap.add_argument("--prepacked", action="store_true",
                    help="time the step with filter packages built before timing (conv2d_prepacked); by default "
                         "every call rebuilds them from the filters")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--sweep", default=None, help="write per-layer, per-algorithm timings to this JSONL file")
    args = ap.parse_args()

    if args.gpus != 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path "
              "(the convolution shards over the batch with no exchange step; see DESIGN.md)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2410_08300_amd import _lib, workloads as W

    _lib.lib()   # fail loudly if the HIP library is missing
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.sweep:
        sweep(args.sweep, max(args.steps, 3))
        return

    wl = args.workload
    layers = W.layers(wl)
    log("bench: workload %s, %d layers, select=%s" % (wl, len(layers), args.select))
    plan, ws = build_plan(layers, W.WORKLOADS.index(wl), dev, args.select)
    torch.cuda.synchronize()  # filter packages were built on the default stream
    for p in plan:
        L = p["layer"]
        log("  %-24s %-14s %s" % (L.name, p["algo"],
                                  " ".join("%s=%.4f" % kv for kv in sorted(p["timings"].items()))))
        log("      %s" % p["describe"])
    # Graph capture needs a stream other than the default one; eager runs use
    # the same stream so both modes launch identically.
    stream = torch.cuda.Stream(dev) if args.graph else torch.cuda.current_stream(dev)
    torch.cuda.set_stream(stream)
    step = make_step(plan, ws, stream.cuda_stream)

    def timed(step_fn):
        """Warm-up, optional graph capture, then K timed steps bracketed by
        device synchronisation; per-layer HIP events on the launch stream."""
        for _ in range(args.warmup):
            step_fn()
        torch.cuda.synchronize()
        graph = None
        if args.graph:
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph, stream=stream):
                step_fn()
            torch.cuda.synchronize()
            for _ in range(args.warmup):
                graph.replay()
            torch.cuda.synchronize()
        nl = len(plan)
        ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(nl)]
              for _ in range(args.steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        if graph is not None:
            for _ in range(args.steps):
                graph.replay()
        else:
            for k in range(args.steps):
                step_fn(ev[k])
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        ms = (t1 - t0) * 1e3 / args.steps
        if graph is None:
            lms = [sum(ev[k][i][0].elapsed_time(ev[k][i][1]) for k in range(args.steps)) / args.steps
                   for i in range(nl)]
        else:
            # graph replay: per-layer times from eager steps with events
            evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(nl)]
            lms = [0.0] * nl
            for _ in range(args.steps):
                step_fn(evs)
                torch.cuda.synchronize()
                for i in range(nl):
                    lms[i] += evs[i][0].elapsed_time(evs[i][1]) / args.steps
        return ms, lms

    step_pk = make_step(plan, ws, stream.cuda_stream, prepacked=True)
    ms_unpk, lms_unpk = timed(step)
    ms_pk, lms_pk = timed(step_pk)
    if args.prepacked:
        ms_per_step, layer_ms, ms_other = ms_pk, lms_pk, ms_unpk
    else:
        ms_per_step, layer_ms, ms_other = ms_unpk, lms_unpk, ms_pk

    total_flops = sum(p["layer"].flops for p in plan)
    value = total_flops / (ms_per_step * 1e-3) / 1e12

    dtype = plan[0]["layer"].dtype
    by_algo = {}
    for p, ms in zip(plan, layer_ms):
        a = by_algo.setdefault(p["algo"], [0.0, 0, 0])
        a[0] += ms
        a[1] += p["layer"].flops
        a[2] += 1

    # Roofline of the dominant kernel: the main-kernel instantiation with the
    # largest share of the step.  Measured on the prepacked step, counting the
    # layers where that kernel is the call's only launch (no split-K reduce),
    # so each HIP-event interval around a call times exactly one launch.
    def main_kernel(desc):
        ks = desc.split("kernels=")[1].split(" ")[0].split(";")
        return [k for k in ks if not k.startswith("pack_filters") and not k.startswith("wino_filter")]
    share = {}
    for p, ms in zip(plan, lms_pk):
        ks = main_kernel(p["describe"])
        if len(ks) == 1:
            share[ks[0]] = share.get(ks[0], 0.0) + ms
    dom = max(share, key=share.get)
    single = [(p, ms) for p, ms in zip(plan, lms_pk) if main_kernel(p["describe"]) == [dom]]
    dom_ms = sum(ms for _, ms in single)
    dom_flops = sum(p["layer"].flops for p, _ in single)
    achieved = dom_flops / (dom_ms * 1e-3) / 1e12 if dom_ms > 0 else 0.0
    peak = PEAKS_TFLOPS[dtype]
    roofline = {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s", "frac": achieved / peak,
                "traffic": None, "kernel": dom, "launches_per_step": len(single),
                "avg_launch_us": dom_ms * 1e3 / max(len(single), 1),
                "time_share_prepacked_step": share[dom] / sum(lms_pk)}

    # The 3x3 layers of the workload (the headline target for ResNet-50).
    sel = [(p, ms) for p, ms in zip(plan, layer_ms) if p["layer"].r == 3]
    extra = {}
    if sel:
        f3 = sum(p["layer"].flops for p, _ in sel)
        t3 = sum(ms for _, ms in sel)
        extra["layers_3x3"] = {"count": len(sel), "gflop": f3 / 1e9, "ms": t3,
                               "tflops": f3 / (t3 * 1e-3) / 1e12, "frac_peak": f3 / (t3 * 1e-3) / 1e12 / peak}
    extra["sum_layer_event_ms"] = sum(layer_ms)
    extra["algos"] = {a: v[2] for a, v in by_algo.items()}
    other = "per_call_filter_packing" if args.prepacked else "prepacked_filters"
    extra[other] = {"ms_per_step": ms_other, "tflops": total_flops / (ms_other * 1e-3) / 1e12}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, args.cpu_budget)

    nbatch = layers[0].n
    out = {"metric": "conv2d TFLOP/s (2*N*K*C/G*R*S*P*Q per layer), best measured algorithm per layer",
           "value": value, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": dtype, "data": "synthetic (seeded normal inputs, Kaiming-normal weights)",
           "config": {"workload": "%s conv layers (%d convs), batch %d, %s data, fp32 accumulate, %s, %s"
                                  % (wl, len(layers), nbatch, dtype, "graph replay" if args.graph else "eager launches",
                                     "prepacked filters" if args.prepacked else "filters packed every call"),
                      "global_batch": nbatch, "layers": len(layers), "parallelism": "none (1 GPU)"},
           "roofline": roofline, "cpu_baseline": cpu, "detail": extra}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
