#!/usr/bin/env python3
"""Measured report of the five workloads (test infrastructure: it uses the
CPU oracle).  Run on one MI355X:

    python tests/report.py OUTDIR [--workloads toy,vgg16,...] [--no-networks]

Writes
  OUTDIR/layers.jsonl    one row per (workload, unique layer, algorithm):
                         status (or "n/a" when the algorithm does not apply),
                         max relative error against the fp64 oracle on the
                         same inputs, tolerance, pass, call time (HIP events
                         around a graph of back-to-back calls), TFLOP/s and
                         fraction of the dtype's MFMA peak, compulsory GB/s
                         and fraction of HBM peak, the roofline that bounds
                         the layer, and the oracle's wall time for the layer
                         on the host's cores;
  OUTDIR/networks.jsonl  whole networks timed as one HIP graph per forward:
                         the VGG-16 chain (convolutions, ReLU, 2x2 max-pools)
                         through the model executor, and the ResNet-50 and
                         random 20-layer convolution chains, each with the
                         per-layer fastest algorithm and with every single
                         algorithm that runs all of its layers;
  OUTDIR/oracle_single_thread.json  the oracle on one thread (toy layer and
                         one ResNet-50 layer at batch 1);
  OUTDIR/summary.md      the tables built from those rows.

Inputs follow the parity tests' recipe (workloads.make_tensors).  The random
20-layer chain (N = 128) is checked on whole output planes of 8 of its
images (the first, the last and six seeded ones), and its oracle time is
that of those 8 images, reported with the extrapolation to 128.
"""
import argparse
import json
import os
import subprocess
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, ROOT)
sys.path.insert(0, HERE)

PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
HBM_GBS = 8000.0
RIDGE = {k: v * 1e12 / (HBM_GBS * 1e9) for k, v in PEAK_TFLOPS.items()}   # FLOP per byte


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def subset_images(L):
    import numpy as np
    from paper_2410_08300_amd import workloads as W
    if L.n <= 32:
        return None
    rng = np.random.default_rng(W.seed_for(77, L.n))
    mid = rng.choice(np.arange(1, L.n - 1), size=6, replace=False)
    return np.sort(np.concatenate([[0, L.n - 1], mid]))


def time_call(x, w, b, L, algo, target_ms=25.0):
    """ms per call: graph replays of back-to-back calls, as many as fit the
    target, median of 5."""
    import paper_2410_08300_amd as cs
    once = cs.time_conv(x, w, b, L.stride, L.pad, L.dilation, L.groups, algo, L.relu, warmup=1, reps=1,
                        launches=1)
    launches = int(max(1, min(40, target_ms / max(once, 1e-3))))
    return cs.time_conv(x, w, b, L.stride, L.pad, L.dilation, L.groups, algo, L.relu, warmup=2, reps=5,
                        launches=launches)


def layer_rows(wl, dev):
    import torch
    import oracle
    import paper_2410_08300_amd as cs
    from paper_2410_08300_amd import workloads as W
    from gpu_util import ALGOS, tolerance, f64

    rows = []
    for li, (L, count) in enumerate(W.unique_layers(W.layers(wl))):
        x, w, b = W.make_tensors(L, (W.WORKLOADS.index(wl), li, 2), device=dev)
        imgs = subset_images(L)
        xs = x if imgs is None else x[torch.as_tensor(imgs, device=dev)]
        t0 = time.perf_counter()
        ref = oracle.conv2d(f64(xs), f64(w), f64(b), L.stride, L.pad, L.dilation, L.groups, L.relu)
        oracle_s = time.perf_counter() - t0
        ref_dev = torch.from_numpy(ref).to(dev)
        del ref
        scale = float(ref_dev.abs().max())
        sel = None if imgs is None else torch.as_tensor(imgs, device=dev)
        supported = cs.supported_algos(x, w, b, L.stride, L.pad, L.dilation, L.groups, L.relu)
        ai = L.flops / L.compulsory_bytes()
        bound = "mfma" if ai >= RIDGE[L.dtype] else "hbm"
        for algo in ALGOS:
            row = dict(workload=wl, layer=L.name, count=count, shape=L.asdict(), algo=algo,
                       flops=L.flops, bytes=L.compulsory_bytes(), intensity=ai, bound=bound,
                       oracle_s=oracle_s, oracle_images=L.n if imgs is None else len(imgs),
                       oracle_s_full_batch=oracle_s * (1 if imgs is None else L.n / len(imgs)),
                       checked_images="all" if imgs is None else [int(i) for i in imgs])
            if algo not in supported:
                row.update(status="n/a")
                rows.append(row)
                continue
            y = cs.conv2d(x, w, b, L.stride, L.pad, L.dilation, L.groups, algo=algo, relu=L.relu)
            ys = y if sel is None else y[sel]
            diff = float((ys.double() - ref_dev).abs().max())
            err = diff / scale if scale > 0 else diff
            del y, ys
            ms = time_call(x, w, b, L, algo)
            tf = L.flops / (ms * 1e-3) / 1e12
            gbs = L.compulsory_bytes() / (ms * 1e-3) / 1e9
            tol = tolerance(L.dtype, algo)
            row.update(status="ok", err=err, tol=tol, passed=bool(err <= tol), ms=ms, tflops=tf,
                       frac_mfma_peak=tf / PEAK_TFLOPS[L.dtype], gbs=gbs, frac_hbm=gbs / HBM_GBS,
                       frac_roof=(tf / PEAK_TFLOPS[L.dtype]) if bound == "mfma" else gbs / HBM_GBS)
            rows.append(row)
            log("%-12s %-20s %-22s err %.2e  %9.4f ms %8.1f TFLOP/s %7.1f GB/s" %
                (wl, L.name, algo, err, ms, tf, gbs))
        del x, w, b, xs, ref_dev
        torch.cuda.empty_cache()
    return rows


def graph_ms(fn, steps, warmup, stream):
    import torch
    fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        fn()
    torch.cuda.synchronize()
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        g.replay()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / steps


def chain_networks(wl, best, dev):
    """The workload's convolutions as one graph step per table: the per-layer
    fastest algorithm, then every algorithm that runs all layers."""
    import torch
    import bench
    import paper_2410_08300_amd as cs
    from paper_2410_08300_amd import workloads as W

    layers = W.layers(wl)
    out = []
    stream = torch.cuda.Stream(dev)
    tables = [("per-layer fastest", {L.name: best[(wl, L.shape_key())] for L in layers})]
    for algo in cs.CONCRETE_ALGOS:
        tables.append((algo, {L.name: algo for L in layers}))
    for name, table in tables:
        unsupported = [L.name for L in layers if table[L.name] not in best.get(("supported", wl, L.shape_key()), ())]
        if unsupported:
            out.append(dict(network=wl, table=name, status="n/a",
                            reason="%d layers not supported (e.g. %s)" % (len(unsupported), unsupported[0])))
            continue
        with torch.cuda.stream(stream):
            plan, ws = bench.build_plan(layers, W.WORKLOADS.index(wl), dev, None, table=table)
            torch.cuda.synchronize()
            step = bench.make_step(plan, ws, stream.cuda_stream)
            slow = name in ("direct", "smm", "kn2row", "im2col_gemm", "implicit_precomp_gemm")
            ms = graph_ms(step, 3 if slow else 20, 1 if slow else 3, stream)
        flops = sum(L.flops for L in layers)
        out.append(dict(network=wl, table=name, status="ok", ms=ms, tflops=flops / (ms * 1e-3) / 1e12,
                        layers=len(layers), what="%d convolutions of %s, one HIP graph per step, filters packed "
                                                 "every call" % (len(layers), wl)))
        log("network %-10s %-20s %10.3f ms" % (wl, name, ms))
        del plan, ws, step
        torch.cuda.empty_cache()
    return out


def vgg_networks(best, dev):
    """VGG-16's 13 convolutions with ReLU after each and a 2x2 max-pool
    between blocks, N = 8, fp32, through the model executor."""
    import torch
    from torch import nn
    import paper_2410_08300_amd as cs
    from paper_2410_08300_amd import workloads as W

    layers = W.layers("vgg16")
    mods, names = [], []
    prev_h = layers[0].h
    for L in layers:
        if L.h != prev_h:
            mods.append(nn.MaxPool2d(2, 2))
            prev_h = L.h
        names.append(str(len(mods)))
        mods.append(nn.Conv2d(L.c, L.k, 3, padding=1))
        mods.append(nn.ReLU())
    net = nn.Sequential(*mods).eval().to(dev)
    x = torch.randn(layers[0].n, 3, 224, 224, generator=torch.Generator(device=dev).manual_seed(16), device=dev)
    flops = sum(L.flops for L in layers)
    out = []
    tables = [("per-layer fastest", {n: best[("vgg16", L.shape_key())] for n, L in zip(names, layers)})]
    for algo in cs.CONCRETE_ALGOS:
        tables.append((algo, {n: algo for n in names}))
    stream = torch.cuda.Stream(dev)
    for name, table in tables:
        model = cs.swap_backend(net, table)
        with torch.no_grad(), torch.cuda.stream(stream):
            slow = name in ("direct", "smm", "kn2row")
            ms = graph_ms(lambda: model(x), 3 if slow else 10, 1 if slow else 2, stream)
        out.append(dict(network="vgg16", table=name, status="ok", ms=ms, tflops=flops / (ms * 1e-3) / 1e12,
                        what="VGG-16 feature extractor (13 convolutions with bias and ReLU, four 2x2 max-pools) "
                             "at N = 8, fp32, through swap_backend, one HIP graph per forward"))
        log("network vgg16      %-20s %10.3f ms" % (name, ms))
        del model
        torch.cuda.empty_cache()
    return out


def single_thread_oracle():
    """The oracle on one thread, in a child process with OMP_NUM_THREADS=1."""
    code = r'''
import json, sys, time
sys.path.insert(0, %r)
import numpy as np
import oracle
from paper_2410_08300_amd import workloads as W
out = []
for wl, name in (("toy", "conv1"), ("resnet50", "layer3.1.conv2")):
    L = [l for l in W.layers(wl, n=1) if l.name == name][0]
    rng = np.random.default_rng(0)
    x = rng.standard_normal((L.n, L.c, L.h, L.w)); w = rng.standard_normal((L.k, L.c // L.groups, L.r, L.s))
    t0 = time.perf_counter(); oracle.conv2d(x, w, None, L.stride, L.pad, L.dilation, L.groups, False)
    s = time.perf_counter() - t0
    out.append(dict(workload=wl, layer=name, batch=1, seconds=s, gflops=L.flops / s / 1e9, threads=1))
print(json.dumps(out))
''' % ROOT
    env = dict(os.environ, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, timeout=600)
    if r.returncode != 0:
        raise RuntimeError(r.stderr)
    return json.loads(r.stdout.strip().splitlines()[-1])


def summary(rows, nets, st):
    lines = []
    by_wl = {}
    for r in rows:
        by_wl.setdefault(r["workload"], []).append(r)
    lines.append("| workload | layer (x count) | best algorithm | ms | TFLOP/s | % of its roof (bound) | "
                 "max err of all algorithms (tol) | all pass | oracle s |")
    lines.append("|---|---|---|---:|---:|---:|---|---|---:|")
    for wl, rs in by_wl.items():
        layers = []
        for r in rs:
            if r["layer"] not in layers:
                layers.append(r["layer"])
        for name in layers:
            lr = [r for r in rs if r["layer"] == name and r["status"] == "ok"]
            b = min(lr, key=lambda r: r["ms"])
            emax = max(r["err"] / r["tol"] for r in lr)
            lines.append("| %s | %s (x%d) | %s | %.4f | %.1f | %.1f%% (%s) | %.2f of tol | %s | %.2f |" % (
                wl, name, b["count"], b["algo"], b["ms"], b["tflops"], 100 * b["frac_roof"], b["bound"], emax,
                "yes" if all(r["passed"] for r in lr) else "NO", b["oracle_s_full_batch"]))
    lines.append("")
    lines.append("| network | table | ms | TFLOP/s |")
    lines.append("|---|---|---:|---:|")
    for n in nets:
        if n["status"] == "ok":
            lines.append("| %s | %s | %.3f | %.1f |" % (n["network"], n["table"], n["ms"], n["tflops"]))
        else:
            lines.append("| %s | %s | n/a | %s |" % (n["network"], n["table"], n["reason"]))
    lines.append("")
    for s in st:
        lines.append("oracle, one thread: %s %s at batch 1: %.3f ms (%.2f GFLOP/s)" %
                     (s["workload"], s["layer"], s["seconds"] * 1e3, s["gflops"]))
    return "\n".join(lines) + "\n"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("outdir")
    ap.add_argument("--workloads", default="toy,vgg16,resnet50,mobilenetv2,random20")
    ap.add_argument("--no-networks", action="store_true")
    args = ap.parse_args()
    import torch
    from paper_2410_08300_amd import _lib
    _lib.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    os.makedirs(args.outdir, exist_ok=True)
    rows = []
    with open(os.path.join(args.outdir, "layers.jsonl"), "w") as f:
        for wl in args.workloads.split(","):
            for r in layer_rows(wl, dev):
                rows.append(r)
                f.write(json.dumps(r) + "\n")
    from paper_2410_08300_amd import workloads as W
    best = {}
    for r in rows:
        if r["status"] != "ok":
            continue
        shapes = {L.name: L.shape_key() for L in W.layers(r["workload"])}
        key = (r["workload"], shapes[r["layer"]])
        best.setdefault(("supported",) + key, set()).add(r["algo"])
        if key not in best or r["ms"] < best[("ms",) + key]:
            best[key] = r["algo"]
            best[("ms",) + key] = r["ms"]
    for (k, v) in list(best.items()):
        if k[0] == "supported":
            best[k] = tuple(sorted(v))
    nets = []
    if not args.no_networks:
        wls = args.workloads.split(",")
        if "vgg16" in wls:
            nets += vgg_networks(best, dev)
        for wl in ("resnet50", "random20"):
            if wl in wls:
                nets += chain_networks(wl, best, dev)
    with open(os.path.join(args.outdir, "networks.jsonl"), "w") as f:
        for n in nets:
            f.write(json.dumps(n) + "\n")
    st = single_thread_oracle()
    with open(os.path.join(args.outdir, "oracle_single_thread.json"), "w") as f:
        json.dump({"threads": 1, "host_cores": os.cpu_count(), "rows": st}, f, indent=1)
    with open(os.path.join(args.outdir, "summary.md"), "w") as f:
        f.write(summary(rows, nets, st))
    log("report written to %s" % args.outdir)


if __name__ == "__main__":
    main()
