#!/usr/bin/env python3
"""Benchmark of the convolution hot path on one MI355X.

A step is one forward pass over every convolution layer of a workload (by
default the 53 convolutions of ResNet-50 at batch 32, bf16 data, fp32
accumulation), each layer running the algorithm chosen for it by measured
per-layer selection (every supported algorithm timed on that layer before
the timed region; the fastest goes into the algorithm table) or taken from a
saved table.  Inputs, weights and outputs are resident in HBM before timing
starts.  Each layer's filter package (the tile-ordered filter copy some
kernels read) is built once before timing, as a framework-managed model
(swap_backend) holds it, and the step calls conv2d_prepacked; with
--pack-per-call the step calls the plain conv2d(), which rebuilds or
regroups the filters in every call.

The headline replays the step as one captured HIP graph (--eager: plain
launches); all four step variants are reported.  Per-layer call durations
come from HIP events around graph replays of back-to-back calls of that
layer; the roofline of the dominant kernel is computed from them.  The CPU
oracle is timed on a bounded sample on the host.

Prints one JSON line (TFLOP/s, 2*N*K*(C/G)*R*S*P*Q per layer).

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload resnet50]
                    [--select measured|default|<algo>] [--eager] [--pack-per-call]
                    [--table FILE] [--save-table FILE] [--sweep FILE]
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


def build_plan(layers, wl_index, device, select, algos_allowed=None, table=None):
    """Resident tensors, descriptors and the chosen algorithm of every layer
    (from ``table``, a {layer name: algorithm} map, when given)."""
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
        if table is not None:
            cache[key] = (table[L.name], {})
        elif key not in cache:
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

    def one(i, args):
        def call():
            st = fn(*args)
            if st:
                raise _lib.Conv2dError(st, "layer %d" % i)
        return call

    def step():
        for i, args in enumerate(calls):
            st = fn(*args)
            if st:
                raise _lib.Conv2dError(st, "layer %d" % i)
    step.calls = [one(i, a) for i, a in enumerate(calls)]
    return step


# Source files of each main kernel (the HBM traffic recorded for a kernel
# under profiles/ is used only while these files are unchanged).
KERNEL_SOURCES = {
    "implicit_gemm_kernel": ("implicit_gemm.hip", "igemm_common.hpp"),
    "pointwise_": ("implicit_gemm.hip", "igemm_common.hpp"),
    "repack_plane_kernel": ("implicit_gemm.hip", "igemm_common.hpp"),
    "repack_s2_rows_kernel": ("implicit_gemm.hip", "igemm_common.hpp"),
    "splitk_reduce_kernel": ("igemm_common.hpp",),
    "implicit_rows_kernel": ("implicit_rows.hip", "igemm_common.hpp"),
    "conv3x3_kernel": ("conv3x3.hip", "igemm_common.hpp"),
    "implicit_ws_kernel": ("implicit_ws.hip", "igemm_common.hpp"),
    "gemm_nt_kernel": ("gemm.hip",),
    "direct_": ("direct.hip",),
    "wino_": ("winograd.hip", "gemm.hip"),
    "im2col_kernel": ("im2col.hip",),
}


def source_digest(kernel):
    import hashlib
    files = None
    for prefix, fs in KERNEL_SOURCES.items():
        if kernel.startswith(prefix):
            files = fs + ("common.hpp", "kernels.hpp")
    if files is None:
        return None
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2410_08300_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def recorded_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` on `workload` from the table in
    profiles/traffic.md (FETCH_SIZE + WRITE_SIZE counters, calibrated against
    a copy kernel), or None when absent or recorded for other sources."""
    path = os.path.join(ROOT, "profiles", "traffic.md")
    if not os.path.exists(path):
        return None
    digest = source_digest(kernel)
    with open(path) as f:
        for line in f:
            cells = [c.strip() for c in line.strip().strip("|").split("|")]
            if len(cells) >= 6 and cells[0] == "`%s`" % kernel and cells[1] == workload and cells[5] == digest:
                try:
                    return {"fetch_bytes": float(cells[2]), "write_bytes": float(cells[3]),
                            "bytes": float(cells[2]) + float(cells[3]), "source_digest": digest}
                except ValueError:
                    return None
    return None


def calibration_copy(mib, device):
    """One plain copy of `mib` MiB through the library (the filter package of
    the direct algorithm is a byte copy), for scaling the HBM byte counters."""
    import torch
    import paper_2410_08300_amd as cs
    kc = mib * (1 << 20) // (2 * 1024)
    w = torch.zeros((kc, 1024, 1, 1), dtype=torch.bfloat16, device=device)
    torch.cuda.synchronize()
    cs.pack_filters(w, (1, 1024, 1, 1), algo="direct")
    torch.cuda.synchronize()
    log("calibration copy: %d bytes read, %d bytes written" % (w.numel() * 2, w.numel() * 2))


def measured_peaks(device):
    """What this machine delivers, beside the nominal peaks: the MFMA rate of a
    register-only probe (bf16 and fp32) and the HBM rate of a plain 16-byte
    copy of 1 GiB (bytes read plus bytes written per second), each the best of
    five timed launches after one warm-up."""
    import torch
    from paper_2410_08300_amd import _lib
    stream = torch.cuda.current_stream(device)
    out = {}
    blocks, iters = 1024, 2000
    sink = torch.empty(blocks * 256, dtype=torch.float32, device=device)
    for dt, flops_per in (("bf16", 32768), ("f32", 4096)):
        its = iters if dt == "bf16" else iters // 4
        best = None
        for rep in range(6):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            _lib.probe_mfma(dt, blocks, its, sink.data_ptr(), stream.cuda_stream)
            e1.record(stream)
            e1.synchronize()
            ms = e0.elapsed_time(e1)
            if rep and (best is None or ms < best):
                best = ms
        tf = blocks * 4 * its * 8 * flops_per / (best * 1e-3) / 1e12
        out["mfma_%s_tflops" % dt] = {"measured": tf, "nominal": PEAKS_TFLOPS[dt], "frac_of_nominal": tf / PEAKS_TFLOPS[dt]}
    nbytes = 1 << 30
    src = torch.empty(nbytes // 4, dtype=torch.float32, device=device)
    src.fill_(1.0)
    dst = torch.empty_like(src)
    best = None
    for rep in range(6):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        _lib.probe_copy(src.data_ptr(), dst.data_ptr(), nbytes, stream.cuda_stream)
        e1.record(stream)
        e1.synchronize()
        ms = e0.elapsed_time(e1)
        if rep and (best is None or ms < best):
            best = ms
    gbs = 2 * nbytes / (best * 1e-3) / 1e9
    out["hbm_copy_gbs"] = {"measured": gbs, "nominal": HBM_GBS, "frac_of_nominal": gbs / HBM_GBS}
    del src, dst, sink
    torch.cuda.empty_cache()
    return out


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
    while images == 0 or (t_total < budget_s and images < 256):
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


def resnet50_module(classes=1000):
    """ResNet-50 v1.5 as an nn.Module whose convolutions carry the layer names
    of ``workloads.resnet50`` (stem, layerS.B.conv1/2/3, layerS.B.downsample),
    with batch norm after every convolution, the 3x3/2 max-pool, residual
    adds, global average pooling and the 2048 -> 1000 linear head."""
    import torch
    from torch import nn

    class Bottleneck(nn.Module):
        def __init__(self, cin, width, stride):
            super().__init__()
            cout = 4 * width
            self.conv1, self.bn1 = nn.Conv2d(cin, width, 1, bias=False), nn.BatchNorm2d(width)
            self.conv2, self.bn2 = nn.Conv2d(width, width, 3, stride, 1, bias=False), nn.BatchNorm2d(width)
            self.conv3, self.bn3 = nn.Conv2d(width, cout, 1, bias=False), nn.BatchNorm2d(cout)
            self.downsample = None
            if stride != 1 or cin != cout:
                self.downsample = nn.Conv2d(cin, cout, 1, stride, bias=False)
                self.down_bn = nn.BatchNorm2d(cout)
            self.relu = nn.ReLU(inplace=True)

        def forward(self, x):
            out = self.relu(self.bn1(self.conv1(x)))
            out = self.relu(self.bn2(self.conv2(out)))
            out = self.bn3(self.conv3(out))
            idt = x if self.downsample is None else self.down_bn(self.downsample(x))
            out += idt
            return self.relu(out)

    class ResNet50(nn.Module):
        def __init__(self):
            super().__init__()
            self.stem, self.bn = nn.Conv2d(3, 64, 7, 2, 3, bias=False), nn.BatchNorm2d(64)
            self.relu = nn.ReLU(inplace=True)
            self.maxpool = nn.MaxPool2d(3, 2, 1)
            cin = 64
            for si, (width, blocks) in enumerate([(64, 3), (128, 4), (256, 6), (512, 3)]):
                layer = []
                for bi in range(blocks):
                    layer.append(Bottleneck(cin, width, 2 if (bi == 0 and si > 0) else 1))
                    cin = 4 * width
                setattr(self, "layer%d" % (si + 1), nn.Sequential(*layer))
            self.avgpool = nn.AdaptiveAvgPool2d((1, 1))
            self.fc = nn.Linear(2048, classes)

        def forward(self, x):
            x = self.maxpool(self.relu(self.bn(self.stem(x))))
            x = self.layer4(self.layer3(self.layer2(self.layer1(x))))
            return self.fc(torch.flatten(self.avgpool(x), 1))

    net = ResNet50()
    g = torch.Generator().manual_seed(50)
    for m in net.modules():
        if isinstance(m, nn.BatchNorm2d):
            c = m.num_features
            m.running_mean.copy_(torch.randn(c, generator=g) * 0.1)
            m.running_var.copy_(torch.rand(c, generator=g) + 0.5)
            m.weight.data.copy_(torch.rand(c, generator=g) + 0.5)
            m.bias.data.copy_(torch.randn(c, generator=g) * 0.1)
    return net.eval()


def executor_forward(plan, steps, warmup):
    """The whole ResNet-50 network (convolutions with the plan's algorithms,
    folded batch norm, pooling, residual adds, the linear head) through
    swap_backend, one HIP graph per forward: ms per forward."""
    import torch
    import paper_2410_08300_amd as cs

    dev = plan[0]["x"].device
    net = resnet50_module().to(torch.bfloat16).to(dev)
    model = cs.swap_backend(net, {p["layer"].name: p["algo"] for p in plan})
    x = plan[0]["x"]
    with torch.no_grad():
        model(x)
        s = torch.cuda.Stream(dev)
        s.wait_stream(torch.cuda.current_stream(dev))
        g = torch.cuda.CUDAGraph()
        with torch.cuda.stream(s):
            model(x)
            s.synchronize()
            with torch.cuda.graph(g, stream=s):
                model(x)
        torch.cuda.synchronize()
        for _ in range(warmup):
            g.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            g.replay()
        torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    return {"ms_per_forward": ms, "ops": len(model.ops),
            "what": "ResNet-50 v1.5 inference forward (53 convolutions with the step's algorithms, folded batch "
                    "norm, max-pool, 16 residual adds, global average pool, 2048x1000 linear) through swap_backend, "
                    "one HIP graph per forward"}


def sweep(path, steps, fit_seeds=0):
    """Every algorithm on every unique layer of all five workloads (or, with
    fit_seeds = S > 0, of the fitting set: the 20-layer random chain at seeds
    1..S and the mixed independent layers at seeds 0..S-1): JSONL rows."""
    import torch
    import paper_2410_08300_amd as cs
    from paper_2410_08300_amd import workloads as W

    dev = torch.device("cuda:0")
    if fit_seeds > 0:
        sets = [("random20/s%d" % sd, W.random20(128, sd)) for sd in range(1, fit_seeds + 1)]
        sets += [("mixed/s%d" % sd, W.mixed(sd)) for sd in range(fit_seeds)]
    else:
        sets = [(wl, W.layers(wl)) for wl in W.WORKLOADS]
    with open(path, "w") as f:
        for wi, (wl, wl_layers) in enumerate(sets):
            for li, (L, count) in enumerate(W.unique_layers(wl_layers)):
                x, w, b = W.make_tensors(L, (wi + (100 if fit_seeds else 0), li, 4), device=dev)
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
    ap.add_argument("--eager", action="store_true",
                    help="headline from eager launches (default: the step captured once as a HIP graph and replayed)")
    ap.add_argument("--pack-per-call", action="store_true",
                    help="headline from plain conv2d calls, every call rebuilding its filter package from the "
                         "filters; by default each layer's package is built once before timing, as a "
                         "framework-managed model (swap_backend) holds it, and the step calls conv2d_prepacked")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-executor", action="store_true",
                    help="skip the whole-network swap_backend forward (ResNet-50 only)")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--sweep", default=None, help="write per-layer, per-algorithm timings to this JSONL file")
    ap.add_argument("--sweep-fit-seeds", type=int, default=0, metavar="S",
                    help="with --sweep: time the algorithm-choice fitting set (random chains at seeds 1..S, "
                         "mixed layers at seeds 0..S-1) instead of the five workloads")
    ap.add_argument("--table", default=None,
                    help="JSON {layer name: algorithm} to use instead of measuring (e.g. a saved --save-table)")
    ap.add_argument("--save-table", default=None, help="write the per-layer algorithm table to this JSON file")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="after timing, run one plain copy of MIB MiB (reference for HBM byte counters)")
    args = ap.parse_args()

    if args.gpus != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              "(the convolution shards over the batch with no exchange step)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2410_08300_amd import _lib, workloads as W

    _lib.lib()   # fail loudly if the HIP library is missing
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    if args.sweep:
        sweep(args.sweep, max(args.steps, 3), args.sweep_fit_seeds)
        return

    wl = args.workload
    layers = W.layers(wl)
    log("bench: workload %s, %d layers, select=%s" % (wl, len(layers), args.select))
    table = None
    if args.table:
        with open(args.table) as f:
            table = json.load(f)["algorithms"]
    plan, ws = build_plan(layers, W.WORKLOADS.index(wl), dev, args.select, table=table)
    if args.save_table:
        with open(args.save_table, "w") as f:
            json.dump({"workload": wl, "batch": layers[0].n, "dtype": layers[0].dtype,
                       "selection": "table" if table else args.select,
                       "algorithms": {p["layer"].name: p["algo"] for p in plan},
                       "timings_ms": {p["layer"].name: p["timings"] for p in plan}}, f, indent=1)
    torch.cuda.synchronize()  # filter packages were built on the default stream
    for p in plan:
        L = p["layer"]
        log("  %-24s %-14s %s" % (L.name, p["algo"],
                                  " ".join("%s=%.4f" % kv for kv in sorted(p["timings"].items()))))
        log("      %s" % p["describe"])
    # All launches go to one side stream (graph capture needs a stream other
    # than the default one), eager or replayed.
    stream = torch.cuda.Stream(dev)
    torch.cuda.set_stream(stream)
    step = make_step(plan, ws, stream.cuda_stream)
    step_pk = make_step(plan, ws, stream.cuda_stream, prepacked=True)

    def timed_steps(step_fn, graph):
        """W warm-up steps, then exactly K timed steps bracketed by device
        synchronisation; with graph=True one step is captured as a HIP graph
        and the K steps are K replays."""
        g = None
        if graph:
            step_fn()
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=stream):
                step_fn()
            torch.cuda.synchronize()
        for _ in range(args.warmup):
            g.replay() if g is not None else step_fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            g.replay() if g is not None else step_fn()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3 / args.steps

    def layer_times(prepacked, launches=40, reps=3):
        """Per-layer duration of one call: `launches` back-to-back calls of
        the layer captured as a HIP graph, replayed between two HIP events on
        the launch stream (median of `reps`, divided by `launches`), so host
        launch overhead and event latency stay out of the figure."""
        calls = make_step(plan, ws, stream.cuda_stream, prepacked=prepacked).calls
        out = []
        for call in calls:
            g = torch.cuda.CUDAGraph()
            call()
            torch.cuda.synchronize()
            with torch.cuda.graph(g, stream=stream):
                for _ in range(launches):
                    call()
            g.replay()
            torch.cuda.synchronize()
            ts = []
            for _ in range(reps):
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                g.replay()
                e1.record(stream)
                e1.synchronize()
                ts.append(e0.elapsed_time(e1) / launches)
            out.append(sorted(ts)[len(ts) // 2])
            del g
        return out

    modes = {"graph": timed_steps(step, True), "graph_prepacked": timed_steps(step_pk, True),
             "eager": timed_steps(step, False), "eager_prepacked": timed_steps(step_pk, False)}
    prepacked = not args.pack_per_call
    head = ("eager" if args.eager else "graph") + ("_prepacked" if prepacked else "")
    ms_per_step = modes[head]
    lms_unpk = layer_times(False)
    lms_pk = layer_times(True)
    layer_ms = lms_pk if prepacked else lms_unpk

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
    # largest share of the prepacked per-layer times, counting the layers
    # where that kernel is the call's only launch (no split-K reduce), so each
    # timed call is exactly one launch of it.
    def main_kernel(desc):
        ks = desc.split("kernels=")[1].split(" ")[0].split(";")
        return [k for k in ks if not k.startswith(("pack_filters", "wino_filter", "rows_pack"))]
    share = {}
    for p, ms in zip(plan, lms_pk):
        ks = main_kernel(p["describe"])
        if len(ks) == 1:
            share[ks[0]] = share.get(ks[0], 0.0) + ms
    if share:
        dom = max(share, key=share.get)
        single = [(p, ms) for p, ms in zip(plan, lms_pk) if main_kernel(p["describe"]) == [dom]]
    else:
        # No layer runs a single main kernel (every call launches several,
        # e.g. Winograd's transforms and products): price whole calls of the
        # algorithm with the largest share instead.
        for p, ms in zip(plan, lms_pk):
            share[p["algo"] + " (whole call)"] = share.get(p["algo"] + " (whole call)", 0.0) + ms
        dom = max(share, key=share.get)
        single = [(p, ms) for p, ms in zip(plan, lms_pk) if p["algo"] + " (whole call)" == dom]
    dom_ms = sum(ms for _, ms in single)
    dom_flops = sum(p["layer"].flops for p, _ in single)
    dom_bytes = sum(p["layer"].compulsory_bytes() for p, _ in single)
    peak = PEAKS_TFLOPS[dtype]
    # The kernel's roofline is the one its launches reach first: MFMA when the
    # flops take longer at peak than the compulsory bytes at HBM peak, else HBM.
    if dom_bytes / (HBM_GBS * 1e9) > dom_flops / (peak * 1e12):
        bound, unit, peak_b = "hbm", "GB/s", HBM_GBS
        achieved = dom_bytes / (dom_ms * 1e-3) / 1e9 if dom_ms > 0 else 0.0
    else:
        bound, unit, peak_b = "mfma", "TFLOP/s", peak
        achieved = dom_flops / (dom_ms * 1e-3) / 1e12 if dom_ms > 0 else 0.0
    wl_name = "%s-n%d-%s" % (wl, layers[0].n, layers[0].dtype)
    traffic = recorded_traffic(dom, wl_name)
    roofline = {"bound": bound, "achieved": achieved, "peak": peak_b, "unit": unit, "frac": achieved / peak_b,
                "algorithmic_bytes_per_launch": dom_bytes / max(len(single), 1),
                "algorithmic_flops_per_launch": dom_flops / max(len(single), 1),
                "tflops": dom_flops / (dom_ms * 1e-3) / 1e12 if dom_ms > 0 else 0.0,
                "traffic": traffic["bytes"] if traffic else None, "traffic_detail": traffic,
                "kernel": dom, "launches_per_step": len(single),
                "avg_launch_us": dom_ms * 1e3 / max(len(single), 1),
                "time_share_prepacked": share[dom] / sum(lms_pk)}

    # The 3x3 layers of the workload (the headline target for ResNet-50).
    sel = [(p, ms) for p, ms in zip(plan, layer_ms) if p["layer"].r == 3]
    extra = {}
    if sel:
        f3 = sum(p["layer"].flops for p, _ in sel)
        t3 = sum(ms for _, ms in sel)
        extra["layers_3x3"] = {"count": len(sel), "gflop": f3 / 1e9, "ms": t3,
                               "tflops": f3 / (t3 * 1e-3) / 1e12, "frac_peak": f3 / (t3 * 1e-3) / 1e12 / peak}
    extra["sum_layer_ms"] = sum(layer_ms)
    extra["algos"] = {a: v[2] for a, v in by_algo.items()}
    # Whole network with the per-layer selection versus every single-algorithm
    # network, all from the selection's own per-layer timings (a network is
    # listed only if its algorithm runs every layer).
    if all(p["timings"] for p in plan):
        import paper_2410_08300_amd as cs
        nets = {"selected": sum(min(p["timings"].values()) for p in plan)}
        for a in cs.CONCRETE_ALGOS:
            if all(a in p["timings"] for p in plan):
                nets[a] = sum(p["timings"][a] for p in plan)
        extra["network_ms_from_selection_timings"] = nets
    extra["steps"] = {m: {"ms_per_step": t, "tflops": total_flops / (t * 1e-3) / 1e12} for m, t in modes.items()}

    if wl == "resnet50" and not args.no_executor:
        extra["executor"] = executor_forward(plan, args.steps, args.warmup)
        extra["executor"]["conv_step_prepacked_ms"] = modes["graph_prepacked"]

    if args.calibrate_copy > 0:
        calibration_copy(args.calibrate_copy, dev)
    extra["measured_peaks"] = measured_peaks(dev)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, args.cpu_budget)

    nbatch = layers[0].n
    out = {"metric": "conv2d TFLOP/s (2*N*K*C/G*R*S*P*Q per layer), best measured algorithm per layer",
           "value": value, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
           "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": dtype, "data": "synthetic (seeded normal inputs, Kaiming-normal weights)",
           "config": {"workload": "%s conv layers (%d convs), batch %d, %s data, fp32 accumulate, %s, %s"
                                  % (wl, len(layers), nbatch, dtype,
                                     "eager launches" if args.eager else "one HIP graph per step",
                                     "filters packaged once before timing" if prepacked
                                     else "filters packed every call"),
                      "global_batch": nbatch, "layers": len(layers), "parallelism": "none (1 GPU)"},
           "roofline": roofline, "cpu_baseline": cpu, "detail": extra}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
