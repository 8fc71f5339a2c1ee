"""Per-layer timing of one algorithm on a workload's unique layers.

    python -m paper_2410_08300_amd.layer_timing --workload resnet50 --algo implicit_gemm --taps 3

Each unique layer (shape, stride, padding, dtype) of the workload is run with
the named algorithm on seeded synthetic tensors resident on the GPU; a call is
timed as the median over HIP-graph replays of ``--launches`` back-to-back
calls (``selection.time_conv``), once with filters packed per call and, with
``--prepacked``, once more with a filter package built beforehand.  One line
per layer gives the time, TFLOP/s, the fraction of the dtype's dense MFMA
peak (bf16 2.5 PFLOP/s, fp32 157.3 TFLOP/s), compulsory HBM bytes per second
and the kernels the call runs.  The run is also what a profiler wraps to
collect counters for one kernel on every shape of a workload.
"""
import argparse
import json

import torch

from . import _lib, selection
from . import workloads as W

PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
HBM_GBS = 8000.0


def run(workload, algo, taps=None, prepacked=False, launches=20, reps=7, n=None, only=None):
    dev = torch.device("cuda:0")
    rows = []
    for li, (L, cnt) in enumerate(W.unique_layers(W.layers(workload, n=n))):
        if (taps is not None and L.r != taps) or (only is not None and L.name != only):
            continue
        x, w, b = W.make_tensors(L, (9, li), device=dev)
        d = _lib.make_desc(L.n, L.c, L.h, L.w, L.k, L.r, L.s, L.stride, L.pad, L.dilation, L.groups,
                           dtype=L.dtype, bias=L.bias, relu=L.relu)
        if _lib.check(d, algo) != 0:
            continue
        row = {"layer": L.name, "count": cnt, "C": L.c, "K": L.k, "H": L.h, "R": L.r, "stride": L.stride,
               "dtype": L.dtype,
               "kernels": _lib.describe(d, algo)}
        ms = selection.time_conv(x, w, b, L.stride, L.pad, L.dilation, L.groups, algo, L.relu,
                                 warmup=3, reps=reps, launches=launches)
        row["us"] = ms * 1e3
        if prepacked:
            ms_pk = selection.time_conv(x, w, b, L.stride, L.pad, L.dilation, L.groups, algo, L.relu,
                                        warmup=3, reps=reps, launches=launches, prepacked=True)
            row["us_prepacked"] = ms_pk * 1e3
        tf = L.flops / (ms * 1e-3) / 1e12
        row["tflops"] = tf
        row["frac_mfma"] = tf / PEAK_TFLOPS[L.dtype]
        row["frac_hbm"] = L.compulsory_bytes() / (ms * 1e-3) / 1e9 / HBM_GBS
        row["flops"] = L.flops
        rows.append(row)
        print(json.dumps(row), flush=True)
    return rows


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", default="resnet50")
    ap.add_argument("--n", type=int, default=None, help="batch (default: the workload's own)")
    ap.add_argument("--algo", default="implicit_gemm")
    ap.add_argument("--taps", type=int, default=None, help="only layers with this filter size")
    ap.add_argument("--layer", default=None, help="only the unique layer of this name")
    ap.add_argument("--prepacked", action="store_true")
    ap.add_argument("--launches", type=int, default=20)
    ap.add_argument("--reps", type=int, default=7)
    a = ap.parse_args()
    rows = run(a.workload, a.algo, a.taps, a.prepacked, a.launches, a.reps, a.n, a.layer)
    fl = sum(r["flops"] * r["count"] for r in rows)
    for key in ("us", "us_prepacked"):
        if rows and key in rows[0]:
            t = sum(r[key] * r["count"] for r in rows)
            print(json.dumps({"total": key, "us": t, "tflops": fl / (t * 1e-6) / 1e12}), flush=True)


if __name__ == "__main__":
    main()
