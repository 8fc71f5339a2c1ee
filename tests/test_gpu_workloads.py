"""GPU parity on the five benchmark workloads' layer shapes.

* reduced batch (N=1): the whole output of every unique layer, every
  algorithm that supports it, against the fp64 oracle;
* full batch (the workload's own N, the shapes the benchmark times): sampled
  outputs, including the corners of the first and last output planes,
  against the oracle evaluated point by point on the sampled images."""
import numpy as np
import pytest
import torch

import oracle
import paper_2410_08300_amd as cs
from paper_2410_08300_amd import workloads as W
from gpu_util import ALGOS, tolerance, rel_err, f64, supports, say

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

DEV = torch.device("cuda:0")


def layer_ids(wl):
    return ["%s" % L.name for L, _ in W.unique_layers(W.layers(wl))]


@pytest.mark.parametrize("wl", W.WORKLOADS)
def test_reduced_batch_full_outputs(wl):
    layers = W.unique_layers(W.layers(wl, n=1))
    for li, (L, _) in enumerate(layers):
        x, w, b = W.make_tensors(L, (W.WORKLOADS.index(wl), li, 1))
        ref = oracle.conv2d(f64(x), f64(w), f64(b), L.stride, L.pad, L.dilation, L.groups, L.relu)
        xd, wd = x.to(DEV), w.to(DEV)
        bd = None if b is None else b.to(DEV)
        for algo in ALGOS:
            if not supports(algo, L.r, L.s, L.stride, L.dilation, L.groups):
                continue
            say("case", wl, L.name, "N=1", algo)
            y = cs.conv2d(xd, wd, bd, L.stride, L.pad, L.dilation, L.groups, algo=algo, relu=L.relu)
            torch.cuda.synchronize()
            err = rel_err(f64(y), ref)
            assert err <= tolerance(L.dtype, algo), "%s %s %s: %.3e" % (wl, L.name, algo, err)


@pytest.mark.parametrize("wl", W.WORKLOADS)
def test_full_batch_sampled_outputs(wl):
    layers = W.unique_layers(W.layers(wl))
    for li, (L, _) in enumerate(layers):
        x, w, b = W.make_tensors(L, (W.WORKLOADS.index(wl), li, 2), device=DEV)
        pts = W.random_points(L, 192, seed=li)
        imgs = np.unique(pts[:, 0])
        remap = {int(n): i for i, n in enumerate(imgs)}
        local = pts.copy()
        local[:, 0] = [remap[int(n)] for n in pts[:, 0]]
        xs = f64(x[torch.as_tensor(imgs, device=DEV)])
        ref = oracle.conv2d_points(xs, f64(w), local, f64(b), L.stride, L.pad, L.dilation, L.groups, L.relu)
        idx = torch.as_tensor(pts, device=DEV)
        for algo in ALGOS:
            if not supports(algo, L.r, L.s, L.stride, L.dilation, L.groups):
                continue
            say("case", wl, L.name, "N=%d" % L.n, algo)
            y = cs.conv2d(x, w, b, L.stride, L.pad, L.dilation, L.groups, algo=algo, relu=L.relu)
            got = y[idx[:, 0], idx[:, 1], idx[:, 2], idx[:, 3]]
            ok_finite = bool(torch.isfinite(y).all())
            torch.cuda.synchronize()
            assert ok_finite, "%s %s %s: non-finite output" % (wl, L.name, algo)
            err = rel_err(f64(got), ref)
            assert err <= tolerance(L.dtype, algo), "%s %s %s: %.3e" % (wl, L.name, algo, err)
            del y
        del x, w, b
        torch.cuda.empty_cache()
