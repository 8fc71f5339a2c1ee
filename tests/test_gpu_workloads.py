"""GPU parity on the five benchmark workloads' layer shapes.

* reduced batch (N=1): the whole output of every unique layer, every
  algorithm that supports it, against the fp64 oracle;
* full batch (the workload's own N: the shapes and launch configurations the
  benchmark times, including the multi-unit persistent walks, split-K and
  image-batched launches that only appear there): the whole output of every
  unique layer, every supported algorithm, against the oracle on the same
  inputs.  The random 20-layer chain (N = 128) is compared on whole output
  planes of 8 of its images (the first, the last and six seeded ones),
  which the GPU computes within the full-batch launch;
* reruns of the full-batch implicit GEMM calls are bit-identical (the split-K
  reduction sums the partials in a fixed order), and so are the same calls
  with a filter package built beforehand."""
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


def full_batch_cases():
    out = []
    for wl in W.WORKLOADS:
        for li, (L, _) in enumerate(W.unique_layers(W.layers(wl))):
            out.append(pytest.param(wl, li, id="%s-%s" % (wl, L.name)))
    return out


def subset_images(L):
    """All images, or for batches above 32 the first, the last and six
    seeded others."""
    if L.n <= 32:
        return None
    rng = np.random.default_rng(W.seed_for(77, L.n))
    mid = rng.choice(np.arange(1, L.n - 1), size=6, replace=False)
    return np.sort(np.concatenate([[0, L.n - 1], mid]))


def dev_rel_err(y, ref_dev):
    """max |y - ref| / max |ref| computed on the GPU in float64."""
    scale = ref_dev.abs().max()
    diff = (y.double() - ref_dev).abs().max()
    return float(diff / scale) if float(scale) > 0 else float(diff)


@pytest.mark.parametrize("wl,li", full_batch_cases())
def test_full_batch_full_outputs(wl, li):
    L, _ = W.unique_layers(W.layers(wl))[li]
    x, w, b = W.make_tensors(L, (W.WORKLOADS.index(wl), li, 2), device=DEV)
    imgs = subset_images(L)
    xs = x if imgs is None else x[torch.as_tensor(imgs, device=DEV)]
    ref = oracle.conv2d(f64(xs), f64(w), f64(b), L.stride, L.pad, L.dilation, L.groups, L.relu)
    ref_dev = torch.from_numpy(ref).to(DEV)
    del ref
    sel = None if imgs is None else torch.as_tensor(imgs, device=DEV)
    for algo in ALGOS:
        if not supports(algo, L.r, L.s, L.stride, L.dilation, L.groups):
            continue
        say("case", wl, L.name, "N=%d" % L.n, algo, "images=%s" % ("all" if imgs is None else list(imgs)))
        y = cs.conv2d(x, w, b, L.stride, L.pad, L.dilation, L.groups, algo=algo, relu=L.relu)
        ys = y if sel is None else y[sel]
        err = dev_rel_err(ys, ref_dev)
        finite = bool(torch.isfinite(y).all())
        assert finite, "%s %s %s: non-finite output" % (wl, L.name, algo)
        assert err <= tolerance(L.dtype, algo), "%s %s %s: %.3e" % (wl, L.name, algo, err)
        if algo == "implicit_gemm":
            y2 = cs.conv2d(x, w, b, L.stride, L.pad, L.dilation, L.groups, algo=algo, relu=L.relu)
            assert torch.equal(y, y2), "%s %s: rerun differs" % (wl, L.name)
            # The prepacked call (another filter path in some kernels, the
            # same reduction order) gives the same bits.
            pk = cs.pack_filters(w, tuple(x.shape), L.stride, L.pad, L.dilation, L.groups, algo,
                                 bias=b is not None, relu=L.relu)
            y2 = cs.conv2d_prepacked(x, pk, tuple(w.shape), b, L.stride, L.pad, L.dilation, L.groups,
                                     algo=algo, relu=L.relu)
            assert torch.equal(y, y2), "%s %s: prepacked call differs" % (wl, L.name)
            del y2, pk
        del y, ys
    del x, w, b, xs, ref_dev
    torch.cuda.empty_cache()
