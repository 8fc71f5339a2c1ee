"""GPU parity: every algorithm of the HIP library against the fp64 CPU oracle
on the same seeded inputs (full outputs at small sizes, sampled outputs at
the workloads' full sizes), plus the intermediate buffers of IM2COL and
Winograd, determinism and edge cases."""
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
TDT = {"f32": torch.float32, "bf16": torch.bfloat16}


def check_full(x, w, b, stride, padding, dilation, groups, relu, algos, label):
    """Run each algorithm on the GPU and compare the whole output."""
    ref = oracle.conv2d(f64(x), f64(w), f64(b), stride, padding, dilation, groups, relu)
    R, S = w.shape[2], w.shape[3]
    xd, wd = x.to(DEV), w.to(DEV)
    bd = None if b is None else b.to(DEV)
    for algo in algos:
        if not supports(algo, R, S, stride, dilation, groups):
            continue
        say("case", label, algo)
        y = cs.conv2d(xd, wd, bd, stride, padding, dilation, groups, algo=algo, relu=relu)
        torch.cuda.synchronize()
        assert y.shape == ref.shape
        err = rel_err(f64(y), ref)
        tol = tolerance(x.dtype, algo)
        assert err <= tol, "%s %s: rel err %.3e > %.0e" % (label, algo, err, tol)


def test_toy_layer_all_algorithms():
    L = W.toy()[0]
    x, w, b = W.make_tensors(L, (0, 0))
    check_full(x, w, b, 1, 1, 1, 1, False, ALGOS, "toy")


def sweep_cases(count, seed):
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < count:
        R = int(rng.choice([1, 2, 3, 3, 3, 5]))
        S = R if rng.random() < 0.8 else int(rng.choice([1, 3]))
        st = (int(rng.integers(1, 4)), int(rng.integers(1, 4))) if rng.random() < 0.3 else int(rng.choice([1, 1, 2]))
        pd = (int(rng.integers(0, 3)), int(rng.integers(0, 3))) if rng.random() < 0.3 else int(rng.integers(0, 3))
        dl = int(rng.choice([1, 1, 1, 2]))
        G = int(rng.choice([1, 1, 1, 2, 4]))
        Cg = int(rng.choice([1, 3, 8, 13, 16, 24, 40]))
        Kg = int(rng.choice([1, 5, 32, 64, 70, 130]))
        if G > 1:
            Kg = min(Kg, 40)
        N = int(rng.integers(1, 4))
        H, Wd = int(rng.integers(1, 34)), int(rng.integers(1, 34))
        P, Q = oracle.output_size(H, Wd, R, S, st, pd, dl)
        if P < 1 or Q < 1:
            continue
        dtype = "bf16" if rng.random() < 0.5 else "f32"
        bias = bool(rng.random() < 0.5)
        relu = bool(rng.random() < 0.3)
        cases.append((N, Cg * G, H, Wd, Kg * G, R, S, st, pd, dl, G, dtype, bias, relu))
    return cases


SWEEP = sweep_cases(48, 2024)


@pytest.mark.parametrize("idx", range(len(SWEEP)), ids=lambda i: "%d_" % i + "x".join(map(str, SWEEP[i][:7])) + "_" + SWEEP[i][11])
def test_random_shape_sweep(idx):
    case = SWEEP[idx]
    N, C, H, Wd, K, R, S, st, pd, dl, G, dtype, bias, relu = case
    g = torch.Generator().manual_seed(W.seed_for(7, idx))
    x = torch.randn(N, C, H, Wd, generator=g).to(TDT[dtype])
    w = (torch.randn(K, C // G, R, S, generator=g) * (2.0 / ((C // G) * R * S)) ** 0.5).to(TDT[dtype])
    b = (torch.randn(K, generator=g) * 0.1).to(TDT[dtype]) if bias else None
    check_full(x, w, b, st, pd, dl, G, relu, ALGOS, str(case))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_winograd_odd_sizes_and_padding(dtype):
    g = torch.Generator().manual_seed(5)
    for (N, C, H, Wd, K, pad) in [(2, 16, 7, 7, 24, 1), (1, 9, 5, 8, 40, 0), (3, 33, 14, 13, 70, 2),
                                  (1, 64, 28, 28, 64, 1), (1, 8, 1, 1, 8, 1)]:
        x = torch.randn(N, C, H, Wd, generator=g).to(TDT[dtype])
        w = (torch.randn(K, C, 3, 3, generator=g) / (3 * C ** 0.5)).to(TDT[dtype])
        b = (torch.randn(K, generator=g) * 0.1).to(TDT[dtype])
        check_full(x, w, b, 1, pad, 1, 1, False, ["winograd"], "wino%s" % ((N, C, H, Wd, K, pad),))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_im2col_buffer_is_bit_exact(dtype):
    g = torch.Generator().manual_seed(6)
    for (N, C, H, Wd, R, S, st, pd, dl, G) in [(2, 3, 9, 11, 3, 3, 1, 1, 1, 1), (1, 8, 12, 7, 5, 3, 2, (2, 1), 1, 2),
                                               (2, 6, 10, 10, 3, 3, (1, 2), 2, 2, 3), (1, 4, 5, 5, 1, 1, 1, 0, 1, 4)]:
        x = torch.randn(N, C, H, Wd, generator=g).to(TDT[dtype])
        say("case im2col", dtype, (N, C, H, Wd, R, S, st, pd, dl, G))
        col = cs.im2col(x.to(DEV), (R, S), st, pd, dl, G)
        torch.cuda.synchronize()
        ref = oracle.im2col(f64(x), R, S, st, pd, dl, G)
        assert col.shape == ref.shape
        assert np.array_equal(f64(col), ref)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_winograd_transforms_match_oracle(dtype):
    g = torch.Generator().manual_seed(7)
    x = torch.randn(2, 24, 9, 10, generator=g).to(TDT[dtype])
    w = torch.randn(16, 24, 3, 3, generator=g).to(TDT[dtype])
    say("case winograd transforms", dtype)
    U = cs.winograd_filter_transform(w.to(DEV))
    V = cs.winograd_input_transform(x.to(DEV), padding=1)
    torch.cuda.synchronize()
    Uo = oracle.winograd_filter_transform(f64(w)).reshape(16, 16, 24)
    Vo = oracle.winograd_input_transform(f64(x), padding=1).reshape(16, -1, 24)
    # Relative to each buffer's largest entry: fp32 carries only the rounding
    # of a few adds (< 1e-6); bf16 adds one rounding of each result (2^-8).
    tol = 1e-6 if dtype == "f32" else 2.0 ** -8
    eu, ev = rel_err(f64(U), Uo), rel_err(f64(V), Vo)
    assert eu <= tol, "U rel err %.3e" % eu
    assert ev <= tol, "V rel err %.3e" % ev


def test_reruns_are_bit_identical():
    g = torch.Generator().manual_seed(8)
    x = torch.randn(4, 64, 20, 20, generator=g).to(DEV, torch.bfloat16)
    w = torch.randn(96, 64, 3, 3, generator=g).to(DEV, torch.bfloat16)
    for algo in ALGOS:
        say("case determinism", algo)
        a = cs.conv2d(x, w, None, 1, 1, algo=algo)
        b = cs.conv2d(x, w, None, 1, 1, algo=algo)
        torch.cuda.synchronize()
        assert torch.equal(a, b)


def test_edge_cases():
    g = torch.Generator().manual_seed(9)
    # empty batch: no-op
    x = torch.empty(0, 4, 8, 8, device=DEV)
    w = torch.randn(4, 4, 3, 3, generator=g).to(DEV)
    for algo in ALGOS:
        say("case empty batch", algo)
        y = cs.conv2d(x, w, None, 1, 1, algo=algo)
        assert y.shape == (0, 4, 8, 8)
    # 1x1 image with large padding; output larger than input
    x = torch.randn(2, 5, 1, 1, generator=g)
    w = torch.randn(7, 5, 3, 3, generator=g)
    check_full(x, w, None, 1, 2, 1, 1, False, ALGOS, "1x1 image pad 2")
    # single output pixel, single channels
    x = torch.randn(1, 1, 3, 3, generator=g)
    w = torch.randn(1, 1, 3, 3, generator=g)
    check_full(x, w, torch.randn(1, generator=g), 1, 0, 1, 1, True, ALGOS, "1x1 output")
    # many output channels: several 128-row tiles plus a ragged tail
    x = torch.randn(1, 32, 6, 7, generator=g).to(torch.bfloat16)
    w = (torch.randn(300, 32, 3, 3, generator=g) * 0.1).to(torch.bfloat16)
    check_full(x, w, None, 1, 1, 1, 1, False, ALGOS, "K=300")
    # non-contiguous input
    xt = torch.randn(2, 9, 12, 8, generator=g).transpose(2, 3)
    check_full(xt.contiguous(), torch.randn(6, 9, 3, 3, generator=g), None, 1, 1, 1, 1, False, ALGOS, "strided")
    yd = cs.conv2d(xt.to(DEV), torch.randn(6, 9, 3, 3, generator=g).to(DEV), None, 1, 1)
    assert yd.shape == (2, 6, 8, 12)
    # output written into a view that is not 16-byte aligned (2-byte offset)
    x = torch.randn(2, 16, 8, 8, generator=g).to(torch.bfloat16)
    w = (torch.randn(40, 16, 3, 3, generator=g) * 0.2).to(torch.bfloat16)
    ref = oracle.conv2d(f64(x), f64(w), None, 1, 1)
    for algo in ALGOS:
        buf = torch.zeros(2 * 40 * 64 + 1, device=DEV, dtype=torch.bfloat16)
        out = buf[1:].view(2, 40, 8, 8)
        say("case unaligned output", algo)
        cs.conv2d(x.to(DEV), w.to(DEV), None, 1, 1, algo=algo, out=out)
        torch.cuda.synchronize()
        assert rel_err(f64(out), ref) <= tolerance("bf16", algo)
        assert float(buf[0]) == 0.0


# Output planes smaller than one 8-pixel store run (P*Q < 8) with several
# images: a run of a tile then crosses several image boundaries, which the
# epilogues must follow one element at a time.  A linear layer run as a
# 1x1 convolution (H = W = 1) is the common case.
TINY = [
    # N, C, H, W, K, R, S, stride, pad
    (3, 32, 1, 1, 10, 1, 1, 1, 0),
    (4, 300, 1, 1, 70, 1, 1, 1, 0),
    (4, 24, 2, 3, 40, 3, 3, 1, 1),
    (5, 16, 3, 3, 72, 3, 3, 2, 1),
    (3, 64, 7, 7, 64, 7, 7, 1, 0),
    (6, 8, 5, 5, 130, 5, 5, 1, 0),
    (9, 40, 2, 2, 24, 1, 1, 1, 0),
    (5, 64, 2, 3, 96, 1, 1, 1, 0),
    (7, 48, 2, 2, 64, 3, 3, 1, 1),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("idx", range(len(TINY)), ids=lambda i: "x".join(map(str, TINY[i][:7])))
def test_tiny_planes_several_images(idx, dtype):
    N, C, H, Wd, K, R, S, st, pd = TINY[idx]
    g = torch.Generator().manual_seed(W.seed_for(17, idx))
    x = torch.randn(N, C, H, Wd, generator=g).to(TDT[dtype])
    w = (torch.randn(K, C, R, S, generator=g) * (2.0 / (C * R * S)) ** 0.5).to(TDT[dtype])
    b = (torch.randn(K, generator=g) * 0.1).to(TDT[dtype])
    check_full(x, w, b, st, pd, 1, 1, False, ALGOS, "tiny %s %s" % (TINY[idx], dtype))


def test_unsupported_and_invalid_calls_raise():
    x = torch.randn(1, 4, 8, 8, device=DEV)
    with pytest.raises(cs.Conv2dError):
        cs.conv2d(x, torch.randn(4, 4, 5, 5, device=DEV), None, 1, 2, algo="winograd")
    with pytest.raises(ValueError):
        cs.conv2d(x, torch.randn(4, 3, 3, 3, device=DEV))
    with pytest.raises(ValueError):
        cs.conv2d(x, torch.randn(4, 4, 3, 3, device=DEV, dtype=torch.bfloat16))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_prepacked_filters_give_identical_outputs(dtype):
    """conv2d_prepacked with a package from conv2d_pack_filters runs the same
    kernels on the same data as conv2d, so the outputs are bit-identical."""
    g = torch.Generator().manual_seed(10)
    for (N, C, H, Wd, K, R, st, pd, G) in [(4, 64, 14, 14, 96, 3, 1, 1, 1), (2, 48, 9, 11, 40, 1, 2, 0, 1),
                                           (3, 24, 12, 12, 24, 3, 1, 1, 24), (1, 512, 7, 7, 512, 3, 1, 1, 1)]:
        x = torch.randn(N, C, H, Wd, generator=g).to(TDT[dtype]).to(DEV)
        w = (torch.randn(K, C // G, R, R, generator=g) * 0.1).to(TDT[dtype]).to(DEV)
        b = (torch.randn(K, generator=g) * 0.1).to(TDT[dtype]).to(DEV)
        for algo in ALGOS:
            if not supports(algo, R, R, st, 1, G):
                continue
            say("case prepacked", dtype, (N, C, H, Wd, K, R, st, pd, G), algo)
            y0 = cs.conv2d(x, w, b, st, pd, 1, G, algo=algo)
            pk = cs.pack_filters(w, tuple(x.shape), st, pd, 1, G, algo, bias=True)
            y1 = cs.conv2d_prepacked(x, pk, tuple(w.shape), b, st, pd, 1, G, algo=algo)
            torch.cuda.synchronize()
            assert torch.equal(y0, y1)


def test_swapped_model_matches_oracle_chain_and_caches_packages():
    """The paper's Listing 1 network, swapped per layer, on the GPU; each
    layer checked against the oracle (fp32), and filter packages reused."""
    import torch.nn.functional as F
    from torch import nn
    torch.manual_seed(0)
    model = nn.Sequential(nn.Conv2d(3, 16, 3, padding=1), nn.ReLU(), nn.MaxPool2d(2, 2),
                          nn.Conv2d(16, 32, 3, padding=1), nn.ReLU())
    x = torch.randn(2, 3, 32, 32)
    ref = x.double().numpy()
    for m in model:
        if isinstance(m, nn.Conv2d):
            ref = oracle.conv2d(ref, m.weight.detach().double().numpy(), m.bias.detach().double().numpy(), 1, 1)
        elif isinstance(m, nn.ReLU):
            ref = np.maximum(ref, 0)
        else:
            ref = F.max_pool2d(torch.from_numpy(ref), 2, 2).numpy()
    model = model.to(DEV)
    for sel in (["direct", "winograd"], ["implicit_gemm", "gemm"], lambda c: "default"):
        table = cs.swap_conv2d(model, sel)
        say("case swapped model", list(table.values()))
        with torch.no_grad():
            out = model(x.to(DEV))
            out2 = model(x.to(DEV))
        torch.cuda.synchronize()
        assert rel_err(f64(out), ref) <= 1e-3
        assert torch.equal(out, out2)
    convs = [m for m in model.modules() if isinstance(m, cs.Conv2dSwap)]
    assert all(len(m._packages) >= 1 for m in convs)
    # Cached selector: the first forward measures every supported algorithm
    # per shape and records the fastest; the second reuses the record, and
    # so does a model swapped with the cache read back from its JSON.
    cache = cs.AlgoCache(device=torch.cuda.get_device_name(0))
    table = cs.swap_conv2d(model, cache)
    with torch.no_grad():
        out = model(x.to(DEV))
    torch.cuda.synchronize()
    assert rel_err(f64(out), ref) <= 1e-3
    assert len(cache) == 2
    for e in cache.entries.values():
        assert e["algo"] == min(e["ms"], key=e["ms"].get) and len(e["ms"]) >= 6
    before = {k: dict(v) for k, v in cache.entries.items()}
    with torch.no_grad():
        out2 = model(x.to(DEV))
    torch.cuda.synchronize()
    assert cache.entries == before and torch.equal(out, out2)
    back = cs.AlgoCache.from_json(cache.to_json())
    cs.swap_conv2d(model, back)
    with torch.no_grad():
        out3 = model(x.to(DEV))
    torch.cuda.synchronize()
    assert back.entries == before and torch.equal(out, out3)


# 1x1 layers take their own kernel (filters used as given, pixel-quad loads
# transposed in registers) when C is a multiple of the 16-byte unit; strided,
# padded or odd-plane layers and unaligned inputs take its gather variant;
# unaligned filters are copied first.  Each case names the path it covers.
POINTWISE = [
    # N, C, H, W, K, stride, pad, dtype, bias, relu, what
    (3, 72, 10, 10, 200, 1, 0, "bf16", True, True, "contiguous, channel / filter / pixel tails"),
    (3, 36, 10, 10, 200, 1, 0, "f32", True, False, "contiguous fp32, channel tail"),
    (2, 64, 15, 15, 96, 2, 0, "bf16", False, False, "stride 2 (gather)"),
    (2, 32, 15, 15, 96, 2, 0, "f32", True, True, "stride 2 fp32 (gather)"),
    (5, 128, 7, 7, 256, 1, 0, "bf16", False, True, "7x7 plane, not a multiple of 4 (gather)"),
    (2, 16, 6, 6, 32, 1, 1, "bf16", True, False, "padding 1 (gather, zero border)"),
    (2, 1000, 7, 7, 300, 1, 0, "bf16", True, True, "channel split over workgroups, tail chunk"),
    (2, 40, 9, 12, 40, 1, 0, "f32", False, False, "K <= 64 tile"),
    (4, 24, 28, 28, 64, 1, 0, "bf16", False, False, "single partial chunk"),
    (3, 256, 14, 14, 300, 1, 0, "bf16", True, False, "14x14 plane read in place as pixel pairs, tiles cross images"),
    (24, 256, 14, 14, 1024, 1, 0, "bf16", True, False, "14x14 whole-image tiles, 192 units"),
    (24, 200, 14, 14, 1024, 1, 0, "bf16", False, True, "14x14 whole-image tiles, channel tail"),
    (40, 256, 14, 14, 1024, 1, 0, "bf16", True, True, "14x14 whole-image tiles, 320 units: two per workgroup"),
    (3, 64, 56, 56, 96, 2, 0, "bf16", True, False, "stride 2, rows of 28 (row-aligned repack)"),
    (4, 128, 28, 28, 64, 2, 0, "bf16", False, True, "stride 2, rows of 14, span tail"),
    (5, 96, 14, 14, 80, 2, 0, "bf16", True, True, "stride 2, rows of 7"),
    (3, 48, 15, 13, 40, 2, 0, "bf16", False, False, "stride 2, odd plane, last loads element by element"),
]


@pytest.mark.parametrize("idx", range(len(POINTWISE)), ids=lambda i: POINTWISE[i][-1].replace(" ", "_"))
def test_pointwise_paths(idx):
    N, C, H, Wd, K, st, pd, dtype, bias, relu, what = POINTWISE[idx]
    g = torch.Generator().manual_seed(W.seed_for(11, idx))
    x = torch.randn(N, C, H, Wd, generator=g).to(TDT[dtype])
    w = (torch.randn(K, C, 1, 1, generator=g) * (2.0 / C) ** 0.5).to(TDT[dtype])
    b = (torch.randn(K, generator=g) * 0.1).to(TDT[dtype]) if bias else None
    check_full(x, w, b, st, pd, 1, 1, relu, ("implicit_gemm", "im2col_gemm", "direct"), what)


@pytest.mark.parametrize("which,side", [("x", 12), ("w", 12), ("x", 14)])
def test_pointwise_unaligned_operands(which, side):
    """1x1 layer with the input (gather variant) or the filters (copied into
    the workspace first) one element past a 16-byte boundary; a 14 x 14
    plane is otherwise read in place as pixel pairs, which needs 4-byte
    alignment."""
    N, C, H, Wd, K = 2, 64, side, side, 80
    g = torch.Generator().manual_seed(W.seed_for(12, 0 if which == "x" else 1))
    x = torch.randn(N, C, H, Wd, generator=g).to(torch.bfloat16)
    w = (torch.randn(K, C, 1, 1, generator=g) * (2.0 / C) ** 0.5).to(torch.bfloat16)
    ref = oracle.conv2d(f64(x), f64(w), None, 1, 0, 1, 1, False)
    xd, wd = x.to(DEV), w.to(DEV)
    if which == "x":
        buf = torch.empty(xd.numel() + 1, dtype=xd.dtype, device=DEV)
        buf[1:].copy_(xd.reshape(-1))
        xd = buf[1:].view(xd.shape)
        assert xd.data_ptr() % 16 != 0
    else:
        buf = torch.empty(wd.numel() + 1, dtype=wd.dtype, device=DEV)
        buf[1:].copy_(wd.reshape(-1))
        wd = buf[1:].view(wd.shape)
        assert wd.data_ptr() % 16 != 0
    say("case unaligned", which)
    y = cs.conv2d(xd, wd, None, algo="implicit_gemm")
    torch.cuda.synchronize()
    assert rel_err(f64(y), ref) <= tolerance("bf16", "implicit_gemm")


def test_pointwise_whole_image_tiles_fall_back_for_unaligned_output():
    """A 14 x 14 layer that would take whole-image tiles (16-byte stores of
    each image's rows) with the output one element past a 16-byte boundary:
    the call takes the pixel-pair kernel and is still correct."""
    from paper_2410_08300_amd import _lib
    N, C, H, Wd, K = 24, 256, 14, 14, 1024
    g = torch.Generator().manual_seed(W.seed_for(12, 7))
    x = torch.randn(N, C, H, Wd, generator=g).to(torch.bfloat16)
    w = (torch.randn(K, C, 1, 1, generator=g) * (2.0 / C) ** 0.5).to(torch.bfloat16)
    desc = _lib.make_desc(N, C, H, Wd, K, 1, 1, 1, 0, 1, 1, "bf16")
    assert "pointwise_img_kernel" in _lib.describe(desc, "implicit_gemm")
    ref = oracle.conv2d(f64(x), f64(w), None, 1, 0, 1, 1, False)
    xd, wd = x.to(DEV), w.to(DEV)
    ybuf = torch.zeros(N * K * H * Wd + 1, dtype=torch.bfloat16, device=DEV)
    y = ybuf[1:]
    assert y.data_ptr() % 16 != 0
    nws = _lib.workspace_bytes(desc, "implicit_gemm")
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=DEV)
    say("case whole-image tiles, unaligned y")
    st = _lib.conv2d_raw(xd.data_ptr(), wd.data_ptr(), None, y.data_ptr(), desc, "implicit_gemm", ws.data_ptr(), nws,
                         torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert st == _lib.CONV_OK
    assert rel_err(f64(y.view(N, K, H, Wd)), ref) <= tolerance("bf16", "implicit_gemm")


# Wide-filter, few-channel bf16 layers (5 <= S <= 8, even column stride,
# C*R <= 64) take the filter-row kernel: the filter width padded to 8 and
# each reduction slice one input row of the staged halo.  Each case names
# the part of it that it covers.
ROWS = [
    # N, C, H, W, K, R, S, stride, pad, dilation, bias, relu, what
    (2, 3, 40, 40, 64, 7, 7, 2, 3, 1, True, True, "stem-like 7x7 s2 (16-byte halo loads)"),
    (3, 3, 23, 29, 64, 7, 7, 2, 3, 1, False, False, "odd plane: tiles cross images"),
    (3, 3, 23, 32, 64, 7, 7, 2, 3, 1, True, False, "16-byte halo loads, tiles cross images"),
    (2, 8, 20, 24, 40, 7, 7, 2, 3, 1, True, False, "C*R = 56 units, K tail"),
    (2, 5, 19, 17, 130, 5, 5, 2, 2, 1, False, True, "5x5 even pad, three K tiles with tail, odd C*R"),
    (2, 2, 17, 30, 64, 3, 8, 2, (1, 2), 1, True, False, "3x8 taps, no lead tap"),
    (2, 3, 26, 26, 32, 6, 6, (1, 2), (2, 3), (2, 1), False, False, "row stride 1, row dilation 2"),
    (1, 1, 9, 70, 64, 5, 7, (3, 4), (0, 5), 1, True, True, "one channel, stride 3x4, wide pad"),
]


@pytest.mark.parametrize("idx", range(len(ROWS)), ids=lambda i: ROWS[i][-1].replace(" ", "_"))
def test_filter_row_kernel(idx):
    N, C, H, Wd, K, R, S, st, pd, dl, bias, relu, what = ROWS[idx]
    g = torch.Generator().manual_seed(W.seed_for(14, idx))
    x = torch.randn(N, C, H, Wd, generator=g).to(torch.bfloat16)
    w = (torch.randn(K, C, R, S, generator=g) * (2.0 / (C * R * S)) ** 0.5).to(torch.bfloat16)
    b = (torch.randn(K, generator=g) * 0.1).to(torch.bfloat16) if bias else None
    check_full(x, w, b, st, pd, dl, 1, relu, ("implicit_gemm", "direct"), what)


def test_filter_row_kernel_unaligned_filters_and_nonfinite_outside_taps():
    """Stem-like layer with the filters one element past a 16-byte boundary,
    and an input whose columns past every window's reach hold infinities:
    the kernel's zero-weight taps (s >= S) must not pick them up."""
    N, C, H, Wd, K = 2, 3, 21, 21, 64
    g = torch.Generator().manual_seed(W.seed_for(15, 0))
    x = torch.randn(N, C, H, Wd, generator=g).to(torch.bfloat16)
    w = (torch.randn(K, C, 7, 7, generator=g) * (2.0 / 147) ** 0.5).to(torch.bfloat16)
    # stride 2, pad 3: P = Q = 11 and the last window covers columns 17..23
    # (21..23 padding), so column 20 is read; stride 2 without padding on
    # the right: Q = 8, windows end at column 20, and tap s = 7 of the last
    # output would read column 21 -- pass width 22 with inf there.
    x2 = torch.cat([x, torch.full((N, C, H, 1), float("inf"), dtype=torch.bfloat16)], dim=3)
    ref = oracle.conv2d(f64(x2), f64(w), None, 2, (3, 0), 1, 1, False)
    assert np.isfinite(ref).all()
    wd = torch.empty(w.numel() + 1, dtype=w.dtype, device=DEV)
    wd[1:].copy_(w.reshape(-1).to(DEV))
    wd = wd[1:].view(w.shape)
    assert wd.data_ptr() % 16 != 0
    from paper_2410_08300_amd import _lib
    desc = _lib.make_desc(N, C, H, Wd + 1, K, 7, 7, 2, (3, 0), 1, 1, "bf16")
    assert "implicit_rows_kernel" in _lib.describe(desc, "implicit_gemm")
    say("case rows unaligned+inf")
    y = cs.conv2d(x2.to(DEV), wd, None, 2, (3, 0), algo="implicit_gemm")
    torch.cuda.synchronize()
    assert torch.isfinite(y).all()
    assert rel_err(f64(y), ref) <= tolerance("bf16", "implicit_gemm")


@pytest.mark.parametrize("C", [64, 40])
def test_3x3_unaligned_filters(C):
    """bf16 3x3 layer whose filters start one element past a 16-byte
    boundary: the package is built element by element (as for C % 16 != 0)
    instead of from 16-byte loads."""
    N, H, Wd, K = 2, 12, 12, 96
    g = torch.Generator().manual_seed(W.seed_for(16, C))
    x = torch.randn(N, C, H, Wd, generator=g).to(torch.bfloat16)
    w = (torch.randn(K, C, 3, 3, generator=g) * (2.0 / (9 * C)) ** 0.5).to(torch.bfloat16)
    ref = oracle.conv2d(f64(x), f64(w), None, 1, 1, 1, 1, False)
    buf = torch.empty(w.numel() + 1, dtype=w.dtype, device=DEV)
    buf[1:].copy_(w.reshape(-1).to(DEV))
    wd = buf[1:].view(w.shape)
    assert wd.data_ptr() % 16 != 0
    say("case 3x3 unaligned filters", C)
    y = cs.conv2d(x.to(DEV), wd, None, 1, 1, algo="implicit_gemm")
    torch.cuda.synchronize()
    assert rel_err(f64(y), ref) <= tolerance("bf16", "implicit_gemm")


# Every byte a call writes must lie in y or in its workspace: the operands
# and the workspace sit in one buffer between guard bands of a fill pattern,
# and after the call the guards and the inputs must be unchanged.
GUARDED = [
    # N, C, H, W, K, R, stride, pad, dtype, algos
    (1, 1024, 14, 14, 512, 1, 1, 0, "bf16", ("implicit_gemm", "im2col_gemm")),
    (2, 2048, 7, 7, 512, 1, 1, 0, "bf16", ("implicit_gemm",)),
    (24, 256, 14, 14, 1024, 1, 1, 0, "bf16", ("implicit_gemm",)),
    (3, 64, 56, 56, 256, 1, 1, 0, "bf16", ("implicit_gemm",)),
    (2, 256, 15, 15, 128, 1, 2, 0, "bf16", ("implicit_gemm", "im2col_gemm")),
    (2, 512, 7, 7, 512, 3, 1, 1, "bf16", ("implicit_gemm", "winograd", "im2col_gemm")),
    (1, 3, 33, 33, 64, 7, 2, 3, "bf16", ("implicit_gemm", "direct", "im2col_gemm")),
    (3, 3, 29, 23, 64, 7, 2, 3, "bf16", ("implicit_gemm",)),
    (2, 96, 9, 11, 40, 1, 1, 0, "f32", ("implicit_gemm", "direct")),
    (2, 64, 10, 10, 64, 3, 1, 1, "f32", ("implicit_gemm", "winograd")),
    (2, 40, 13, 11, 70, 3, 2, 1, "f32", ("implicit_precomp_gemm", "kn2row", "smm")),
    (3, 24, 9, 17, 130, 5, 1, 2, "bf16", ("implicit_precomp_gemm", "kn2row", "smm")),
    (1, 3, 33, 33, 64, 7, 2, 3, "bf16", ("implicit_precomp_gemm", "kn2row", "smm")),
]


@pytest.mark.parametrize("idx", range(len(GUARDED)), ids=lambda i: "x".join(map(str, GUARDED[i][:6])) + "_" + GUARDED[i][8])
def test_writes_stay_in_output_and_workspace(idx):
    from paper_2410_08300_amd import _lib
    N, C, H, Wd, K, R, st, pd, dtype, algos = GUARDED[idx]
    tdt = TDT[dtype]
    es = 2 if dtype == "bf16" else 4
    g = torch.Generator().manual_seed(W.seed_for(13, idx))
    x = torch.randn(N, C, H, Wd, generator=g).to(tdt)
    w = (torch.randn(K, C, R, R, generator=g) * (2.0 / (C * R * R)) ** 0.5).to(tdt)
    b = (torch.randn(K, generator=g) * 0.1).to(tdt)
    desc = _lib.make_desc(N, C, H, Wd, K, R, R, st, pd, 1, 1, dtype, True, False)
    P, Q = _lib.output_shape(desc)
    ref = oracle.conv2d(f64(x), f64(w), f64(b), st, pd, 1, 1, False)
    guard = 4096
    for algo in algos:
        nws = _lib.workspace_bytes(desc, algo)
        sizes = [x.numel() * es, w.numel() * es, b.numel() * es, nws, N * K * P * Q * es]
        offs, pos = [], guard
        for sz in sizes:
            offs.append(pos)
            pos += (sz + 255) // 256 * 256 + guard
        buf = torch.full((pos,), 0xA5, dtype=torch.uint8, device=DEV)
        for t, o in zip((x, w, b), offs):
            buf[o:o + t.numel() * es].copy_(t.reshape(-1).view(torch.uint8).to(DEV))
        before = buf.cpu()
        base = buf.data_ptr()
        say("case guarded", GUARDED[idx][:9], algo)
        stv = _lib.conv2d_raw(base + offs[0], base + offs[1], base + offs[2], base + offs[4], desc, algo,
                              base + offs[3] if nws else None, nws, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        assert stv == _lib.CONV_OK
        after = buf.cpu()
        ys, ye = offs[4], offs[4] + sizes[4]
        wss, wse = offs[3], offs[3] + nws
        changed = (after != before).nonzero().flatten()
        outside = changed[~(((changed >= ys) & (changed < ye)) | ((changed >= wss) & (changed < wse)))]
        assert outside.numel() == 0, "%s wrote %d bytes outside y and the workspace (first at offset %d)" % (
            algo, outside.numel(), int(outside[0]) - ys)
        y = after[ys:ye].view(tdt).reshape(N, K, P, Q)
        assert rel_err(f64(y), ref) <= tolerance(dtype, algo)
