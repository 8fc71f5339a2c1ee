"""GPU checks of the model executor (swap_backend): whole networks and each
of the executor's own kernels against a float64 host reference built from
the oracle's convolution and plain numpy definitions of batch norm, ReLU,
pooling, adds and linear layers (tests/ref_net.py).

Tolerances (max |y - ref| / max |ref| over the network output): fp32
networks 1e-3 -- every convolution is within 1e-4 of its own output (1e-3
for Winograd) and a chain of at most eight layers, with pooling and adds
that do not amplify relative error, stays within their sum; bf16 networks
4e-2 -- each of up to eight layers rounds its output to bf16 (relative
2^-9 ~ 2e-3), the folded batch-norm filters are rounded once more, and the
reference keeps every intermediate in float64, so the rounding adds up over
the chain (twice the single-layer bf16 bar).  A single convolution with a
fused residual add is held to the single-layer bars: 1e-4 (fp32) and 2e-2
(bf16: the convolution's output and the sum are each rounded once).  The
pooling, ReLU and add kernels compute maxima, sums of at most 49 terms and
single adds: 1e-6 in fp32, exact maxima and ReLU."""
import numpy as np
import pytest
import torch

import paper_2410_08300_amd as cs
from gpu_util import rel_err, f64, say
from paper_2410_08300_amd import _lib
import ref_net
from nets import ConvStack, ConvPlusResidual, ResNetSmall, randomize_bn

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

DEV = torch.device("cuda:0")


def reference(net, x):
    """The network evaluated in float64 by the oracle and numpy."""
    return ref_net.reference(net, x)


@pytest.mark.parametrize("sel", ["default", ("direct", "smm"), ("kn2row", "implicit_precomp_gemm"),
                                 ("winograd", "im2col_gemm"), ("implicit_gemm", "implicit_gemm")])
def test_listing1_network(sel):
    torch.manual_seed(0)
    net = ConvStack().eval()
    x = torch.randn(2, 3, 32, 32)
    ref = reference(net, x)
    model = cs.swap_backend(net.to(DEV), list(sel) if isinstance(sel, tuple) else sel)
    say("case listing1", sel)
    with torch.no_grad():
        y = model(x.to(DEV))
    torch.cuda.synchronize()
    assert y.shape == ref.shape
    assert rel_err(f64(y), ref) <= 1e-3


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_residual_network(dtype):
    torch.manual_seed(1)
    net = randomize_bn(ResNetSmall(), 7)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    net = net.to(tdt)
    x = torch.randn(3, 3, 64, 64).to(tdt)
    ref = reference(net, x)
    for sel in ("default", "implicit_gemm", "direct"):
        model = cs.swap_backend(net.to(DEV), sel)
        say("case residual", dtype, sel)
        with torch.no_grad():
            y = model(x.to(DEV))
        torch.cuda.synchronize()
        err = rel_err(f64(y), ref)
        assert err <= (1e-3 if dtype == "f32" else 4e-2), "%s %s: %.3e" % (dtype, sel, err)


def test_new_shape_replans_and_graph_replays_match_eager():
    torch.manual_seed(3)
    net = randomize_bn(ResNetSmall(), 9).to(DEV)
    model = cs.swap_backend(net, "default")
    x2 = torch.randn(2, 3, 48, 48, device=DEV)
    x5 = torch.randn(5, 3, 64, 64, device=DEV)
    with torch.no_grad():
        y2 = model(x2)
        y5 = model(x5)
    torch.cuda.synchronize()
    assert rel_err(f64(y2), reference(net, x2)) <= 1e-3
    assert rel_err(f64(y5), reference(net, x5)) <= 1e-3
    # Capture one forward (planned already) and replay it three times, with
    # eager work between the replays; every replay equals the eager result.
    static_x = x5.clone()
    eager = model(static_x).clone()
    s = torch.cuda.Stream(DEV)
    s.wait_stream(torch.cuda.current_stream(DEV))
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        model(static_x)                       # warm-up on the capture stream
        s.synchronize()
        with torch.cuda.graph(g, stream=s):
            out = model(static_x)
    torch.cuda.current_stream(DEV).wait_stream(s)
    for i in range(3):
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), "replay %d" % i
        _ = model(torch.randn(5, 3, 64, 64, device=DEV))   # eager work in between
        torch.cuda.synchronize()


# One convolution whose output is added to the network input (or to a 1 x 1
# projection of it): every implicit GEMM kernel variant the library picks,
# with and without split-K, planes below eight pixels over several images,
# with and without the ReLU after the add.  (dtype, N, C, H, W, K, R, stride,
# pad, ReLU, kernel the convolution runs: the executor's calls are prepacked)
RESIDUAL = [
    ("bf16", 4, 64, 14, 14, 256, 1, 1, 0, True, "pointwise_dma_kernel<4,4,4>"),
    ("bf16", 4, 256, 14, 14, 64, 1, 1, 0, False, "pointwise_dma_kernel<4,4,4> "),
    ("bf16", 4, 1024, 14, 14, 64, 1, 1, 0, False, "pointwise_dma_kernel<4,4,4>;splitk_reduce_kernel"),
    ("bf16", 24, 256, 14, 14, 1024, 1, 1, 0, True, "kernels=pointwise_img_kernel<7>"),
    ("bf16", 32, 256, 14, 14, 1024, 1, 1, 0, False, "kernels=pointwise_img_kernel<7>"),
    ("bf16", 5, 64, 2, 3, 96, 1, 1, 0, True, "repack_plane_kernel;pointwise_dma_kernel<16,4,4>"),
    ("bf16", 4, 1024, 7, 7, 256, 1, 1, 0, True, "repack_plane_kernel;pointwise_dma_kernel<16,4,4>;splitk_reduce_kernel"),
    ("bf16", 3, 64, 3, 3, 64, 1, 1, 0, False, "repack_plane_kernel;pointwise_dma_kernel<16,4,4>"),
    ("bf16", 2, 64, 28, 28, 64, 3, 1, 1, True, "conv3x3_kernel<32,2,2,1,1,0,8,1,1,0>"),
    ("bf16", 3, 32, 8, 8, 32, 3, 1, 1, False, "conv3x3_kernel<32,2,2,1,1,0,8,1,1,0>"),
    ("bf16", 2, 256, 7, 7, 256, 3, 1, 1, True, "conv3x3_kernel<32,2,2,1,1,0,4,1,1,0>;splitk_reduce_kernel"),
    ("bf16", 2, 24, 9, 9, 40, 3, 1, 1, True, "implicit_ws_kernel<64,0,1>"),
    ("bf16", 32, 256, 14, 14, 256, 3, 1, 1, True, "conv3x3_kernel<32,2,2,2,1,0,8,1,1,0>"),
    ("bf16", 32, 128, 28, 28, 128, 3, 1, 1, False, "conv3x3_kernel<16,2,2,2,2,0,8,1,0,1>"),
    ("bf16", 32, 64, 56, 56, 64, 3, 1, 1, True, "conv3x3_kernel<16,4,1,4,2,0,8,1,0,0>"),
    ("bf16", 32, 128, 56, 56, 128, 3, 2, 1, True, "conv3x3_kernel<16,2,2,2,2,1,8,1,0,1>"),
    ("bf16", 2, 128, 112, 112, 64, 3, 1, 1, False, "conv3x3_kernel<32,2,2,2,1,0,8,1,0,1>"),
    ("bf16", 2, 256, 28, 28, 256, 3, 2, 1, True, "conv3x3_kernel<32,2,2,1,1,1,8,1,0,1>;splitk_reduce_kernel"),
    ("bf16", 4, 256, 14, 14, 256, 3, 1, 1, False, "conv3x3_kernel<32,2,2,1,1,0,8,1,1,0>;splitk_reduce_kernel"),
    ("bf16", 7, 48, 2, 2, 64, 3, 1, 1, True, "implicit_gemm_kernel<bf16,64,2,9>;splitk_reduce_kernel"),
    ("bf16", 2, 3, 32, 32, 16, 3, 1, 1, False, "implicit_gemm_kernel<bf16,64,1,9>"),
    ("bf16", 2, 3, 64, 64, 64, 7, 2, 3, True, "implicit_rows_kernel"),
    ("f32", 2, 64, 28, 28, 64, 3, 1, 1, True, "implicit_gemm_kernel<f32,64,2,9>;splitk_reduce_kernel"),
    ("f32", 3, 16, 16, 16, 16, 3, 1, 1, False, "implicit_gemm_kernel<f32,64,2,9>"),
    ("f32", 5, 64, 2, 3, 96, 1, 1, 0, True, "pointwise_gemm_kernel<f32,64,1,2>"),
    ("f32", 4, 1024, 7, 7, 256, 1, 1, 0, False, "pointwise_gemm_kernel<f32,64,1,2>;splitk_reduce_kernel"),
    ("f32", 4, 64, 56, 56, 256, 1, 1, 0, True, "pointwise_gemm_kernel<f32,64,0,2>"),
    ("f32", 2, 3, 64, 64, 64, 7, 2, 3, False, "implicit_gemm_kernel<f32,64,1,0>"),
]


@pytest.mark.parametrize("case", RESIDUAL, ids=lambda c: "%s-%dx%dx%dx%d-k%d-r%d" % c[:7])
def test_residual_add_fused_into_each_kernel(case):
    dtype, n, c, h, w, k, r, stride, pad, relu, kernels = case
    torch.manual_seed(11)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    net = ConvPlusResidual(c, k, r, stride, pad, relu).to(tdt).eval()
    x = torch.randn(n, c, h, w).to(tdt)
    ref = reference(net, x)
    model = cs.swap_backend(net.to(DEV), {"conv": "implicit_gemm", "proj": "direct"})
    model.plan(x.shape)
    d = model.describe()
    say("case residual-fused", case, d.splitlines()[-3:])
    conv_line = [line for line in d.splitlines() if " conv v0 " in line and "implicit_gemm" in line][0]
    assert " + v" in conv_line and (" relu " in conv_line + " ") == relu
    assert any(line.split()[1] == "add" and " fused " in line + " " for line in d.splitlines())
    desc = _lib.make_desc(n, c, h, w, k, r, r, stride, pad, dtype=dtype, bias=True)
    assert "kernels=" in _lib.describe(desc, "implicit_gemm")
    assert kernels in _lib.describe(desc, "implicit_gemm")
    with torch.no_grad():
        y = model(x.to(DEV))
    torch.cuda.synchronize()
    assert y.shape == ref.shape
    err = rel_err(f64(y), ref)
    assert err <= (1e-4 if dtype == "f32" else 2e-2), "%s: %.3e" % (case, err)


def test_resnet50_through_the_executor():
    """ResNet-50 v1.5 (53 convolutions with folded batch norm, 16 residual
    adds fused into epilogues, max-pool, global average pool, linear head)
    in fp32 at batch 2, 64 x 64, each layer on the library's default choice,
    against the module in fp64 on the CPU: within 1e-3 (fp32 layers are
    within 1e-4 of their own outputs, 1e-3 for Winograd; normalisation keeps
    the magnitudes from growing along the chain)."""
    import bench
    torch.manual_seed(5)
    net = randomize_bn(bench.resnet50_module(), 13)
    x = torch.randn(2, 3, 64, 64)
    ref = reference(net, x)
    model = cs.swap_backend(net.to(DEV), "default")
    model.plan(x.shape)
    d = model.describe()
    assert sum(" fused" in line for line in d.splitlines()) == 16
    say("case resnet50 fp32", len(model.ops), "ops")
    with torch.no_grad():
        y = model(x.to(DEV))
    torch.cuda.synchronize()
    assert y.shape == ref.shape == (2, 1000)
    err = rel_err(f64(y), ref)
    say("resnet50 fp32 rel err %.3e" % err)
    assert err <= 1e-3


def _identity_conv(c, dtype):
    """A 1 x 1 convolution whose output equals its input exactly (unit
    filters, zero bias): gives a parameterised network whose next operation
    runs on the executor's own kernel."""
    conv = torch.nn.Conv2d(c, c, 1)
    with torch.no_grad():
        conv.weight.copy_(torch.eye(c).reshape(c, c, 1, 1))
        conv.bias.zero_()
    return conv.to(dtype)


# (kind, kernel, stride, pad, N, C, H, W): windows of 2x2 to 7x7, strides
# 1-3, padding up to half the window, odd planes.
POOLS = [
    ("max", 2, 2, 0, 2, 5, 13, 11), ("max", 3, 2, 1, 3, 4, 15, 15), ("max", 3, 1, 1, 2, 3, 9, 7),
    ("max", 5, 2, 2, 1, 6, 17, 12), ("max", 3, 3, 0, 2, 4, 10, 14), ("max", 7, 1, 3, 1, 2, 8, 9),
    ("avg", 2, 2, 0, 2, 5, 13, 11), ("avg", 3, 2, 1, 3, 4, 15, 15), ("avg", 3, 1, 1, 2, 3, 9, 7),
    ("avg", 5, 2, 2, 1, 6, 17, 12), ("avg", 3, 3, 0, 2, 4, 10, 14), ("avg", 7, 1, 3, 1, 2, 8, 9),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", POOLS, ids=lambda c: "%s%d-s%d-p%d-%dx%dx%dx%d" % c)
def test_pool_kernel(case, dtype):
    kind, k, st, pad, n, c, h, w = case
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    pool = torch.nn.MaxPool2d(k, st, pad) if kind == "max" else torch.nn.AvgPool2d(k, st, pad)
    net = torch.nn.Sequential(_identity_conv(c, tdt), pool).eval()
    g = torch.Generator().manual_seed(POOLS.index(case))
    x = torch.randn(n, c, h, w, generator=g).to(tdt)
    ref = reference(net, x)
    model = cs.swap_backend(net.to(DEV), "direct")
    say("case pool", case, dtype)
    with torch.no_grad():
        y = model(x.to(DEV))
    torch.cuda.synchronize()
    assert tuple(y.shape) == ref.shape
    got = f64(y)
    if kind == "max":
        assert np.array_equal(got, ref)       # a maximum is one of the inputs
    else:
        # fp32 sum of at most 49 inputs / bf16: the average rounded once
        assert rel_err(got, ref) <= (1e-6 if dtype == "f32" else 2 ** -8)


@pytest.mark.parametrize("hw", [(1, 1), (7, 7), (5, 3), (13, 17), (2, 9)])
def test_global_avgpool_kernel(hw):
    h, w = hw
    net = torch.nn.Sequential(_identity_conv(6, torch.float32), torch.nn.AdaptiveAvgPool2d(1)).eval()
    x = torch.randn(3, 6, h, w, generator=torch.Generator().manual_seed(h * 31 + w))
    ref = reference(net, x)
    model = cs.swap_backend(net.to(DEV), "direct")
    say("case global_avgpool", hw)
    with torch.no_grad():
        y = model(x.to(DEV))
    torch.cuda.synchronize()
    assert tuple(y.shape) == ref.shape == (3, 6, 1, 1)
    assert rel_err(f64(y), ref) <= 1e-6


class _PoolAddRelu(torch.nn.Module):
    """Two pools of one convolution output, added, then a ReLU: neither add
    operand is a convolution output and the ReLU follows the add's second
    reader, so the add and the ReLU run on their own kernels."""

    def __init__(self, c):
        super().__init__()
        self.conv = _identity_conv(c, torch.float32)
        self.p1 = torch.nn.MaxPool2d(3, 1, 1)
        self.p2 = torch.nn.AvgPool2d(3, 1, 1)

    def forward(self, x):
        y = self.conv(x)
        s = self.p1(y) + self.p2(y)
        return torch.relu(self.p1(s)) + s


def test_add_and_relu_kernels():
    net = _PoolAddRelu(5).eval()
    x = torch.randn(2, 5, 11, 9, generator=torch.Generator().manual_seed(4))
    ref = reference(net, x)
    model = cs.swap_backend(net.to(DEV), "direct")
    kinds = [k for k, _ in model.ops]
    assert kinds.count("add") == 2 and kinds.count("relu") == 1
    model.plan(x.shape)
    assert not any(" fused" in line for line in model.describe().splitlines())
    say("case add+relu kernels")
    with torch.no_grad():
        y = model(x.to(DEV))
    torch.cuda.synchronize()
    assert rel_err(f64(y), ref) <= 1e-6
