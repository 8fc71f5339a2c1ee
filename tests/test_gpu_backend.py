"""GPU checks of the model executor (swap_backend): whole networks against
the same modules evaluated in float64 on the CPU.

Tolerances (max |y - ref| / max |ref| over the network output): fp32
networks 1e-3 -- every convolution is within 1e-4 of its own output (1e-3
for Winograd) and a chain of at most eight layers, with pooling and adds
that do not amplify relative error, stays within their sum; bf16 networks
4e-2 -- each of up to eight layers rounds its output to bf16 (relative
2^-9 ~ 2e-3), the folded batch-norm filters are rounded once more, and the
reference keeps every intermediate in float64, so the rounding adds up over
the chain (twice the single-layer bf16 bar)."""
import numpy as np
import pytest
import torch

import paper_2410_08300_amd as cs
from gpu_util import rel_err, f64, say
from nets import ConvNet, ResNetSmall, randomize_bn

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

DEV = torch.device("cuda:0")


def reference(net, x):
    """The module in float64 on the CPU (the network's own definition)."""
    import copy
    ref = copy.deepcopy(net).to("cpu").double().eval()
    with torch.no_grad():
        return ref(x.double().cpu()).numpy()


@pytest.mark.parametrize("sel", ["default", ("direct", "smm"), ("kn2row", "implicit_precomp_gemm"),
                                 ("winograd", "im2col_gemm"), ("implicit_gemm", "implicit_gemm")])
def test_listing1_network(sel):
    torch.manual_seed(0)
    net = ConvNet().eval()
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
