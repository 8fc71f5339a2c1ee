"""GPU checks of conv2d_static_scratch(), the allocation-free variant of
conv2d(): on the same inputs it runs the same kernels with the library's
static scratch as workspace, so its output equals conv2d()'s bit for bit.
Two calls in a row on each case, the second with a smaller input (the
scratch keeps the first call's contents), and layers whose workspace holds
split-K partial sums, repacked planes, filter packages, a column matrix and
Winograd transforms."""
import pytest
import torch

from paper_2410_08300_amd import _lib, workloads as W
from gpu_util import say

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

DEV = torch.device("cuda:0")

# (name, dtype, N first, N second, C, H, W, K, R, stride, pad, bias, algo)
CASES = [
    ("3x3 split-K partials", "bf16", 32, 4, 256, 14, 14, 256, 3, 1, 1, False, "implicit_gemm"),
    ("3x3 stride 2", "bf16", 32, 3, 512, 14, 14, 512, 3, 2, 1, True, "implicit_gemm"),
    ("1x1 repacked stride-2 planes", "bf16", 32, 8, 256, 56, 56, 512, 1, 2, 0, False, "implicit_gemm"),
    ("1x1 split 7x7", "bf16", 32, 2, 2048, 7, 7, 512, 1, 1, 0, True, "implicit_gemm"),
    ("fp32 3x3 package", "f32", 8, 2, 64, 56, 56, 64, 3, 1, 1, True, "implicit_gemm"),
    ("im2col column matrix", "f32", 4, 1, 32, 28, 28, 48, 3, 1, 1, True, "im2col_gemm"),
    ("winograd transforms", "f32", 4, 2, 64, 28, 28, 64, 3, 1, 1, True, "winograd"),
    ("kn2row partial planes", "bf16", 4, 1, 64, 20, 20, 32, 5, 1, 2, True, "kn2row"),
]


def run_pair(case, n):
    name, dt, _, _, c, h, w, k, r, st, pd, bias, algo = case
    tdt = torch.float32 if dt == "f32" else torch.bfloat16
    g = torch.Generator(device=DEV).manual_seed(W.seed_for(55, n, c, k, r))
    x = torch.randn(n, c, h, w, generator=g, device=DEV).to(tdt)
    wt = (torch.randn(k, c, r, r, generator=g, device=DEV) * (2.0 / (c * r * r)) ** 0.5).to(tdt)
    b = (torch.randn(k, generator=g, device=DEV) * 0.1).to(tdt) if bias else None
    desc = _lib.make_desc(n, c, h, w, k, r, r, st, pd, dtype=dt, bias=bias)
    p = (h + 2 * pd - r) // st + 1
    q = (w + 2 * pd - r) // st + 1
    need = _lib.workspace_bytes(desc, algo)
    assert need <= _lib.static_scratch_capacity(), (name, need)
    ws = torch.empty(max(need, 256), dtype=torch.uint8, device=DEV)
    y_ref = torch.full((n, k, p, q), float("nan"), dtype=tdt, device=DEV)
    y = torch.full((n, k, p, q), float("nan"), dtype=tdt, device=DEV)
    stream = torch.cuda.current_stream(DEV).cuda_stream
    bp = b.data_ptr() if b is not None else None
    st0 = _lib.conv2d_raw(x.data_ptr(), wt.data_ptr(), bp, y_ref.data_ptr(), desc, algo, ws.data_ptr(), need,
                          stream)
    st1 = _lib.conv2d_static_scratch_raw(x.data_ptr(), wt.data_ptr(), bp, y.data_ptr(), desc, algo, stream)
    torch.cuda.synchronize()
    assert st0 == _lib.CONV_OK and st1 == _lib.CONV_OK, (name, n, st0, st1)
    return y, y_ref, need


@pytest.mark.parametrize("case", CASES, ids=lambda c: c[0].replace(" ", "-"))
def test_static_scratch_matches_conv2d_twice(case):
    for n in (case[2], case[3]):
        say("case static-scratch", case[0], "N=%d" % n)
        y, y_ref, need = run_pair(case, n)
        assert need > 0
        assert torch.isfinite(y_ref).all()
        assert torch.equal(y, y_ref), "%s N=%d differs from conv2d" % (case[0], n)


def test_static_scratch_refuses_oversized_workspace_on_the_gpu():
    desc = _lib.make_desc(128, 256, 112, 112, 512, 1, 1, 1, 0, 1, 1, "bf16")
    x = torch.zeros(16, device=DEV)
    y = torch.full((16,), 7.0, device=DEV)
    st = _lib.conv2d_static_scratch_raw(x.data_ptr(), x.data_ptr(), None, y.data_ptr(), desc, "im2col_gemm",
                                        torch.cuda.current_stream(DEV).cuda_stream)
    torch.cuda.synchronize()
    assert st == _lib.CONV_ERR_WORKSPACE
    assert bool((y == 7.0).all())
