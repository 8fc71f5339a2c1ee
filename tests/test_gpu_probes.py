"""The measurement probes that bench.py times beside the step (conv2d_probe_mfma,
conv2d_probe_copy): the copy is bit-exact, including a ragged tail and an
unaligned source, and the MFMA probe writes the sum its operands fix.  Host-side
argument checks run without a GPU."""
import numpy as np
import pytest
import torch

from paper_2410_08300_amd import _lib

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

DEV = torch.device("cuda:0")


def test_copy_probe_is_bit_exact():
    stream = torch.cuda.current_stream(DEV)
    src = torch.randint(0, 256, (1 << 20,), dtype=torch.uint8, device=DEV)
    for offset, nbytes in ((0, 1 << 20), (0, (1 << 20) - 5), (3, 1000)):
        dst = torch.zeros(1 << 20, dtype=torch.uint8, device=DEV)
        _lib.probe_copy(src.data_ptr() + offset, dst.data_ptr(), nbytes, stream.cuda_stream)
        torch.cuda.synchronize()
        assert torch.equal(dst[:nbytes], src[offset:offset + nbytes])
        assert int(dst[nbytes:].abs().sum()) == 0


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_mfma_probe_sum(dtype):
    # Every accumulator element of every lane gets iters * k products
    # a_lane' * b_lane'' summed over the reduction slice; with constant
    # operands per lane the 16 x 8 accumulators of a lane sum to a value
    # that only depends on the operands, so all workgroups agree.
    stream = torch.cuda.current_stream(DEV)
    blocks, iters = 8, 3
    sink = torch.full((blocks * 256,), float("nan"), dtype=torch.float32, device=DEV)
    _lib.probe_mfma(dtype, blocks, iters, sink.data_ptr(), stream.cuda_stream)
    torch.cuda.synchronize()
    s = sink.cpu().numpy().reshape(blocks, 256)
    assert np.isfinite(s).all()
    assert (s == s[0]).all()
    assert (np.abs(s) > 0).all()


def test_probe_arguments_are_checked():
    with pytest.raises(_lib.Conv2dError):
        _lib.probe_mfma("bf16", 0, 1, 0, 0)
