"""Pins of the executor tests' host reference (tests/ref_net.py): its pooling
against hand-worked values, and whole networks against PyTorch's own fp64
CPU evaluation of the same modules (an independent implementation of every
operation)."""
import numpy as np
import torch

import ref_net
from nets import ConvStack, ResNetSmall, randomize_bn


def test_pool_closed_forms():
    x = np.ones((1, 1, 4, 4))
    # 3x3 average, stride 1, pad 1 over ones: padded cells count as zeros,
    # so corners see 4 of 9 cells, edges 6, the interior 9.
    avg = ref_net.pool2d(x, "avg", 3, 1, 1)[0, 0]
    assert np.allclose(avg[0, 0], 4 / 9) and np.allclose(avg[0, 1], 6 / 9) and np.allclose(avg[1, 1], 1.0)
    # Max over a ramp: 2x2 windows at stride 2 take each block's last cell.
    ramp = np.arange(16, dtype=np.float64).reshape(1, 1, 4, 4)
    assert np.array_equal(ref_net.pool2d(ramp, "max", 2, 2, 0)[0, 0], [[5, 7], [13, 15]])
    # Padding never wins a max, even over negative inputs.
    neg = -1.0 - ramp
    assert ref_net.pool2d(neg, "max", 3, 2, 1)[0, 0, 0, 0] == -1.0
    # Output size floor((H + 2p - k) / s) + 1.
    assert ref_net.pool2d(np.zeros((2, 3, 15, 15)), "max", 3, 2, 1).shape == (2, 3, 8, 8)


def test_networks_match_pytorch_fp64():
    torch.manual_seed(0)
    for net, shape in ((ConvStack(), (2, 3, 32, 32)), (randomize_bn(ResNetSmall(), 3), (2, 3, 40, 40))):
        x = torch.randn(*shape)
        ref = ref_net.reference(net, x)
        with torch.no_grad():
            want = net.double()(x.double()).numpy()
        assert ref.shape == want.shape
        assert np.max(np.abs(ref - want)) <= 1e-10 * np.max(np.abs(want))
