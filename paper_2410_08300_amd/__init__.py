"""Forward 2-D convolution for AMD MI355X (gfx950) with per-layer choice of
algorithm -- direct, implicit GEMM, implicit precomputed-index GEMM, IM2COL +
GEMM, KN2ROW, SMM and Winograd F(2x2,3x3) --
after the framework of "A Framework to Enable Algorithmic Design Choice
Exploration in DNNs" (arXiv 2410.08300).

The compute runs in hand-written HIP kernels behind a C ABI
(include/convsel.h, libconvsel.so); PyTorch supplies device memory and
streams.
"""
from ._lib import Conv2dError, ALGOS
from .conv import (conv2d, conv2d_prepacked, pack_filters, describe, im2col, winograd_filter_transform,
                   winograd_input_transform)
from .selection import (AlgoTable, AlgoCache, Conv2dSwap, swap_conv2d, select_fastest, tune, time_conv, supported_algos,
                        CONCRETE_ALGOS)
from .backend import swap_backend, Model

__all__ = ["Conv2dError", "ALGOS", "conv2d", "conv2d_prepacked", "pack_filters", "describe", "im2col", "winograd_filter_transform", "winograd_input_transform",
           "AlgoTable", "AlgoCache", "Conv2dSwap", "swap_conv2d", "select_fastest", "tune", "time_conv", "supported_algos",
           "CONCRETE_ALGOS", "swap_backend", "Model"]
