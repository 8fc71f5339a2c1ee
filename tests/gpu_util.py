"""Helpers shared by the GPU tests: tolerances, error metric, oracle calls."""
import numpy as np
import torch

import oracle

ALGOS = ("direct", "implicit_gemm", "implicit_precomp_gemm", "im2col_gemm", "kn2row", "smm", "winograd")


def tolerance(dtype, algo):
    """Max relative error allowed against the fp64 oracle: 1e-4 for fp32
    direct / implicit GEMM (both variants) / IM2COL+GEMM / KN2ROW / SMM, 1e-3
    for fp32 Winograd, 2e-2 for bf16 data (any algorithm)."""
    if dtype in ("bf16", torch.bfloat16):
        return 2e-2
    return 1e-3 if algo == "winograd" else 1e-4


def rel_err(got, ref):
    """max |got - ref| / max |ref| (infinity-norm relative error)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    scale = np.max(np.abs(ref)) if ref.size else 0.0
    diff = np.max(np.abs(got - ref)) if ref.size else 0.0
    return diff / scale if scale > 0 else diff


def f64(t):
    return None if t is None else t.detach().double().cpu().numpy()


def supports(algo, r, s, stride, dilation, groups):
    if algo != "winograd":
        return True
    st = stride if isinstance(stride, tuple) else (stride, stride)
    dl = dilation if isinstance(dilation, tuple) else (dilation, dilation)
    return (r, s) == (3, 3) and st == (1, 1) and dl == (1, 1) and groups == 1


def say(*args):
    print(*args, flush=True)
