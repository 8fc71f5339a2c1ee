"""CPU oracle for the forward 2-D convolution -- test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The library's product path never
imports it, and this package imports nothing from the product package.

Contents (all fp64; callers widen fp32 / bf16 data exactly first):

* ``conv2d`` / ``conv2d_points`` -- the definition of the layer (paper,
  Sec. II-B and Sec. IV: every algorithm must reproduce PyTorch's Conv2d
  output), written as plain nested loops in C (``conv2d_oracle.c``).
* ``im2col`` -- the column matrix of the IM2COL / GEMM algorithms (paper,
  Sec. II-B item (a) and Sec. V-B item (c)): the input patches that the GEMM
  reduces over, gathered in plain numpy.
* ``winograd_*`` -- the three transforms of Winograd minimal filtering
  F(2x2, 3x3) (paper, Sec. V-B item (d), which cites Lavin and Gray,
  "Fast Algorithms for Convolutional Neural Networks", 2016), and their
  composition, in plain numpy, following the published definition.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None


def _load():
    global _lib
    if _lib is None:
        path = _build.build(force=False)
        lib = ctypes.CDLL(path)
        i64 = ctypes.c_int64
        dp = ctypes.POINTER(ctypes.c_double)
        lib.oracle_conv2d_f64.argtypes = [dp, dp, dp, dp] + [i64] * 14 + [ctypes.c_int32]
        lib.oracle_conv2d_f64.restype = ctypes.c_int
        lib.oracle_conv2d_points_f64.argtypes = ([dp, dp, dp] + [i64] * 14 + [ctypes.c_int32,
                                                  ctypes.POINTER(ctypes.c_int64), i64, dp])
        lib.oracle_conv2d_points_f64.restype = ctypes.c_int
        _lib = lib
    return _lib


def _pair(v):
    if isinstance(v, (tuple, list)):
        assert len(v) == 2
        return int(v[0]), int(v[1])
    return int(v), int(v)


def output_size(H, W, R, S, stride=1, padding=0, dilation=1):
    """P, Q by the floor formula of PyTorch's Conv2d (the paper's reference
    implementation, Sec. IV); values below 1 mean the layer is invalid."""
    sh, sw = _pair(stride)
    ph, pw = _pair(padding)
    dh, dw = _pair(dilation)
    P = (H + 2 * ph - dh * (R - 1) - 1) // sh + 1
    Q = (W + 2 * pw - dw * (S - 1) - 1) // sw + 1
    return P, Q


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def conv2d(x, w, b=None, stride=1, padding=0, dilation=1, groups=1, relu=False):
    """Full fp64 output y[N, K, P, Q] of the convolution definition."""
    x = _f64(x)
    w = _f64(w)
    N, C, H, W = x.shape
    K, Cg, R, S = w.shape
    if Cg * groups != C:
        raise ValueError("weight has %d input channels per group, input has %d channels, groups=%d"
                         % (Cg, C, groups))
    sh, sw = _pair(stride)
    ph, pw = _pair(padding)
    dh, dw = _pair(dilation)
    P, Q = output_size(H, W, R, S, stride, padding, dilation)
    y = np.empty((N, K, max(P, 0), max(Q, 0)), dtype=np.float64)
    bb = None if b is None else _f64(b)
    rc = _load().oracle_conv2d_f64(_ptr(x), _ptr(w), None if bb is None else _ptr(bb), _ptr(y),
                                   N, C, H, W, K, R, S, sh, sw, ph, pw, dh, dw, groups, int(relu))
    if rc != 0:
        raise ValueError("invalid convolution arguments (oracle status %d)" % rc)
    return y


def conv2d_points(x, w, idx, b=None, stride=1, padding=0, dilation=1, groups=1, relu=False):
    """fp64 values of y at the (n, k, p, q) rows of ``idx`` (shape [npts, 4])."""
    x = _f64(x)
    w = _f64(w)
    idx = np.ascontiguousarray(idx, dtype=np.int64).reshape(-1, 4)
    N, C, H, W = x.shape
    K, Cg, R, S = w.shape
    if Cg * groups != C:
        raise ValueError("weight/input channel mismatch for groups=%d" % groups)
    sh, sw = _pair(stride)
    ph, pw = _pair(padding)
    dh, dw = _pair(dilation)
    out = np.empty(idx.shape[0], dtype=np.float64)
    bb = None if b is None else _f64(b)
    rc = _load().oracle_conv2d_points_f64(
        _ptr(x), _ptr(w), None if bb is None else _ptr(bb), N, C, H, W, K, R, S,
        sh, sw, ph, pw, dh, dw, groups, int(relu),
        idx.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), idx.shape[0], _ptr(out))
    if rc != 0:
        raise ValueError("invalid convolution arguments or point index (oracle status %d)" % rc)
    return out


def im2col(x, R, S, stride=1, padding=0, dilation=1, groups=1):
    """Column matrix of the explicit-GEMM algorithm, fp64.

    Layout [N][G][P*Q][(C/G)*R*S]: one row per output pixel (p*Q + q) of each
    image and group, holding that pixel's receptive field in (c, r, s)
    row-major order (c within the group), zero where the field leaves the
    image.  With Wmat = w.reshape(K, (C/G)*R*S), group g of the output is
    Wmat[g*K/G:(g+1)*K/G] @ col[n, g].T -- the GEMM of Sec. V-B item (c).
    """
    x = _f64(x)
    N, C, H, W = x.shape
    sh, sw = _pair(stride)
    ph, pw = _pair(padding)
    dh, dw = _pair(dilation)
    P, Q = output_size(H, W, R, S, stride, padding, dilation)
    Cg = C // groups
    xp = np.zeros((N, C, H + 2 * ph, W + 2 * pw), dtype=np.float64)
    xp[:, :, ph:ph + H, pw:pw + W] = x
    col = np.empty((N, groups, P * Q, Cg * R * S), dtype=np.float64)
    for g in range(groups):
        for c in range(Cg):
            for r in range(R):
                for s in range(S):
                    h0, w0 = r * dh, s * dw
                    patch = xp[:, g * Cg + c, h0:h0 + sh * (P - 1) + 1:sh, w0:w0 + sw * (Q - 1) + 1:sw]
                    col[:, g, :, (c * R + r) * S + s] = patch.reshape(N, P * Q)
    return col


# Winograd minimal filtering F(2x2, 3x3): the three matrices of Lavin and Gray
# (2016) for the 1-D algorithm F(2, 3), nested for two dimensions.  For input
# tile d (4x4) and filter g (3x3) the 2x2 output tile of the correlation is
#   Y = A^T [ (G g G^T) * (B^T d B) ] A      (* = elementwise product).
WINO_BT = np.array([[1, 0, -1, 0],
                    [0, 1, 1, 0],
                    [0, -1, 1, 0],
                    [0, 1, 0, -1]], dtype=np.float64)
WINO_G = np.array([[1, 0, 0],
                   [0.5, 0.5, 0.5],
                   [0.5, -0.5, 0.5],
                   [0, 0, 1]], dtype=np.float64)
WINO_AT = np.array([[1, 1, 1, 0],
                    [0, 1, -1, -1]], dtype=np.float64)


def winograd_tiles(P, Q):
    """Number of 2x2 output tiles along each axis: ceil(P/2), ceil(Q/2)."""
    return (P + 1) // 2, (Q + 1) // 2


def winograd_filter_transform(w):
    """U[4][4][K][C] = G g_{k,c} G^T for every filter plane (3x3 filters)."""
    w = _f64(w)
    K, C, R, S = w.shape
    if (R, S) != (3, 3):
        raise ValueError("F(2x2,3x3) needs 3x3 filters")
    U = np.empty((4, 4, K, C), dtype=np.float64)
    for k in range(K):
        for c in range(C):
            U[:, :, k, c] = WINO_G @ w[k, c] @ WINO_G.T
    return U


def winograd_input_transform(x, padding=1):
    """V[4][4][T][C] = B^T d B for every 4x4 input tile d.

    Tile t = (n*TP + tp)*TQ + tq covers output rows 2tp, 2tp+1 and columns
    2tq, 2tq+1; its input tile starts at row 2tp - ph and column 2tq - pw and
    reads zero outside the image (this also covers the part of the last tile
    that lies past an odd P or Q).
    """
    x = _f64(x)
    N, C, H, W = x.shape
    ph, pw = _pair(padding)
    P, Q = output_size(H, W, 3, 3, 1, padding, 1)
    TP, TQ = winograd_tiles(P, Q)
    xp = np.zeros((N, C, 2 * TP + 2, 2 * TQ + 2), dtype=np.float64)
    hh, ww = min(H, 2 * TP + 2 - ph), min(W, 2 * TQ + 2 - pw)
    xp[:, :, ph:ph + hh, pw:pw + ww] = x[:, :, :hh, :ww]
    V = np.empty((4, 4, N * TP * TQ, C), dtype=np.float64)
    t = 0
    for n in range(N):
        for tp in range(TP):
            for tq in range(TQ):
                for c in range(C):
                    d = xp[n, c, 2 * tp:2 * tp + 4, 2 * tq:2 * tq + 4]
                    V[:, :, t, c] = WINO_BT @ d @ WINO_BT.T
                t += 1
    return V


def winograd_output_transform(M, N, P, Q, b=None):
    """y[N][K][P][Q] from M[4][4][K][T]: each tile's 2x2 block A^T M A, plus
    bias, keeping only rows < P and columns < Q."""
    M = _f64(M)
    K = M.shape[2]
    TP, TQ = winograd_tiles(P, Q)
    y = np.empty((N, K, P, Q), dtype=np.float64)
    for n in range(N):
        for tp in range(TP):
            for tq in range(TQ):
                t = (n * TP + tp) * TQ + tq
                for k in range(K):
                    blk = WINO_AT @ M[:, :, k, t] @ WINO_AT.T
                    if b is not None:
                        blk = blk + float(b[k])
                    for i in range(2):
                        for j in range(2):
                            p, q = 2 * tp + i, 2 * tq + j
                            if p < P and q < Q:
                                y[n, k, p, q] = blk[i, j]
    return y


def winograd_conv2d(x, w, b=None, padding=1):
    """The whole F(2x2,3x3) algorithm (stride 1, dilation 1, one group):
    transform filters and inputs, multiply elementwise and sum over input
    channels (M[xi][nu] = U[xi][nu] @ V[xi][nu]^T), transform back."""
    x = _f64(x)
    N, C, H, W = x.shape
    P, Q = output_size(H, W, 3, 3, 1, padding, 1)
    U = winograd_filter_transform(w)
    V = winograd_input_transform(x, padding)
    M = np.einsum("abkc,abtc->abkt", U, V)
    return winograd_output_transform(M, N, P, Q, b)
