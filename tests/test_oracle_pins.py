"""Pins of the CPU oracle to facts that do not come from the oracle itself.

The oracle is the definition of the layer (paper, Sec. IV: outputs must equal
PyTorch's Conv2d), so it is checked against: an independent brute force on
tiny integer problems (exact), PyTorch's own CPU convolution in fp64 (the
paper's reference implementation, Sec. IV test suite), hand-worked closed
forms (tests/golden/), and algebraic invariants.  The im2col and Winograd
oracles are pinned by reducing exactly to the direct definition.
"""
import itertools
import json
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2410_08300_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def brute_force_int(x, w, b, stride, pad, dil, groups):
    """Exact integer convolution by the definition, in Python ints."""
    N, C, H, Wd = x.shape
    K, Cg, R, S = w.shape
    sh, sw = stride
    ph, pw = pad
    dh, dw = dil
    P = (H + 2 * ph - dh * (R - 1) - 1) // sh + 1
    Q = (Wd + 2 * pw - dw * (S - 1) - 1) // sw + 1
    Kg = K // groups
    y = [[[[0] * Q for _ in range(P)] for _ in range(K)] for _ in range(N)]
    for n in range(N):
        for k in range(K):
            g = k // Kg
            for p in range(P):
                for q in range(Q):
                    acc = int(b[k]) if b is not None else 0
                    for c in range(Cg):
                        for r in range(R):
                            for s in range(S):
                                hh = p * sh - ph + r * dh
                                ww = q * sw - pw + s * dw
                                if 0 <= hh < H and 0 <= ww < Wd:
                                    acc += int(x[n, g * Cg + c, hh, ww]) * int(w[k, c, r, s])
                    y[n][k][p][q] = acc
    return np.array(y, dtype=np.float64)


def tiny_cases(count, seed):
    """Seeded tiny problems covering stride 1-3, pad 0-2, dilation 1-2, filter
    sizes 1-3 per axis and every group count dividing C and K."""
    rng = np.random.default_rng(seed)
    grid = list(itertools.product([1, 2, 3], [0, 1, 2], [1, 2], [1, 2, 3]))
    cases = []
    i = 0
    while len(cases) < count:
        st, pd, dl, R = grid[i % len(grid)]
        i += 1
        S = int(rng.integers(1, 4))
        G = int(rng.choice([1, 2, 4]))
        Cg = int(rng.integers(1, 3)) if G > 1 else int(rng.integers(1, 5))
        Kg = int(rng.integers(1, 3)) if G > 1 else int(rng.integers(1, 5))
        H, Wd = int(rng.integers(1, 7)), int(rng.integers(1, 7))
        N = int(rng.integers(1, 3))
        stride = (st, int(rng.integers(1, 4)))
        pad = (pd, int(rng.integers(0, 3)))
        dil = (dl, int(rng.integers(1, 3)))
        P, Q = oracle.output_size(H, Wd, R, S, stride, pad, dil)
        if P < 1 or Q < 1:
            continue
        x = rng.integers(-3, 4, (N, Cg * G, H, Wd))
        w = rng.integers(-3, 4, (Kg * G, Cg, R, S))
        b = rng.integers(-3, 4, Kg * G) if rng.random() < 0.5 else None
        cases.append((x, w, b, stride, pad, dil, G))
    return cases


def test_bruteforce_exact_on_tiny_integer_problems():
    for x, w, b, stride, pad, dil, G in tiny_cases(240, seed=1):
        ref = brute_force_int(x, w, b, stride, pad, dil, G)
        got = oracle.conv2d(x, w, b, stride, pad, dil, G)
        assert got.shape == ref.shape
        assert np.array_equal(got, ref), (x.shape, w.shape, stride, pad, dil, G)


def test_matches_torch_fp64_reference_on_random_sweep():
    rng = np.random.default_rng(7)
    for x, w, b, stride, pad, dil, G in tiny_cases(120, seed=2):
        xf = rng.standard_normal(x.shape)
        wf = rng.standard_normal(w.shape)
        bf = None if b is None else rng.standard_normal(b.shape)
        got = oracle.conv2d(xf, wf, bf, stride, pad, dil, G)
        ref = torch.nn.functional.conv2d(torch.from_numpy(xf), torch.from_numpy(wf),
                                         None if bf is None else torch.from_numpy(bf),
                                         stride=stride, padding=pad, dilation=dil, groups=G).numpy()
        assert got.shape == ref.shape
        assert np.max(np.abs(got - ref)) <= 1e-12 * max(1.0, np.max(np.abs(ref)))


@pytest.mark.parametrize("workload", W.WORKLOADS)
def test_matches_torch_fp64_on_workload_layers(workload):
    """One layer of each shape family of every workload (batch cut to 1 and
    the image cut to at most 28x28, keeping channels, filter, stride, pad)."""
    layers = W.layers(workload, n=1)
    picks = [layers[0], layers[len(layers) // 2], layers[-1]]
    for L in picks:
        hw = min(L.h, 28)
        Lc = W.Layer(L.name, 1, L.c, hw, hw, L.k, L.r, L.s, L.stride, L.pad, L.dilation, L.groups,
                     L.bias, L.relu, "f32", L.relu_input, L.weight_std_one)
        x, w, b = W.make_tensors(Lc, (5, layers.index(L)))
        got = oracle.conv2d(x.double().numpy(), w.double().numpy(), None if b is None else b.double().numpy(),
                            L.stride, L.pad, L.dilation, L.groups, relu=L.relu)
        ref = torch.nn.functional.conv2d(x.double(), w.double(), None if b is None else b.double(),
                                         stride=L.stride, padding=L.pad, dilation=L.dilation,
                                         groups=L.groups)
        if L.relu:
            ref = ref.clamp(min=0)
        ref = ref.numpy()
        assert np.max(np.abs(got - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_golden_closed_forms():
    with open(os.path.join(GOLDEN, "conv_closed_forms.json")) as f:
        g = json.load(f)
    a = g["all_ones_3x3_pad1"]
    Cg = a["Cg"]
    x = np.ones((1, 2 * Cg, a["H"], a["W"]))
    w = np.ones((4, Cg, 3, 3))
    y = oracle.conv2d(x, w, None, 1, 1, 1, groups=2)
    exp = np.array(a["expected_over_Cg"], dtype=np.float64) * Cg
    for k in range(4):
        assert np.array_equal(y[0, k], exp)
    e = g["integer_example"]
    y = oracle.conv2d(np.array(e["x"], float)[None, None], np.array(e["w"], float)[None, None],
                      np.array([e["b"]], float))
    assert np.array_equal(y[0, 0], np.array(e["y"], float))
    e = g["stride2_pad1_example"]
    y = oracle.conv2d(np.arange(16.0).reshape(1, 1, 4, 4), np.ones((1, 1, 3, 3)), None, 2, 1)
    assert np.array_equal(y[0, 0], np.array(e["y"], float))
    e = g["dilation2_example"]
    y = oracle.conv2d(np.arange(25.0).reshape(1, 1, 5, 5), np.ones((1, 1, 2, 2)), None, 1, 0, 2)
    assert np.array_equal(y[0, 0], np.array(e["y"], float))


def test_identity_and_shifted_delta_kernels():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((2, 5, 9, 7))
    C = 5
    eye = np.zeros((C, C, 1, 1))
    eye[np.arange(C), np.arange(C), 0, 0] = 1.0
    assert np.array_equal(oracle.conv2d(x, eye), x)
    assert np.array_equal(oracle.conv2d(x, eye, stride=2), x[:, :, ::2, ::2])
    for r0 in range(3):
        for s0 in range(3):
            d = np.zeros((C, C, 3, 3))
            d[np.arange(C), np.arange(C), r0, s0] = 1.0
            y = oracle.conv2d(x, d, padding=1)
            # y[p, q] = x[p + r0 - 1, q + s0 - 1], zero outside the image
            xp = np.zeros((2, C, 9 + 2, 7 + 2))
            xp[:, :, 1:10, 1:8] = x
            assert np.array_equal(y, xp[:, :, r0:r0 + 9, s0:s0 + 7])


def test_depthwise_is_per_channel_correlation():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((2, 6, 8, 8))
    w = rng.standard_normal((6, 1, 3, 3))
    y = oracle.conv2d(x, w, None, 2, 1, 1, groups=6)
    for c in range(6):
        yc = oracle.conv2d(x[:, c:c + 1], w[c:c + 1], None, 2, 1, 1)
        assert np.array_equal(y[:, c:c + 1], yc)


def test_linearity_bias_groups_translation():
    rng = np.random.default_rng(5)
    x1, x2 = rng.standard_normal((2, 2, 4, 10, 9))
    w1, w2 = rng.standard_normal((2, 6, 2, 3, 3))
    b = rng.standard_normal(6)
    args = dict(stride=1, padding=1, dilation=1, groups=2)
    y1, y2 = oracle.conv2d(x1, w1, **args), oracle.conv2d(x2, w1, **args)
    tol = 1e-12 * 40
    assert np.max(np.abs(oracle.conv2d(2.5 * x1 - 0.75 * x2, w1, **args) - (2.5 * y1 - 0.75 * y2))) < tol
    assert np.max(np.abs(oracle.conv2d(x1, 2.0 * w1 + w2, **args)
                         - (2.0 * y1 + oracle.conv2d(x1, w2, **args)))) < tol
    assert np.max(np.abs(oracle.conv2d(x1, w1, b, **args) - (y1 + b[None, :, None, None]))) < tol
    # groups: each group of 3 outputs sees only its 2 input channels
    for g in range(2):
        yg = oracle.conv2d(x1[:, 2 * g:2 * g + 2], w1[3 * g:3 * g + 3], stride=1, padding=1)
        assert np.array_equal(y1[:, 3 * g:3 * g + 3], yg)
    # translation: shifting the input by one row shifts the interior of the output
    xs = np.roll(x1, 1, axis=2)
    ys = oracle.conv2d(xs, w1, **args)
    assert np.array_equal(ys[:, :, 2:-1, 1:-1], y1[:, :, 1:-2, 1:-1])


def test_relu_and_points_match_full_output():
    rng = np.random.default_rng(6)
    x = rng.standard_normal((3, 8, 11, 13))
    w = rng.standard_normal((12, 4, 3, 2))
    b = rng.standard_normal(12)
    args = dict(stride=(2, 1), padding=(1, 2), dilation=(1, 2), groups=2)
    y = oracle.conv2d(x, w, b, **args)
    yr = oracle.conv2d(x, w, b, relu=True, **args)
    assert np.array_equal(yr, np.maximum(y, 0.0))
    idx = np.stack(np.meshgrid(*[np.arange(s) for s in y.shape], indexing="ij"), -1).reshape(-1, 4)
    assert np.array_equal(oracle.conv2d_points(x, w, idx, b, **args), y.reshape(-1))
    assert np.array_equal(oracle.conv2d_points(x, w, idx, b, relu=True, **args), yr.reshape(-1))


def test_invalid_shapes_are_rejected():
    x = np.zeros((1, 4, 5, 5))
    with pytest.raises(ValueError):
        oracle.conv2d(x, np.zeros((3, 2, 3, 3)), groups=2)      # K not divisible by G
    with pytest.raises(ValueError):
        oracle.conv2d(x, np.zeros((4, 4, 7, 7)))                # output would be empty
    with pytest.raises(ValueError):
        oracle.conv2d_points(x, np.zeros((4, 4, 3, 3)), [[0, 0, 3, 0]])  # p out of range


def test_im2col_times_weight_equals_direct():
    rng = np.random.default_rng(8)
    for (N, C, H, Wd, K, R, S, st, pd, dl, G) in [(2, 3, 9, 8, 4, 3, 3, 1, 1, 1, 1),
                                                  (1, 4, 10, 11, 6, 3, 2, 2, 1, 2, 2),
                                                  (2, 6, 7, 7, 6, 3, 3, 2, 1, 1, 6),
                                                  (1, 5, 6, 9, 3, 1, 1, 1, 0, 1, 1)]:
        x = rng.standard_normal((N, C, H, Wd))
        w = rng.standard_normal((K, C // G, R, S))
        col = oracle.im2col(x, R, S, st, pd, dl, G)
        P, Q = oracle.output_size(H, Wd, R, S, st, pd, dl)
        Kg = K // G
        wm = w.reshape(K, -1)
        y = np.empty((N, K, P * Q))
        for n in range(N):
            for g in range(G):
                y[n, g * Kg:(g + 1) * Kg] = wm[g * Kg:(g + 1) * Kg] @ col[n, g].T
        ref = oracle.conv2d(x, w, None, st, pd, dl, G)
        assert np.max(np.abs(y.reshape(ref.shape) - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_im2col_entries_by_definition():
    """A few entries of the column matrix of an arange input, by hand: pixel
    (p, q) row, column (c*R + r)*S + s holds x[c, p*s_h - p_h + r*d_h, q*s_w - p_w + s*d_w]."""
    x = np.arange(2 * 4 * 5, dtype=np.float64).reshape(1, 2, 4, 5)
    col = oracle.im2col(x, 3, 3, stride=2, padding=1, dilation=1)
    # P = (4 + 2 - 2 - 1)//2 + 1 = 2, Q = (5 + 2 - 2 - 1)//2 + 1 = 3
    assert col.shape == (1, 1, 6, 18)
    assert col[0, 0, 0, 0] == 0.0                  # (c0, r0, s0) of pixel (0,0) is padding
    assert col[0, 0, 0, 4] == x[0, 0, 0, 0]        # (c0, r1, s1) -> row 0, col 0
    assert col[0, 0, 4, 9 + 8] == x[0, 1, 3, 3]    # pixel (1,1), (c1, r2, s2) -> row 3, col 3
    assert col[0, 0, 5, 9 + 5] == 0.0              # pixel (1,2), (c1, r1, s2) -> col 5 is padding


def test_winograd_1d_worked_example():
    with open(os.path.join(GOLDEN, "winograd_f23_1d.json")) as f:
        g = json.load(f)
    d = np.array(g["d"], float)
    f_ = np.array(g["g"], float)
    m = (oracle.WINO_G @ f_) * (oracle.WINO_BT @ d)
    assert np.array_equal(m, np.array(g["m"]))
    assert np.array_equal(oracle.WINO_AT @ m, np.array(g["y"]))


def test_winograd_2d_integer_tiles_exact():
    rng = np.random.default_rng(9)
    for _ in range(50):
        d = rng.integers(-5, 6, (4, 4)).astype(float)
        f_ = rng.integers(-5, 6, (3, 3)).astype(float)
        U = oracle.WINO_G @ f_ @ oracle.WINO_G.T
        V = oracle.WINO_BT @ d @ oracle.WINO_BT.T
        Y = oracle.WINO_AT @ (U * V) @ oracle.WINO_AT.T
        direct = np.array([[np.sum(d[i:i + 3, j:j + 3] * f_) for j in range(2)] for i in range(2)])
        assert np.array_equal(Y, direct)


@pytest.mark.parametrize("shape", [(2, 5, 8, 8, 6), (1, 3, 7, 7, 4), (2, 4, 5, 9, 3), (1, 2, 1, 1, 2)])
def test_winograd_whole_algorithm_equals_direct(shape):
    """Even and odd output sizes (the last tile of an odd P or Q is partial)."""
    N, C, H, Wd, K = shape
    rng = np.random.default_rng(10)
    x = rng.standard_normal((N, C, H, Wd))
    w = rng.standard_normal((K, C, 3, 3))
    b = rng.standard_normal(K)
    ref = oracle.conv2d(x, w, b, 1, 1, 1)
    got = oracle.winograd_conv2d(x, w, b, padding=1)
    assert np.max(np.abs(got - ref)) <= 1e-12 * np.max(np.abs(ref))
    ref0 = oracle.conv2d(x, w, None, 1, 0, 1) if min(H, Wd) >= 3 else None
    if ref0 is not None:
        got0 = oracle.winograd_conv2d(x, w, None, padding=0)
        assert np.max(np.abs(got0 - ref0)) <= 1e-12 * np.max(np.abs(ref0))
