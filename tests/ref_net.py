"""Reference evaluation of whole networks for the executor tests.

A network is traced with torch.fx and evaluated node by node in float64 on
the host: every convolution by the oracle (``oracle.conv2d``), everything
else by the plain numpy definitions below (batch norm with inference
statistics, ReLU, max / average pooling with zero-padded windows, global
average pooling, adds, flatten, linear layers).  No torch operator computes
any value, so the executor is judged against the oracle, not against
PyTorch's own kernels.
"""
import operator

import numpy as np
import torch
import torch.nn.functional as F
from torch import nn

import oracle


def _pair(v):
    return tuple(v) if isinstance(v, (tuple, list)) else (v, v)


def np64(t):
    return None if t is None else t.detach().double().cpu().numpy()


def batchnorm(x, bn):
    """(x - mean) / sqrt(var + eps) * gamma + beta per channel."""
    mean, var = np64(bn.running_mean), np64(bn.running_var)
    g = np64(bn.weight) if bn.weight is not None else np.ones_like(mean)
    b = np64(bn.bias) if bn.bias is not None else np.zeros_like(mean)
    scale = g / np.sqrt(var + bn.eps)
    return (x - mean[None, :, None, None]) * scale[None, :, None, None] + b[None, :, None, None]


def pool2d(x, kind, kernel, stride, pad):
    """Max or average over each kh x kw window at stride (sh, sw) of the input
    padded by (ph, pw): padded cells never win a max and count as zeros in
    the average, whose divisor is always kh * kw (count_include_pad).
    Output size floor((H + 2 ph - kh) / sh) + 1 (no ceil mode)."""
    kh, kw = _pair(kernel)
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    n, c, h, w = x.shape
    p = (h + 2 * ph - kh) // sh + 1
    q = (w + 2 * pw - kw) // sw + 1
    fill = -np.inf if kind == "max" else 0.0
    xp = np.full((n, c, h + 2 * ph, w + 2 * pw), fill)
    xp[:, :, ph:ph + h, pw:pw + w] = x
    out = np.empty((n, c, p, q))
    for i in range(p):
        for j in range(q):
            win = xp[:, :, i * sh:i * sh + kh, j * sw:j * sw + kw]
            out[:, :, i, j] = win.max(axis=(2, 3)) if kind == "max" else win.sum(axis=(2, 3)) / (kh * kw)
    return out


def linear(x, lin):
    y = x @ np64(lin.weight).T
    return y + np64(lin.bias) if lin.bias is not None else y


def reference(net, x):
    """The network's output for input x, evaluated as described above."""
    import torch.fx as fx
    gm = fx.symbolic_trace(net.eval())
    mods = dict(gm.named_modules())
    env = {}
    for n in gm.graph.nodes:
        args = [env[a] if isinstance(a, fx.Node) else a for a in n.args]
        if n.op == "placeholder":
            v = np64(x)
        elif n.op == "output":
            return env[n.args[0]]
        elif n.op == "call_module":
            m = mods[n.target]
            a = args[0]
            if isinstance(m, nn.Conv2d):
                assert m.padding_mode == "zeros" and not isinstance(m.padding, str)
                v = oracle.conv2d(a, np64(m.weight), np64(m.bias), _pair(m.stride), _pair(m.padding),
                                  _pair(m.dilation), m.groups, False)
            elif isinstance(m, nn.BatchNorm2d):
                v = batchnorm(a, m)
            elif isinstance(m, nn.ReLU):
                v = np.maximum(a, 0.0)
            elif isinstance(m, nn.MaxPool2d):
                v = pool2d(a, "max", m.kernel_size, m.stride, m.padding)
            elif isinstance(m, nn.AvgPool2d):
                assert m.count_include_pad and not m.ceil_mode
                v = pool2d(a, "avg", m.kernel_size, m.stride, m.padding)
            elif isinstance(m, nn.AdaptiveAvgPool2d):
                assert m.output_size in (1, (1, 1))
                v = a.mean(axis=(2, 3), keepdims=True)
            elif isinstance(m, nn.Linear):
                v = linear(a, m)
            elif isinstance(m, nn.Flatten):
                v = a.reshape(a.shape[0], -1)
            elif isinstance(m, (nn.Dropout, nn.Identity)):
                v = a
            else:
                raise NotImplementedError(type(m).__name__)
        elif n.op == "call_function" and n.target in (F.relu, torch.relu):
            v = np.maximum(args[0], 0.0)
        elif n.op == "call_function" and n.target in (operator.add, operator.iadd, torch.add):
            v = args[0] + args[1]
        elif n.op == "call_function" and n.target is torch.flatten:
            v = args[0].reshape(args[0].shape[0], -1)
        elif n.op == "call_method" and n.target == "relu":
            v = np.maximum(args[0], 0.0)
        else:
            raise NotImplementedError("%s %s" % (n.op, n.target))
        env[n] = v
    raise AssertionError("the traced graph has no output")
