"""Whole-model execution (paper, Sec. IV: ``swap_backend`` replaces every
module of a model and returns a model the framework manages).

``swap_backend(module, selector)`` traces an inference network with
``torch.fx`` and lowers it to the library's model executor
(include/convsel_model.h): convolutions (any algorithm, chosen per layer by
the same selector forms as ``swap_conv2d``), linear layers, ReLU, max and
average pooling, global average pooling, residual adds and flattens.  On the
way:

* a BatchNorm2d that directly follows a convolution (its only user) is
  folded into that convolution's filters and bias (inference statistics);
* a ReLU that is the only user of a convolution, linear layer or add is
  fused into that operation's epilogue;
* Dropout and Identity are dropped (inference);
* a linear layer runs as a 1 x 1 convolution with the library's default
  algorithm, or the one a dict selector names for it.

Anything else raises ``NotImplementedError`` at swap time, naming the node.
The returned ``Model`` plans on the first call for each input shape, takes
one device arena from PyTorch's allocator, packs every filter into it, and
then runs each call as one sequence of library launches on PyTorch's
current stream.  Python here only walks the traced graph and marshals
arguments; the network runs in the library.
"""
import operator

import torch
import torch.nn.functional as F
from torch import nn

from . import _lib
from .selection import _canonical, _padding_pair

_RELU_FUNCS = (F.relu, torch.relu)
_ADD_FUNCS = (operator.add, operator.iadd, torch.add)


def _dtype_name(dt):
    if dt == torch.float32:
        return "f32"
    if dt == torch.bfloat16:
        return "bf16"
    raise ValueError("model parameters must be float32 or bfloat16, not %s" % dt)


def _fold_bn(conv, bn):
    """Filters and bias of conv followed by bn (eval statistics), in fp64."""
    w = conv.weight.detach().double()
    b = conv.bias.detach().double() if conv.bias is not None else torch.zeros(w.shape[0], dtype=torch.float64,
                                                                               device=w.device)
    scale = bn.weight.detach().double() / torch.sqrt(bn.running_var.detach().double() + bn.eps)
    w = w * scale.reshape(-1, 1, 1, 1)
    b = (b - bn.running_mean.detach().double()) * scale + bn.bias.detach().double()
    return w, b


class Model:
    """A network lowered to the library's executor.  Call it with an input
    of the traced network's input layout (N x C x H x W, on the GPU, in the
    parameters' dtype)."""

    def __init__(self, native, tensors, dtype, described_ops):
        self._native = native
        self._tensors = tensors      # filters / biases the library reads at bind time
        self.dtype = dtype
        self.ops = described_ops     # (kind, detail) per lowered operation
        self._planned = None
        self._arena = None

    def plan(self, shape):
        """Plan (and bind) for an input shape; returns the arena bytes."""
        n, c, h, w = (int(v) for v in shape)
        nbytes = self._native.plan(n, c, h, w)
        dev = self._tensors[0].device if self._tensors else torch.device("cuda")
        # 256-byte alignment: PyTorch's caching allocator returns at least 512-byte aligned blocks.
        self._arena = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)
        if self._arena.data_ptr() % 256:
            raise RuntimeError("arena is not 256-byte aligned")
        self._native.bind(self._arena.data_ptr(), nbytes, torch.cuda.current_stream(dev).cuda_stream)
        self._planned = (n, c, h, w)
        self.out_shape = self._native.output_shape()
        return nbytes

    def describe(self):
        return self._native.describe()

    def __call__(self, x):
        if not x.is_cuda:
            raise ValueError("the library runs on the GPU: move the input to a HIP device")
        tdt = torch.float32 if self.dtype == "f32" else torch.bfloat16
        if x.dtype != tdt or x.dim() != 4:
            raise ValueError("expected a 4-D %s input, got %s %s" % (tdt, x.dtype, tuple(x.shape)))
        x = x.contiguous()
        if self._planned != tuple(x.shape):
            self.plan(x.shape)
        y = torch.empty(self.out_shape, dtype=tdt, device=x.device)
        self._native.forward(x.data_ptr(), y.data_ptr(), torch.cuda.current_stream(x.device).cuda_stream)
        return y


def _conv_selector(selector, convs):
    """Algorithm per Conv2d (trace order) from the swap_conv2d selector forms."""
    if isinstance(selector, (list, tuple)) and len(selector) != len(convs):
        raise ValueError("selector list has %d entries but the model has %d Conv2d modules"
                         % (len(selector), len(convs)))
    out = {}
    for i, (name, m) in enumerate(convs):
        if isinstance(selector, str):
            a = selector
        elif isinstance(selector, (list, tuple)):
            a = selector[i]
        elif isinstance(selector, dict):
            a = selector.get(name, "default")
        elif callable(selector):
            a = selector(m)
        else:
            raise ValueError("selector must be a name, a list of names, a callable or a dict")
        a = _canonical(a)
        if a in ("torch", "cached"):
            raise ValueError("%s: %r is not available in swap_backend (the whole model runs in the library)"
                             % (name, a))
        out[name] = a
    return out


def swap_backend(module, selector="default"):
    """Lower ``module`` (an inference network, put in eval mode) to the
    library and return the ``Model``.  The module's parameters must be on
    the GPU, all float32 or all bfloat16."""
    import torch.fx as fx

    module = module.eval()
    gm = fx.symbolic_trace(module)
    mods = dict(gm.named_modules())
    params = list(module.parameters())
    if not params:
        raise ValueError("the model has no parameters")
    dtype = _dtype_name(params[0].dtype)
    for p in params:
        if p.dtype != params[0].dtype:
            raise ValueError("all parameters must share one dtype")
    tdt = params[0].dtype
    convs = [(n.target, mods[n.target]) for n in gm.graph.nodes
             if n.op == "call_module" and isinstance(mods[n.target], nn.Conv2d)]
    algos = _conv_selector(selector, convs)

    def is_relu(n):
        return ((n.op == "call_module" and isinstance(mods[n.target], nn.ReLU))
                or (n.op == "call_function" and n.target in _RELU_FUNCS)
                or (n.op == "call_method" and n.target == "relu"))

    def only_user(n):
        users = list(n.users)
        return users[0] if len(users) == 1 else None

    native = _lib.NativeModel(dtype)
    tensors = []
    ops = []
    val = {}          # fx node -> library value number (or alias)
    folded_bn = set()
    fused_relu = set()
    placeholders = [n for n in gm.graph.nodes if n.op == "placeholder"]
    if len(placeholders) != 1:
        raise NotImplementedError("swap_backend takes models with exactly one input")

    def keep(t):
        t = t.detach().to(dtype=tdt).contiguous()
        tensors.append(t)
        return t.data_ptr()

    def fuse_relu_after(n):
        u = only_user(n)
        if u is not None and is_relu(u):
            fused_relu.add(u)
            return True
        return False

    for n in gm.graph.nodes:
        if n.op == "placeholder":
            val[n] = 0
            continue
        if n.op == "output":
            out = n.args[0]
            if not isinstance(out, fx.Node):
                raise NotImplementedError("swap_backend takes models with exactly one tensor output")
            native.set_output(val[out])
            continue
        if n in folded_bn or n in fused_relu:
            val[n] = val[n.args[0]]
            continue
        m = mods.get(n.target) if n.op == "call_module" else None
        if isinstance(m, nn.Conv2d):
            if m.padding_mode != "zeros":
                raise NotImplementedError("%s: padding_mode=%r" % (n.target, m.padding_mode))
            u = only_user(n)
            if u is not None and u.op == "call_module" and isinstance(mods[u.target], nn.BatchNorm2d):
                w, b = _fold_bn(m, mods[u.target])
                folded_bn.add(u)
                relu_from = u
            else:
                w = m.weight
                b = m.bias
                relu_from = n
            relu = fuse_relu_after(relu_from)
            v = native.conv(val[n.args[0]], m.in_channels, m.out_channels, m.kernel_size[0], m.kernel_size[1],
                            m.stride, _padding_pair(m), m.dilation, m.groups, algos[n.target], keep(w),
                            keep(b) if b is not None else None, relu)
            ops.append(("conv", n.target))
        elif isinstance(m, nn.Linear):
            relu = fuse_relu_after(n)
            lin_algo = _canonical(selector.get(n.target, "default")) if isinstance(selector, dict) else "default"
            v = native.linear(val[n.args[0]], m.in_features, m.out_features, lin_algo, keep(m.weight),
                              keep(m.bias) if m.bias is not None else None, relu)
            ops.append(("linear", n.target))
        elif isinstance(m, (nn.Dropout, nn.Identity)):
            v = val[n.args[0]]
        elif isinstance(m, nn.BatchNorm2d):
            raise NotImplementedError("%s: BatchNorm2d is supported only right after a convolution" % n.target)
        elif is_relu(n):
            v = native.relu(val[n.args[0]])
            ops.append(("relu", str(n.target)))
        elif isinstance(m, nn.MaxPool2d):
            if m.ceil_mode or m.dilation not in (1, (1, 1)) or m.return_indices:
                raise NotImplementedError("%s: MaxPool2d with ceil_mode, dilation or indices" % n.target)
            v = native.pool(val[n.args[0]], "max", m.kernel_size, m.stride, m.padding)
            ops.append(("maxpool", n.target))
        elif isinstance(m, nn.AvgPool2d):
            if m.ceil_mode or not m.count_include_pad or m.divisor_override is not None:
                raise NotImplementedError("%s: AvgPool2d with ceil_mode, count_include_pad=False or a divisor"
                                          % n.target)
            v = native.pool(val[n.args[0]], "avg", m.kernel_size, m.stride, m.padding)
            ops.append(("avgpool", n.target))
        elif isinstance(m, nn.AdaptiveAvgPool2d):
            if m.output_size not in (1, (1, 1)):
                raise NotImplementedError("%s: AdaptiveAvgPool2d to %r (only 1x1)" % (n.target, m.output_size))
            v = native.global_avgpool(val[n.args[0]])
            ops.append(("global_avgpool", n.target))
        elif isinstance(m, nn.Flatten) or (n.op == "call_function" and n.target is torch.flatten) \
                or (n.op == "call_method" and n.target == "flatten"):
            start = m.start_dim if m is not None else (n.args[1] if len(n.args) > 1 else n.kwargs.get("start_dim", 0))
            end = m.end_dim if m is not None else (n.args[2] if len(n.args) > 2 else n.kwargs.get("end_dim", -1))
            if start != 1 or end != -1:
                raise NotImplementedError("%s: flatten other than (start_dim=1, end_dim=-1)" % n.name)
            v = native.flatten(val[n.args[0]])
            ops.append(("flatten", n.name))
        elif n.op == "call_function" and n.target in _ADD_FUNCS:
            a, b = n.args[0], n.args[1]
            if not (isinstance(a, fx.Node) and isinstance(b, fx.Node)) or n.kwargs:
                raise NotImplementedError("%s: add of two tensors only" % n.name)
            relu = fuse_relu_after(n)
            v = native.add(val[a], val[b], relu)
            ops.append(("add", n.name))
        else:
            raise NotImplementedError("swap_backend does not support node %s (%s %s)" % (n.name, n.op, n.target))
        val[n] = v
    return Model(native, tensors, dtype, ops)
