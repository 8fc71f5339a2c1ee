"""Host-side checks of the model executor: lowering of traced networks,
batch-norm folding, the arena plan (no two simultaneously live values share
bytes) and argument errors.  No kernel is launched: planning is host-only
and the filter pointers are never read before binding."""
import itertools

import numpy as np
import pytest
import torch
from torch import nn

import oracle
import paper_2410_08300_amd as cs
from paper_2410_08300_amd import _lib, backend
from nets import ConvStack, ResNetSmall, randomize_bn


def test_listing1_lowering_and_plan():
    m = cs.swap_backend(ConvStack(), ["direct", "smm"])
    assert m.ops == [("conv", "0"), ("maxpool", "2"), ("conv", "3"), ("flatten", "_5")]
    nbytes = m._native.plan(2, 3, 32, 32)
    assert m._native.output_shape() == (2, 32 * 16 * 16)
    d = m._native.describe()
    assert "0 conv v0 -> v1 [2 16 32 32] algo=direct relu" in d
    assert "2 conv v2 -> v3 [2 32 16 16] algo=smm relu offset=-1" in d   # writes the caller's output
    assert nbytes > 0


def test_residual_net_lowering_fuses_and_folds():
    torch.manual_seed(0)
    net = randomize_bn(ResNetSmall(), 1)
    m = cs.swap_backend(net, "default")
    kinds = [k for k, _ in m.ops]
    # BN folded (no bn ops), ReLUs fused (no relu ops), dropout dropped
    assert kinds == ["conv", "maxpool", "conv", "conv", "add", "conv", "conv", "conv", "add", "avgpool",
                     "global_avgpool", "flatten", "linear"]
    nbytes = m._native.plan(3, 3, 64, 64)
    assert m._native.output_shape() == (3, 10)
    d = m._native.describe().splitlines()
    assert d[0].startswith("0 conv v0 -> v1 [3 16 32 32]") and d[0].split()[-2] == "relu"
    assert "add v" in d[4] and " relu " in d[4] + " "
    # Both residual adds are fused into the epilogue of the convolution that
    # produces one operand; that convolution reads the other operand and takes
    # over the add's ReLU, and the add's output is the convolution's output.
    fused = [line for line in d if " add " in " " + line]
    assert len(fused) == 2 and all(line.split()[-2] == "fused" for line in fused)
    for line in fused:
        toks = line.split()
        a, b = int(toks[2][1:]), int(toks[4][1:])
        convs = [c for c in d if c.split()[1] == "conv" and c.split()[4] in ("v%d" % a, "v%d" % b)
                 and " + v" in c]
        assert len(convs) == 1
        ctoks = convs[0].split()
        x = int(ctoks[4][1:])
        y = b if x == a else a
        assert ctoks[ctoks.index("+") + 1] == "v%d" % y and ctoks[ctoks.index("+") + 2] == "relu"
    # Arena plan: values live at the same time never share bytes, all within
    # the arena, 256-byte aligned.  A fused add's output is stored where the
    # convolution's output is, so its reads extend that value's lifetime.
    reads, prod, alias = [], {}, {}
    for i, line in enumerate(d[:-1]):
        toks = line.split()
        ins = [int(t[1:]) for t in toks[2:toks.index("->")] if t.startswith("v")]
        out = int(toks[toks.index("->") + 1][1:])
        reads.append(ins)
        prod[out] = i
        if toks[-2] == "fused":
            alias[out] = [v for v in ins if "+ v" in d[prod[v]]][0]
    last = dict(prod)
    for i, ins in enumerate(reads):
        for v in ins:
            r = alias.get(v, v)
            last[r] = max(last.get(r, -1), i)
    place = {}
    for v in prod:
        off, nb = m._native.placement(v)
        if off >= 0:
            place[v] = (off, nb)
            assert off % 256 == 0 and off + nb <= nbytes
    # flatten's output shares its input's storage
    fl = [i for i, (k, _) in enumerate(m.ops) if k == "flatten"][0]
    assert m._native.placement(fl + 1)[0] == m._native.placement(fl)[0]
    for v, x in alias.items():
        assert place[v] == place[x]
    roots = {v: p for v, p in place.items() if m.ops[prod[v]][0] != "flatten" and v not in alias}
    for a, b in itertools.combinations(roots, 2):
        la, lb = (prod[a], last[a]), (prod[b], last[b])
        if la[0] <= lb[1] and lb[0] <= la[1]:
            (oa, na), (ob, nb2) = roots[a], roots[b]
            assert oa + na <= ob or ob + nb2 <= oa, (a, b)
    # some reuse happened: the activation region is smaller than the sum of the values
    lo = min(o for o, _ in roots.values())
    hi = max(o + nb for o, nb in roots.values())
    assert sum(nb for _, nb in roots.values()) > hi - lo


def test_bn_fold_matches_conv_then_bn():
    torch.manual_seed(2)
    conv = nn.Conv2d(5, 7, 3, 2, 1, bias=True).double()
    bn = randomize_bn(nn.Sequential(nn.BatchNorm2d(7)), 3)[0].double()
    x = torch.randn(2, 5, 9, 8, dtype=torch.float64)
    ref = bn(conv(x)).detach().numpy()
    w, b = backend._fold_bn(conv, bn)
    got = oracle.conv2d(x.numpy(), w.numpy(), b.numpy(), 2, 1)
    assert np.max(np.abs(got - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_unsupported_nodes_and_errors():
    class Sig(nn.Module):
        def __init__(self):
            super().__init__()
            self.c = nn.Conv2d(3, 4, 3)

        def forward(self, x):
            return torch.sigmoid(self.c(x))

    with pytest.raises(NotImplementedError):
        cs.swap_backend(Sig())
    with pytest.raises(NotImplementedError):
        cs.swap_backend(nn.Sequential(nn.Conv2d(3, 4, 3), nn.ReLU(), nn.BatchNorm2d(4)))   # BN not after a conv
    with pytest.raises(ValueError):
        cs.swap_backend(ConvStack(), ["direct"])                                            # list length
    with pytest.raises(ValueError):
        cs.swap_backend(ConvStack(), "torch")
    m = cs.swap_backend(ConvStack())
    with pytest.raises(_lib.Conv2dError):
        m._native.plan(2, 4, 32, 32)                  # 4 input channels, conv1 expects 3
    with pytest.raises(_lib.Conv2dError):
        m._native.forward(1 << 20, 2 << 20, None)     # not bound
    with pytest.raises(_lib.Conv2dError):
        m._native.plan(2, 3, 1, 1)                    # the 2x2 pool has no output
    nm = _lib.NativeModel("f32")
    with pytest.raises(_lib.Conv2dError):
        nm.plan(1, 3, 8, 8)                           # no output set
    with pytest.raises(_lib.Conv2dError):
        nm.relu(5)                                    # no such value
    v = nm.flatten(0)
    nm.set_output(v)
    with pytest.raises(_lib.Conv2dError):
        nm.plan(1, 3, 8, 8)                           # the output is the input itself
    with pytest.raises(ValueError):
        m(torch.randn(2, 3, 32, 32))                  # CPU input


def test_library_exports_model_functions():
    import os
    import re
    hdr = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "convsel_model.h")
    text = re.sub(r"/\*.*?\*/", "", open(hdr).read(), flags=re.S)
    names = sorted(set(re.findall(r"\b(convsel_model_[a-z_]+)\s*\(", text)))
    assert names == sorted(_lib.EXPORTED_MODEL)
    L = _lib.lib()
    for n in names:
        assert hasattr(L, n), n


def _lowered(net, shape):
    m = cs.swap_backend(net, "implicit_gemm")
    m._native.plan(*shape)
    return m._native.describe().splitlines()[:-1]


def test_residual_fusion_only_where_it_is_exact():
    """An add goes into a convolution's epilogue only when that is the same
    computation: the convolution's output is read by nothing else, the
    convolution has no ReLU of its own, and the other operand already
    exists when the convolution runs."""
    class Twice(nn.Module):          # conv output read twice: by the add and by the output add
        def __init__(self):
            super().__init__()
            self.c = nn.Conv2d(8, 8, 3, 1, 1)

        def forward(self, x):
            y = self.c(x)
            return (y + x) + y

    class Relu(nn.Module):           # the conv's own ReLU comes before the add
        def __init__(self):
            super().__init__()
            self.c = nn.Conv2d(8, 8, 3, 1, 1)

        def forward(self, x):
            return torch.relu(self.c(x)) + x

    class Later(nn.Module):          # the other operand is computed after the conv
        def __init__(self):
            super().__init__()
            self.a = nn.Conv2d(8, 8, 3, 1, 1)
            self.b = nn.Conv2d(8, 8, 1)

        def forward(self, x):
            y = self.a(x)
            z = self.b(x)
            return y + z

    class Self(nn.Module):           # y + y
        def __init__(self):
            super().__init__()
            self.c = nn.Conv2d(8, 8, 3, 1, 1)

        def forward(self, x):
            y = self.c(x)
            return y + y

    class Plain(nn.Module):          # fused: conv(x) + x, then ReLU
        def __init__(self):
            super().__init__()
            self.c = nn.Conv2d(8, 8, 3, 1, 1)

        def forward(self, x):
            return torch.relu(self.c(x) + x)

    shape = (2, 8, 6, 6)
    for net in (Twice(), Relu(), Self()):
        d = _lowered(net, shape)
        assert not any(" fused" in line for line in d), (type(net).__name__, d)
        assert not any(" + v" in line for line in d if " conv " in line)
    d = _lowered(Later(), shape)
    # b runs after a, so a cannot take z as its residual, but b can take a's output
    conv_b = [line for line in d if line.startswith("1 conv")][0]
    assert " + v1" in conv_b and any(line.split()[1] == "add" and " fused" in line for line in d)
    d = _lowered(Plain(), shape)
    assert d[0].startswith("0 conv v0 -> v1") and " + v0 relu " in d[0] + " " and d[1].endswith("fused offset=-1")
