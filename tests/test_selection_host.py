"""Selector semantics of swap_conv2d / AlgoTable (paper, Sec. IV) on the CPU.

The HIP call is replaced by a fake backend that evaluates the CPU oracle, so
the swap mechanics are tested without a GPU; the GPU tests run the same
models through the real library."""
import numpy as np
import pytest
import torch
from torch import nn

import oracle
import paper_2410_08300_amd as cs
from paper_2410_08300_amd import selection
from nets import ConvStack


class Deep(nn.Module):
    def __init__(self):
        super().__init__()
        self.stem = nn.Conv2d(3, 8, 5, padding=2)
        self.block = nn.Sequential(nn.Conv2d(8, 8, 3, padding=1, groups=8), nn.ReLU(), nn.Conv2d(8, 12, 1))

    def forward(self, x):
        return self.block(self.stem(x))


@pytest.fixture
def fake_backend(monkeypatch):
    calls = []

    def fake(x, w, b=None, stride=1, padding=0, dilation=1, groups=1, algo="default", relu=False, out=None):
        calls.append(algo)
        y = oracle.conv2d(x.detach().double().numpy(), w.detach().double().numpy(),
                          None if b is None else b.detach().double().numpy(), stride, padding, dilation, groups,
                          relu)
        return torch.from_numpy(y).to(x.dtype)

    monkeypatch.setattr(selection, "conv2d", fake)
    return calls


def test_single_name_list_and_callable(fake_backend):
    torch.manual_seed(0)
    m = ConvStack()
    x = torch.randn(2, 3, 16, 16)
    ref = m(x)
    t = cs.swap_conv2d(m, "direct")
    assert list(t.items()) == [("0", "direct"), ("3", "direct")]
    assert torch.allclose(m(x), ref, atol=1e-5)
    t = cs.swap_conv2d(m, ["implicit_gemm", "gemm"])
    assert list(t.values()) == ["implicit_gemm", "im2col_gemm"]
    fake_backend.clear()
    assert torch.allclose(m(x), ref, atol=1e-5)
    assert fake_backend == ["implicit_gemm", "im2col_gemm"]
    t = cs.swap_conv2d(m, lambda conv: "winograd" if conv.in_channels > 8 else "direct")
    assert list(t.values()) == ["direct", "winograd"]


def test_table_edit_changes_algorithm_without_reswapping(fake_backend):
    m = ConvStack()
    t = cs.swap_conv2d(m, "direct")
    x = torch.randn(1, 3, 8, 8)
    t.set("3", "winograd")
    fake_backend.clear()
    m(x)
    assert fake_backend == ["direct", "winograd"]
    t2 = cs.AlgoTable.from_json(t.to_json())
    assert t2 == t


def test_torch_choice_keeps_pytorch_module(fake_backend):
    torch.manual_seed(1)
    m = Deep()
    x = torch.randn(2, 3, 9, 9)
    ref = m(x)
    t = cs.swap_conv2d(m, ["torch", "direct", "default"])
    assert list(t.values()) == ["torch", "direct", "default"]
    fake_backend.clear()
    assert torch.allclose(m(x), ref, atol=1e-5)
    assert fake_backend == ["direct", "default"]


def test_dict_selector_and_reswap():
    m = Deep()
    t = cs.swap_conv2d(m, {"block.2": "im2col_gemm"})
    assert t["stem"] == "default" and t["block.0"] == "default" and t["block.2"] == "im2col_gemm"
    t2 = cs.swap_conv2d(m, "direct")
    assert all(v == "direct" for v in t2.values())
    assert all(mod.table is t2 for _, mod in m.named_modules() if isinstance(mod, cs.Conv2dSwap))


def test_selector_errors():
    with pytest.raises(ValueError):
        cs.swap_conv2d(ConvStack(), ["direct"])                 # list length mismatch
    with pytest.raises(ValueError):
        cs.swap_conv2d(ConvStack(), "fft")                      # unknown name
    with pytest.raises(ValueError):
        cs.swap_conv2d(Deep(), "winograd")                    # 5x5 stem cannot use F(2x2,3x3)
    with pytest.raises(ValueError):
        cs.swap_conv2d(Deep(), lambda c: 42)
    m = nn.Sequential(nn.Conv2d(3, 4, 3, padding=1, padding_mode="reflect"))
    with pytest.raises(ValueError):
        cs.swap_conv2d(m, "direct")
    assert cs.swap_conv2d(m, "torch")["0"] == "torch"


def test_cpu_tensors_are_refused():
    with pytest.raises(ValueError):
        cs.conv2d(torch.randn(1, 3, 8, 8), torch.randn(4, 3, 3, 3))


def test_algo_cache_measures_each_shape_once_and_persists(fake_backend, monkeypatch, tmp_path):
    timed = []

    def fake_select(x, w, b=None, stride=1, padding=0, dilation=1, groups=1, relu=False, **kw):
        timed.append(tuple(x.shape))
        return "smm", {"smm": 1.0, "direct": 2.0}

    monkeypatch.setattr(selection, "select_fastest", fake_select)
    torch.manual_seed(3)
    m = ConvStack()
    x = torch.randn(2, 3, 16, 16)
    ref = m(x)
    cache = cs.AlgoCache(device="test")
    t = cs.swap_conv2d(m, cache)
    assert list(t.values()) == ["cached", "cached"] and t.cache is cache
    fake_backend.clear()
    assert torch.allclose(m(x), ref, atol=1e-5)
    assert fake_backend == ["smm", "smm"] and len(timed) == 2 and len(cache) == 2
    m(x)                                                   # same shapes: no new timing
    assert len(timed) == 2
    m(torch.randn(1, 3, 16, 16))                           # new batch size: a new shape
    assert len(timed) == 4 and len(cache) == 4
    path = tmp_path / "cache.json"
    cache.save(str(path))
    back = cs.AlgoCache.load(str(path))
    assert back.entries == cache.entries and back.device == "test"
    key = cs.AlgoCache.key_for(x, m[0].weight, m[0].bias, (1, 1), (1, 1), (1, 1), 1)
    assert back.lookup(key) == "smm"
    # a loaded cache answers without timing
    m2 = ConvStack()
    cs.swap_conv2d(m2, back)
    timed.clear()
    m2(x)
    assert timed == []


def test_algo_cache_keys_and_errors():
    k1 = cs.AlgoCache.key((2, 8, 9, 9), (4, 8, 3, 3), 1, 1, 1, 1, "bf16", True, False)
    k2 = cs.AlgoCache.key((2, 8, 9, 9), (4, 8, 3, 3), (1, 1), (1, 1), (1, 1), 1, "bf16", True, False)
    assert k1 == k2
    assert k1 != cs.AlgoCache.key((2, 8, 9, 9), (4, 8, 3, 3), 2, 1, 1, 1, "bf16", True, False)
    assert k1 != cs.AlgoCache.key((2, 8, 9, 9), (4, 8, 3, 3), 1, 1, 1, 1, "f32", True, False)
    with pytest.raises(ValueError):
        cs.AlgoCache.key((2, 8, 9, 9), (4, 3, 3, 3), 1, 1, 1, 1)    # channels do not match groups
    c = cs.AlgoCache()
    with pytest.raises(ValueError):
        c.record(k1, "default")                                     # entries are concrete algorithms
    c.record(k1, "gemm")
    assert c.lookup(k1) == "im2col_gemm"
    with pytest.raises(ValueError):
        cs.AlgoCache.from_json('{"version": 99, "entries": {}}')
    t = cs.AlgoTable()
    t.set("0", "cached")
    m = ConvStack()
    cs.swap_conv2d(m, {"0": "cached"})
    with pytest.raises(ValueError):
        m(torch.randn(1, 3, 8, 8))                                  # "cached" without a cache


def test_non_zero_padding_modes_never_reach_the_library(fake_backend):
    """The library pads with zeros only: every selector form that would run
    a reflect / replicate / circular module on the library is refused at swap
    time, and a later table edit to a library algorithm is refused at call
    time; "torch" keeps such a module working."""
    for mode in ("reflect", "replicate", "circular"):
        def net():
            return nn.Sequential(nn.Conv2d(3, 4, 3, padding=1, padding_mode=mode), nn.Conv2d(4, 4, 1))
        for sel in ("default", "direct", ["default", "direct"], {"1": "direct"}, lambda c: "default",
                    cs.AlgoCache()):
            with pytest.raises(ValueError, match="padding_mode"):
                cs.swap_conv2d(net(), sel)
        m = net()
        x = torch.randn(1, 3, 6, 6)
        ref = m(x)
        t = cs.swap_conv2d(m, {"0": "torch", "1": "direct"})
        fake_backend.clear()
        assert torch.allclose(m(x), ref, atol=1e-5) and fake_backend == ["direct"]
        for algo in ("direct", "default", "cached"):
            t.set("0", algo)
            with pytest.raises(ValueError, match="padding_mode"):
                m(x)
