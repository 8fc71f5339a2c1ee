"""Layer shapes of the five benchmark workloads and their seeded synthetic data.

This module holds shapes and random-number generation only -- none of the
convolution arithmetic -- so both the HIP path and the CPU oracle can take
their inputs from it.

Workloads (the paper benchmarks single convolutions and whole CNNs at batch 10,
Sec. V-A; these stand in for them with synthetic data of the same layer
shapes, since no dataset or trained weights are used):

1. ``toy``        one 3->16 3x3 pad-1 layer on a 1x3x32x32 input, fp32, with bias
                  (the first convolution of the paper's Listing 1).
2. ``vgg16``      the 13 3x3 convolutions of VGG-16, batch 8, 224x224, fp32,
                  bias + ReLU after every layer, 2x2 max-pool between blocks.
3. ``resnet50``   the 53 convolutions of ResNet-50 v1.5 (stride on the 3x3 of
                  each stage's first block, 1x1 projection shortcuts), batch
                  32, 224x224, bf16 data with fp32 accumulation, no bias.
4. ``mobilenetv2`` the 52 convolutions of MobileNetV2 (width 1.0) including
                  17 depthwise layers, batch 64, 224x224, fp32, no bias.
5. ``random20``   a seeded 20-layer chain, batch 128, 112x112, bf16, bias +
                  ReLU, channel counts from {64,128,256,512}, kernels from
                  {1,3,5}, strides from {1,2}.

Data recipe: inputs i.i.d. N(0,1) (for layers that follow a ReLU in the
network, the ReLU of such a sample); weights N(0, 2/fan_in) with fan_in =
(C/G)*R*S (Kaiming normal), except the toy layer whose weights are N(0,1);
bias N(0, 0.1^2).  bf16 workloads round the fp32 samples to nearest-even.
Each tensor has its own seed, derived from (workload, layer, tensor, extra).
"""
from dataclasses import dataclass, asdict, field
import math

import numpy as np

BASE_SEED = 2410_08300

WORKLOADS = ("toy", "vgg16", "resnet50", "mobilenetv2", "random20")


@dataclass(frozen=True)
class Layer:
    """One convolution: x is [n, c, h, w], weight [k, c/groups, r, s]."""
    name: str
    n: int
    c: int
    h: int
    w: int
    k: int
    r: int
    s: int
    stride: int = 1
    pad: int = 0
    dilation: int = 1
    groups: int = 1
    bias: bool = False
    relu: bool = False
    dtype: str = "f32"          # "f32" or "bf16"
    relu_input: bool = False    # the input follows a ReLU in the network
    weight_std_one: bool = False

    @property
    def p(self):
        return (self.h + 2 * self.pad - self.dilation * (self.r - 1) - 1) // self.stride + 1

    @property
    def q(self):
        return (self.w + 2 * self.pad - self.dilation * (self.s - 1) - 1) // self.stride + 1

    @property
    def flops(self):
        """2*N*K*(C/G)*R*S*P*Q."""
        return 2 * self.n * self.k * (self.c // self.groups) * self.r * self.s * self.p * self.q

    def compulsory_bytes(self):
        """Bytes every algorithm must move at least once: x, w, bias, y."""
        dt = 4 if self.dtype == "f32" else 2
        elems = (self.n * self.c * self.h * self.w + self.k * (self.c // self.groups) * self.r * self.s
                 + self.n * self.k * self.p * self.q + (self.k if self.bias else 0))
        return dt * elems

    def shape_key(self):
        return (self.n, self.c, self.h, self.w, self.k, self.r, self.s, self.stride, self.pad,
                self.dilation, self.groups, self.bias, self.relu, self.dtype)

    def with_batch(self, n):
        d = asdict(self)
        d["n"] = n
        return Layer(**d)

    def asdict(self):
        return asdict(self)


def toy():
    return [Layer("conv1", 1, 3, 32, 32, 16, 3, 3, 1, 1, bias=True, weight_std_one=True)]


def vgg16(n=8):
    chans = [(3, 64), (64, 64), (64, 128), (128, 128), (128, 256), (256, 256), (256, 256),
             (256, 512), (512, 512), (512, 512), (512, 512), (512, 512), (512, 512)]
    sizes = [224, 224, 112, 112, 56, 56, 56, 28, 28, 28, 14, 14, 14]
    names = ["conv1_1", "conv1_2", "conv2_1", "conv2_2", "conv3_1", "conv3_2", "conv3_3",
             "conv4_1", "conv4_2", "conv4_3", "conv5_1", "conv5_2", "conv5_3"]
    return [Layer(nm, n, c, hw, hw, k, 3, 3, 1, 1, bias=True, relu=True, relu_input=(i > 0))
            for i, (nm, (c, k), hw) in enumerate(zip(names, chans, sizes))]


def resnet50(n=32):
    L = [Layer("stem", n, 3, 224, 224, 64, 7, 7, 2, 3, dtype="bf16")]
    cin, hw = 64, 56
    for si, (width, blocks) in enumerate([(64, 3), (128, 4), (256, 6), (512, 3)]):
        cout = width * 4
        for bi in range(blocks):
            stride = 2 if (bi == 0 and si > 0) else 1
            pre = "layer%d.%d." % (si + 1, bi)
            L.append(Layer(pre + "conv1", n, cin, hw, hw, width, 1, 1, 1, 0, dtype="bf16", relu_input=True))
            L.append(Layer(pre + "conv2", n, width, hw, hw, width, 3, 3, stride, 1, dtype="bf16",
                           relu_input=True))
            hw2 = hw // stride
            L.append(Layer(pre + "conv3", n, width, hw2, hw2, cout, 1, 1, 1, 0, dtype="bf16",
                           relu_input=True))
            if bi == 0:
                L.append(Layer(pre + "downsample", n, cin, hw, hw, cout, 1, 1, stride, 0, dtype="bf16",
                               relu_input=True))
            cin, hw = cout, hw2
    return L


def mobilenetv2(n=64):
    L = [Layer("stem", n, 3, 224, 224, 32, 3, 3, 2, 1)]
    cin, hw = 32, 112
    bidx = 0
    for t, c, reps, s in [(1, 16, 1, 1), (6, 24, 2, 2), (6, 32, 3, 2), (6, 64, 4, 2), (6, 96, 3, 1),
                          (6, 160, 3, 2), (6, 320, 1, 1)]:
        for i in range(reps):
            stride = s if i == 0 else 1
            hid = cin * t
            pre = "block%d." % bidx
            if t != 1:
                L.append(Layer(pre + "expand", n, cin, hw, hw, hid, 1, 1, 1, 0, relu_input=True))
            L.append(Layer(pre + "dw", n, hid, hw, hw, hid, 3, 3, stride, 1, groups=hid,
                           relu_input=True))
            hw2 = (hw + 2 - 3) // stride + 1
            L.append(Layer(pre + "project", n, hid, hw2, hw2, c, 1, 1, 1, 0, relu_input=True))
            cin, hw = c, hw2
            bidx += 1
    L.append(Layer("head", n, cin, hw, hw, 1280, 1, 1, 1, 0))
    return L


def random20(n=128, seed=0):
    """Seeded 20-layer chain: C0, then per layer K, kernel size and stride drawn
    in that order; pad = R // 2; stride forced to 1 if stride 2 would leave an
    output smaller than 7x7; every layer has bias and a ReLU."""
    rng = np.random.default_rng(seed)
    chans, ksz, strides = [64, 128, 256, 512], [1, 3, 5], [1, 2]
    c = int(rng.choice(chans))
    hw = 112
    L = []
    for i in range(20):
        k = int(rng.choice(chans))
        r = int(rng.choice(ksz))
        st = int(rng.choice(strides))
        pad = r // 2
        if st == 2 and (hw + 2 * pad - r) // 2 + 1 < 7:
            st = 1
        L.append(Layer("layer%d" % i, n, c, hw, hw, k, r, r, st, pad, bias=True, relu=True,
                       dtype="bf16", relu_input=(i > 0)))
        hw = (hw + 2 * pad - r) // st + 1
        c = k
    return L


def mixed(seed=0, count=20):
    """Seeded independent layers of mixed kind, for fitting an algorithm-choice
    rule (not a network: each layer stands alone).  Per layer, drawn in this
    order: dtype (bf16 or fp32), kind (dense 70%, depthwise 20%, grouped 10%),
    C and K from {3, 16, 32, 64, 96, 128, 256, 512, 1024} (depthwise: K = C =
    groups; grouped: groups from {2, 4, 32} dividing both), kernel from
    {1, 3, 5, 7} (depthwise {3, 5}), stride from {1, 2}, dilation 1 (2 with
    probability 0.1), H = W from {7, 14, 28, 56, 112, 224}, N from
    {1, 8, 32, 64, 128}, bias and ReLU each with probability 0.5; pad =
    dilation * (R // 2).  A draw is rejected (and redrawn) when the output is
    empty, the input exceeds 2^28 elements, or the layer exceeds 1 TFLOP."""
    rng = np.random.default_rng(seed_for(77, seed))
    chans = [3, 16, 32, 64, 96, 128, 256, 512, 1024]
    out = []
    while len(out) < count:
        dtype = "bf16" if rng.random() < 0.5 else "f32"
        u = rng.random()
        kind = "dense" if u < 0.7 else ("dw" if u < 0.9 else "grouped")
        c = int(rng.choice(chans))
        k = int(rng.choice(chans))
        g = 1
        if kind == "dw":
            k, g = c, c
        elif kind == "grouped":
            g = int(rng.choice([2, 4, 32]))
        r = int(rng.choice([3, 5])) if kind == "dw" else int(rng.choice([1, 3, 5, 7]))
        st = int(rng.choice([1, 2]))
        dl = 2 if rng.random() < 0.1 else 1
        hw = int(rng.choice([7, 14, 28, 56, 112, 224]))
        n = int(rng.choice([1, 8, 32, 64, 128]))
        bias = bool(rng.random() < 0.5)
        relu = bool(rng.random() < 0.5)
        if c % g or k % g:
            continue
        pad = dl * (r // 2)
        L = Layer("mix%d_%d" % (seed, len(out)), n, c, hw, hw, k, r, r, st, pad, dl, g, bias=bias, relu=relu,
                  dtype=dtype)
        if L.p < 1 or L.q < 1 or n * c * hw * hw > (1 << 28) or L.flops > 1e12:
            continue
        out.append(L)
    return out


def layers(workload, n=None, seed=0):
    if workload == "toy":
        return toy()
    if workload == "vgg16":
        return vgg16(8 if n is None else n)
    if workload == "resnet50":
        return resnet50(32 if n is None else n)
    if workload == "mobilenetv2":
        return mobilenetv2(64 if n is None else n)
    if workload == "random20":
        return random20(128 if n is None else n, seed)
    raise ValueError("unknown workload %r" % workload)


def unique_layers(layer_list):
    """First layer of each distinct shape, with the count of its repeats."""
    seen = {}
    for L in layer_list:
        key = L.shape_key()
        if key in seen:
            seen[key][1] += 1
        else:
            seen[key] = [L, 1]
    return [tuple(v) for v in seen.values()]


def seed_for(*key):
    """64-bit seed derived from the base seed and a tuple of small integers."""
    ss = np.random.SeedSequence([BASE_SEED] + [int(k) for k in key])
    return int(ss.generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1))


def _normal(shape, seed, device):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32)


def make_tensors(layer, key, device="cpu"):
    """Seeded (x, w, b) torch tensors of ``layer`` on ``device``.

    ``key`` is a tuple of small integers naming the tensor set (for example
    (workload index, layer index)).  The tensors have the layer's dtype
    (fp32 or bf16, the latter rounded to nearest-even from fp32 samples);
    b is None for layers without bias.
    """
    import torch
    dt = torch.float32 if layer.dtype == "f32" else torch.bfloat16
    x = _normal((layer.n, layer.c, layer.h, layer.w), seed_for(*key, 0), device)
    if layer.relu_input:
        x.clamp_(min=0.0)
    fan_in = (layer.c // layer.groups) * layer.r * layer.s
    w = _normal((layer.k, layer.c // layer.groups, layer.r, layer.s), seed_for(*key, 1), device)
    if not layer.weight_std_one:
        w.mul_(math.sqrt(2.0 / fan_in))
    b = None
    if layer.bias:
        b = _normal((layer.k,), seed_for(*key, 2), device).mul_(0.1)
    return x.to(dt), w.to(dt), (None if b is None else b.to(dt))


def random_points(layer, count, seed):
    """``count`` seeded output coordinates (n, k, p, q) of ``layer``, always
    including the four corners of the first and last output planes."""
    rng = np.random.default_rng(seed_for(99, seed))
    n, k, p, q = layer.n, layer.k, layer.p, layer.q
    pts = np.stack([rng.integers(0, n, count), rng.integers(0, k, count),
                    rng.integers(0, p, count), rng.integers(0, q, count)], axis=1)
    corners = np.array([[nn, kk, pp, qq] for nn, kk in ((0, 0), (n - 1, k - 1))
                        for pp in (0, p - 1) for qq in (0, q - 1)], dtype=np.int64)
    return np.concatenate([corners, pts.astype(np.int64)], axis=0)
