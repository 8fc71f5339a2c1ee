"""Small inference networks shared by the executor and selection tests: a
plain convolution stack built from a layer specification, and a residual
network with batch norm, pooling and a linear head."""
import torch
from torch import nn

# Two 3x3 convolutions around a 2x2 max-pool, each followed by a ReLU,
# starting from the toy workload's layer (3 -> 16 channels, pad 1, bias).
# Entries: ("conv", in, out, kernel, pad), ("relu",), ("maxpool", k),
# ("flatten",).
TOY_STACK = (("conv", 3, 16, 3, 1), ("relu",), ("maxpool", 2), ("conv", 16, 32, 3, 1), ("relu",),
             ("flatten",))


class ConvStack(nn.Sequential):
    """A sequential network from a layer specification (see TOY_STACK);
    its Conv2d modules are named "0", "3", ... by position."""

    def __init__(self, spec=TOY_STACK):
        layers = []
        for item in spec:
            kind = item[0]
            if kind == "conv":
                _, ci, co, k, pad = item
                layers.append(nn.Conv2d(ci, co, k, padding=pad))
            elif kind == "relu":
                layers.append(nn.ReLU())
            elif kind == "maxpool":
                layers.append(nn.MaxPool2d(item[1], item[1]))
            elif kind == "flatten":
                layers.append(nn.Flatten())
            else:
                raise ValueError("unknown layer kind %r" % (kind,))
        super().__init__(*layers)

    def conv_names(self):
        return [n for n, m in self.named_children() if isinstance(m, nn.Conv2d)]


class Block(nn.Module):
    def __init__(self, c, stride=1):
        super().__init__()
        self.c1 = nn.Conv2d(c, 2 * c if stride == 2 else c, 3, stride, 1, bias=False)
        co = self.c1.out_channels
        self.b1 = nn.BatchNorm2d(co)
        self.c2 = nn.Conv2d(co, co, 3, 1, 1, bias=False)
        self.b2 = nn.BatchNorm2d(co)
        self.down = None
        if stride == 2:
            self.down = nn.Sequential(nn.Conv2d(c, co, 1, 2, bias=False), nn.BatchNorm2d(co))
        self.relu = nn.ReLU(inplace=True)

    def forward(self, x):
        out = self.relu(self.b1(self.c1(x)))
        out = self.b2(self.c2(out))
        idt = x if self.down is None else self.down(x)
        out += idt
        return self.relu(out)


class ResNetSmall(nn.Module):
    """7x7/2 stem + BN + ReLU, 3x3/2 max-pool, two basic blocks (the second
    with a strided 1x1 projection), an average pool, global average pool,
    flatten and a linear head."""

    def __init__(self, classes=10):
        super().__init__()
        self.stem = nn.Conv2d(3, 16, 7, 2, 3, bias=False)
        self.bn = nn.BatchNorm2d(16)
        self.relu = nn.ReLU()
        self.pool = nn.MaxPool2d(3, 2, 1)
        self.layer = nn.Sequential(Block(16), Block(16, 2))
        self.avg = nn.AvgPool2d(3, 1, 1)
        self.gap = nn.AdaptiveAvgPool2d((1, 1))
        self.drop = nn.Dropout(0.5)
        self.fc = nn.Linear(32, classes)

    def forward(self, x):
        x = self.pool(self.relu(self.bn(self.stem(x))))
        x = self.avg(self.layer(x))
        return self.fc(self.drop(torch.flatten(self.gap(x), 1)))


class ConvPlusResidual(nn.Module):
    """One convolution plus the input (or a 1 x 1 projection of it when the
    shapes differ), optionally followed by a ReLU."""

    def __init__(self, c, k, r, stride, pad, relu):
        super().__init__()
        self.proj = None if (c == k and stride == 1) else nn.Conv2d(c, k, 1, stride, 0)
        self.conv = nn.Conv2d(c, k, r, stride, pad)
        self.relu = relu

    def forward(self, x):
        idt = x if self.proj is None else self.proj(x)
        y = self.conv(x) + idt
        return torch.relu(y) if self.relu else y


def randomize_bn(model, seed):
    """Non-trivial running statistics and affine parameters."""
    g = torch.Generator().manual_seed(seed)
    for m in model.modules():
        if isinstance(m, nn.BatchNorm2d):
            c = m.num_features
            m.running_mean.copy_(torch.randn(c, generator=g) * 0.2)
            m.running_var.copy_(torch.rand(c, generator=g) + 0.5)
            m.weight.data.copy_(torch.rand(c, generator=g) + 0.5)
            m.bias.data.copy_(torch.randn(c, generator=g) * 0.1)
    return model.eval()
