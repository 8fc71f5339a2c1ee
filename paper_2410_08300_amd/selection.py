"""Per-layer algorithm selection (paper, Sec. IV).

* ``AlgoTable``: an ordered map from a convolution module's qualified name to
  the algorithm it runs.  Swapped modules read it at every call, so editing
  the table changes the algorithm without touching the model.
* ``swap_conv2d(model, selector)``: replaces, in place, every
  ``torch.nn.Conv2d`` with a ``Conv2dSwap`` wrapper.  The selector is one of
  the paper's three kinds -- a single algorithm name for every layer, a list
  indexed by the layer's position among the model's Conv2d modules, or a
  callable that receives the module and returns a name -- or an existing
  ``AlgoTable`` / dict keyed by qualified name.  "torch" keeps a module as it
  is; "default" lets the library pick per call.
* ``select_fastest`` / ``tune``: measured selection -- time every algorithm
  that supports a layer and record the fastest in the table.
* ``AlgoCache``: measured choices keyed by layer shape and persisted as JSON,
  so each shape is timed once per device and deployment; passed as the
  selector of ``swap_conv2d`` it makes every layer "cached": the first call
  of a shape measures, later calls (and later processes that load the file)
  reuse the pick.  "default" is the library's own prediction without any
  timing (a decision tree fitted to measured sweeps, see
  ``conv2d_default_algo``).
"""
import collections
import json

import torch
from torch import nn

from . import _lib
from .conv import conv2d, prepare, pack_filters, conv2d_prepacked, resolve_algo

ALGO_CHOICES = ("default", "direct", "implicit_gemm", "implicit_precomp_gemm", "im2col_gemm", "gemm", "kn2row",
                "smm", "winograd", "torch", "cached")
CONCRETE_ALGOS = ("direct", "implicit_gemm", "implicit_precomp_gemm", "im2col_gemm", "kn2row", "smm", "winograd")


def _canonical(name):
    if not isinstance(name, str) or name not in ALGO_CHOICES:
        raise ValueError("unknown convolution algorithm %r (choose from %s)" % (name, ", ".join(ALGO_CHOICES)))
    return "im2col_gemm" if name == "gemm" else name


def _pair(v):
    return tuple(v) if isinstance(v, (tuple, list)) else (v, v)


class AlgoCache:
    """Measured algorithm choices keyed by layer shape, persisted as JSON.

    A key holds everything the choice depends on: dtype, input N x C x H x W,
    filter K x C/groups x R x S, stride, padding, dilation, groups, bias and
    fused ReLU.  ``select`` returns the recorded algorithm of a shape, or
    times every supported algorithm (``select_fastest``) and records the
    fastest.  The file also names the device the timings were taken on.
    """
    VERSION = 1

    def __init__(self, device=None):
        self.device = device
        self.entries = collections.OrderedDict()   # key -> {"algo": name, "ms": {algo: ms}}

    @staticmethod
    def key(x_shape, w_shape, stride=1, padding=0, dilation=1, groups=1, dtype="f32", bias=False, relu=False):
        n, c, h, w = (int(v) for v in x_shape)
        k, cg, r, s = (int(v) for v in w_shape)
        if c != cg * groups:
            raise ValueError("filter channels %d x groups %d != input channels %d" % (cg, groups, c))
        sh, sw = _pair(stride)
        ph, pw = _pair(padding)
        dh, dw = _pair(dilation)
        return "%s n%d c%d h%d w%d k%d r%d s%d st%dx%d pad%dx%d dil%dx%d g%d bias%d relu%d" % (
            dtype, n, c, h, w, k, r, s, sh, sw, ph, pw, dh, dw, groups, int(bool(bias)), int(bool(relu)))

    @staticmethod
    def key_for(x, w, b=None, stride=1, padding=0, dilation=1, groups=1, relu=False):
        dt = {torch.float32: "f32", torch.bfloat16: "bf16"}.get(x.dtype, str(x.dtype))
        return AlgoCache.key(x.shape, w.shape, stride, padding, dilation, groups, dt, b is not None, relu)

    def __len__(self):
        return len(self.entries)

    def lookup(self, key):
        e = self.entries.get(key)
        return None if e is None else e["algo"]

    def record(self, key, algo, timings=None):
        algo = _canonical(algo)
        if algo not in CONCRETE_ALGOS:
            raise ValueError("a cache entry must name a concrete algorithm, not %r" % algo)
        self.entries[key] = {"algo": algo, "ms": dict(timings or {})}

    def select(self, x, w, b=None, stride=1, padding=0, dilation=1, groups=1, relu=False, warmup=2, reps=5):
        key = self.key_for(x, w, b, stride, padding, dilation, groups, relu)
        algo = self.lookup(key)
        if algo is None:
            algo, timings = select_fastest(x, w, b, stride, padding, dilation, groups, relu, warmup=warmup, reps=reps)
            self.record(key, algo, timings)
        return algo

    def to_json(self):
        return json.dumps({"version": self.VERSION, "device": self.device, "entries": self.entries}, indent=1)

    @classmethod
    def from_json(cls, text):
        d = json.loads(text)
        if d.get("version") != cls.VERSION:
            raise ValueError("unsupported algorithm cache version %r" % d.get("version"))
        c = cls(d.get("device"))
        for k, e in d["entries"].items():
            c.record(k, e["algo"], e.get("ms"))
        return c

    def save(self, path):
        with open(path, "w") as f:
            f.write(self.to_json())

    @classmethod
    def load(cls, path):
        with open(path) as f:
            return cls.from_json(f.read())


class AlgoTable(collections.OrderedDict):
    """qualified module name -> algorithm name.  Entries "cached" resolve per
    call through ``cache`` (an AlgoCache)."""

    cache = None

    def set(self, name, algo):
        self[name] = _canonical(algo)

    def get_algo(self, name):
        return self.get(name, "default")

    def to_json(self):
        return json.dumps(list(self.items()))

    @classmethod
    def from_json(cls, text):
        t = cls()
        for name, algo in json.loads(text):
            t.set(name, algo)
        return t


def _padding_pair(m):
    if isinstance(m.padding, str):
        if m.padding == "valid":
            return (0, 0)
        # "same" with stride 1: symmetric only when the dilated extent is odd.
        pads = []
        for d, k in zip(m.dilation, m.kernel_size):
            total = d * (k - 1)
            if total % 2:
                raise ValueError("padding='same' with an even filter extent needs asymmetric padding, "
                                 "which the library does not offer")
            pads.append(total // 2)
        return tuple(pads)
    return tuple(m.padding)


def _static_check(name, m, algo):
    """Reject, at swap time, picks that cannot run whatever the input shape.
    Every choice but "torch" runs the library, whose convolutions pad with
    zeros only: "default" and "cached" included."""
    if algo == "torch":
        return
    if m.padding_mode != "zeros":
        raise ValueError("%s: padding_mode=%r is not supported by the library (zero padding only); "
                         "select 'torch' for this module" % (name, m.padding_mode))
    if algo in ("default", "cached"):
        return
    if algo == "winograd":
        if tuple(m.kernel_size) != (3, 3) or tuple(m.stride) != (1, 1) or tuple(m.dilation) != (1, 1) \
                or m.groups != 1:
            raise ValueError("%s: winograd F(2x2,3x3) needs a 3x3 filter, stride 1, dilation 1 and groups 1"
                             % name)


class Conv2dSwap(nn.Module):
    """Slim replacement of an nn.Conv2d whose forward calls the HIP library
    with the algorithm the shared ``AlgoTable`` holds for this module."""

    def __init__(self, conv, table, name):
        super().__init__()
        self.in_channels, self.out_channels = conv.in_channels, conv.out_channels
        self.kernel_size, self.stride, self.dilation = conv.kernel_size, conv.stride, conv.dilation
        self.padding = _padding_pair(conv) if conv.padding_mode == "zeros" else conv.padding
        self.groups, self.padding_mode = conv.groups, conv.padding_mode
        self.weight = conv.weight
        self.bias = conv.bias
        self.table = table
        self.name = name
        # The original module serves the "torch" choice.  It is kept out of
        # the module tree (its parameters are this module's parameters), so
        # it is neither listed again as a Conv2d nor moved twice.
        object.__setattr__(self, "_torch_conv", conv)
        # Filter packages (see conv2d_prepacked) for inference calls, keyed by
        # algorithm, input shape and the weight's identity and version; a
        # weight update or a new shape builds a new one.
        self._packages = {}
        self.cache_filters = True

    @property
    def algo(self):
        return self.table.get_algo(self.name)

    def forward(self, x):
        algo = self.algo
        if algo == "torch":
            return self._torch_conv(x)
        if self.padding_mode != "zeros":
            # A table edit can name a library algorithm after the swap.
            raise ValueError("%s: padding_mode=%r is not supported by the library (zero padding only); "
                             "select 'torch' for this module" % (self.name, self.padding_mode))
        w = self.weight
        if algo == "cached":
            if self.table.cache is None:
                raise ValueError("%s: the table has no AlgoCache for its 'cached' entries" % self.name)
            with torch.no_grad():
                algo = self.table.cache.select(x, w.detach(), None if self.bias is None else self.bias.detach(),
                                               self.stride, self.padding, self.dilation, self.groups)
        if not self.cache_filters or (torch.is_grad_enabled() and w.requires_grad) or not x.is_cuda:
            return conv2d(x, w, self.bias, self.stride, self.padding, self.dilation, self.groups, algo=algo)
        algo = resolve_algo(x, w, self.bias, self.stride, self.padding, self.dilation, self.groups, algo)
        key = (algo, tuple(x.shape), x.dtype, w.data_ptr(), w._version)
        pk = self._packages.get(key)
        if pk is None:
            if len(self._packages) >= 4:
                self._packages.clear()
            pk = pack_filters(w.detach(), tuple(x.shape), self.stride, self.padding, self.dilation, self.groups,
                              algo, self.bias is not None)
            self._packages[key] = pk
        return conv2d_prepacked(x, pk, tuple(w.shape), self.bias, self.stride, self.padding, self.dilation,
                                self.groups, algo=algo)

    def extra_repr(self):
        return "%d, %d, kernel_size=%s, stride=%s, padding=%s, groups=%d, algo=%s" % (
            self.in_channels, self.out_channels, self.kernel_size, self.stride, self.padding, self.groups, self.algo)


def _set_submodule(model, name, new):
    parent = model
    parts = name.split(".")
    for p in parts[:-1]:
        parent = getattr(parent, p)
    setattr(parent, parts[-1], new)


def swap_conv2d(model, selector="default"):
    """Replace every nn.Conv2d of ``model`` in place; return the AlgoTable.

    Modules already swapped are re-pointed at the new table.
    """
    all_convs = [(n, m) for n, m in model.named_modules() if isinstance(m, (nn.Conv2d, Conv2dSwap))]
    if isinstance(selector, (list, tuple)) and len(selector) != len(all_convs):
        raise ValueError("selector list has %d entries but the model has %d Conv2d modules"
                         % (len(selector), len(all_convs)))
    table = AlgoTable()
    if isinstance(selector, AlgoCache):
        table.cache = selector
    for idx, (name, m) in enumerate(all_convs):
        base = m._torch_conv if isinstance(m, Conv2dSwap) else m
        if isinstance(selector, AlgoCache):
            algo = "cached"
        elif isinstance(selector, str):
            algo = selector
        elif isinstance(selector, (list, tuple)):
            algo = selector[idx]
        elif isinstance(selector, dict):
            algo = selector.get(name, "default")
        elif callable(selector):
            algo = selector(base)
        else:
            raise ValueError("selector must be a name, a list of names, a callable, a table or an AlgoCache")
        algo = _canonical(algo)
        _static_check(name, base, algo)
        table[name] = algo
    for name, m in all_convs:
        if isinstance(m, Conv2dSwap):
            m.table = table
        else:
            # Modules left on "torch" are wrapped too: the wrapper runs the
            # original module while the table says "torch", so a later table
            # edit can still move them to the library.
            _set_submodule(model, name, Conv2dSwap(m, table, name))
    return table


def supported_algos(x, w, b=None, stride=1, padding=0, dilation=1, groups=1, relu=False):
    """Concrete algorithms the library accepts for this layer."""
    from .conv import _desc_for
    desc = _desc_for(x, w, b, stride, padding, dilation, groups, relu)
    return [a for a in CONCRETE_ALGOS if _lib.check(desc, a) == _lib.CONV_OK]


def time_conv(x, w, b=None, stride=1, padding=0, dilation=1, groups=1, algo="default", relu=False,
              warmup=2, reps=5, launches=10, graph=True, prepacked=False):
    """Median milliseconds per call of the GPU work of one convolution.

    The call's arguments are marshalled once; ``launches`` calls are then
    captured in a HIP graph and replayed between two HIP events (so host
    launch overhead is not counted), median over ``reps`` replays.  With
    ``graph=False`` (or if capture fails) the calls are launched back to back
    instead, which also counts whatever host time the queue cannot hide.
    """
    x, w = x.contiguous(), w.contiguous()
    b = None if b is None else b.contiguous()
    stream = torch.cuda.Stream(x.device)
    with torch.cuda.stream(stream):
        call, out = prepare(x, w, b, stride, padding, dilation, groups, algo=algo, relu=relu, prepacked=prepacked)
        for _ in range(warmup):
            call()
        stream.synchronize()
        g = None
        if graph:
            try:
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=stream):
                    for _ in range(launches):
                        call()
                g.replay()
                stream.synchronize()
            except RuntimeError:
                g = None
        times = []
        for _ in range(reps):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            if g is not None:
                g.replay()
            else:
                for _ in range(launches):
                    call()
            e1.record(stream)
            e1.synchronize()
            times.append(e0.elapsed_time(e1) / launches)
    times.sort()
    return times[len(times) // 2]


def select_fastest(x, w, b=None, stride=1, padding=0, dilation=1, groups=1, relu=False, algos=None,
                   warmup=2, reps=5, prepacked=False):
    """(fastest algorithm, {algorithm: median ms}) over the supported ones."""
    cands = supported_algos(x, w, b, stride, padding, dilation, groups, relu)
    if algos is not None:
        cands = [a for a in cands if a in algos]
    timings = {a: time_conv(x, w, b, stride, padding, dilation, groups, a, relu, warmup, reps,
                            prepacked=prepacked) for a in cands}
    best = min(timings, key=timings.get)
    return best, timings


def tune(model, example_input, table=None, warmup=2, reps=5, cache=None):
    """Measured per-layer selection on a swapped model: capture every
    Conv2dSwap's input with one forward pass, time each supported algorithm
    on it and write the fastest into the table.  With ``cache`` (an
    AlgoCache) shapes already recorded are not timed again, and new ones are
    recorded.  Returns the table."""
    mods = [(n, m) for n, m in model.named_modules() if isinstance(m, Conv2dSwap)]
    if table is None:
        table = mods[0][1].table if mods else AlgoTable()
    captured = {}
    hooks = [m.register_forward_pre_hook(lambda mod, inp, n=n: captured.__setitem__(n, inp[0]))
             for n, m in mods]
    try:
        with torch.no_grad():
            model(example_input)
    finally:
        for h in hooks:
            h.remove()
    with torch.no_grad():
        for n, m in mods:
            if n not in captured or table.get_algo(n) == "torch":
                continue
            if cache is not None:
                best = cache.select(captured[n], m.weight, m.bias, m.stride, m.padding, m.dilation, m.groups,
                                    warmup=warmup, reps=reps)
            else:
                best, _ = select_fastest(captured[n], m.weight, m.bias, m.stride, m.padding, m.dilation,
                                         m.groups, warmup=warmup, reps=reps)
            table[n] = best
    return table
