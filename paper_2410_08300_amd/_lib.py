"""ctypes binding of libconvsel.so (the C ABI in include/convsel.h).

Argument marshalling only: every step of the convolution runs in the HIP
library.  Loading fails loudly when the library has not been built; there is
no fallback implementation.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libconvsel.so")

CONV_OK = 0
CONV_ERR_INVALID_ARG = 1
CONV_ERR_UNSUPPORTED = 2
CONV_ERR_WORKSPACE = 3
CONV_ERR_DEVICE = 4

ALGOS = {"default": 0, "direct": 1, "implicit_gemm": 2, "im2col_gemm": 3, "winograd": 4,
         "implicit_precomp_gemm": 5, "kn2row": 6, "smm": 7}
ALGO_NAMES = {v: k for k, v in ALGOS.items()}
DTYPES = {"f32": 0, "bf16": 1}

EXPORTED = ("conv2d_output_shape", "conv2d_check", "conv2d_workspace_bytes", "conv2d_default_algo",
            "conv2d", "conv2d_packed_filter_bytes", "conv2d_pack_filters", "conv2d_prepacked_workspace_bytes",
            "conv2d_prepacked", "conv2d_describe", "conv2d_im2col", "conv2d_winograd_filter_transform",
            "conv2d_winograd_input_transform", "conv2d_status_string", "conv2d_algo_name",
            "conv2d_algo_from_name", "conv2d_static_scratch", "conv2d_static_scratch_capacity",
            "conv2d_probe_mfma", "conv2d_probe_copy")


EXPORTED_MODEL = ("convsel_model_create", "convsel_model_destroy", "convsel_model_conv", "convsel_model_linear",
                  "convsel_model_relu", "convsel_model_pool", "convsel_model_global_avgpool", "convsel_model_add",
                  "convsel_model_flatten", "convsel_model_set_output", "convsel_model_plan",
                  "convsel_model_output_shape", "convsel_model_value_placement", "convsel_model_bind",
                  "convsel_model_forward", "convsel_model_describe")


class Desc(ctypes.Structure):
    """conv2d_desc_t."""
    _fields_ = [("n", ctypes.c_int64), ("c", ctypes.c_int64), ("h", ctypes.c_int64), ("w", ctypes.c_int64),
                ("k", ctypes.c_int64), ("r", ctypes.c_int64), ("s", ctypes.c_int64),
                ("stride_h", ctypes.c_int32), ("stride_w", ctypes.c_int32),
                ("pad_h", ctypes.c_int32), ("pad_w", ctypes.c_int32),
                ("dil_h", ctypes.c_int32), ("dil_w", ctypes.c_int32),
                ("groups", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("has_bias", ctypes.c_int32), ("fuse_relu", ctypes.c_int32)]


class Conv2dError(RuntimeError):
    """A non-OK status from the library; ``status`` holds the code."""

    def __init__(self, status, what=""):
        self.status = status
        msg = status_string(status)
        super().__init__("%s: %s (status %d)" % (what, msg, status) if what else "%s (status %d)" % (msg, status))


_lib = None


def lib():
    """The loaded library (ImportError if it was never built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libconvsel.so is not built (expected at %s); run __graft_entry__.build() "
                              "or python paper_2410_08300_amd/build.py" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        dp = ctypes.POINTER(Desc)
        vp = ctypes.c_void_p
        i32 = ctypes.c_int
        L.conv2d_output_shape.argtypes = [dp, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int64)]
        L.conv2d_output_shape.restype = i32
        L.conv2d_check.argtypes = [dp, i32]
        L.conv2d_check.restype = i32
        L.conv2d_workspace_bytes.argtypes = [dp, i32, ctypes.POINTER(ctypes.c_size_t)]
        L.conv2d_workspace_bytes.restype = i32
        L.conv2d_default_algo.argtypes = [dp]
        L.conv2d_default_algo.restype = i32
        L.conv2d.argtypes = [vp, vp, vp, vp, dp, i32, vp, ctypes.c_size_t, vp]
        L.conv2d.restype = i32
        L.conv2d_static_scratch.argtypes = [vp, vp, vp, vp, dp, i32, vp]
        L.conv2d_static_scratch.restype = i32
        L.conv2d_static_scratch_capacity.argtypes = []
        L.conv2d_static_scratch_capacity.restype = ctypes.c_size_t
        L.conv2d_packed_filter_bytes.argtypes = [dp, i32, ctypes.POINTER(ctypes.c_size_t)]
        L.conv2d_packed_filter_bytes.restype = i32
        L.conv2d_pack_filters.argtypes = [vp, vp, dp, i32, vp]
        L.conv2d_pack_filters.restype = i32
        L.conv2d_prepacked_workspace_bytes.argtypes = [dp, i32, ctypes.POINTER(ctypes.c_size_t)]
        L.conv2d_prepacked_workspace_bytes.restype = i32
        L.conv2d_prepacked.argtypes = [vp, vp, vp, vp, dp, i32, vp, ctypes.c_size_t, vp]
        L.conv2d_prepacked.restype = i32
        L.conv2d_describe.argtypes = [dp, i32, ctypes.c_char_p, ctypes.c_size_t]
        L.conv2d_describe.restype = i32
        L.conv2d_im2col.argtypes = [vp, vp, dp, vp]
        L.conv2d_im2col.restype = i32
        L.conv2d_winograd_filter_transform.argtypes = [vp, vp, dp, vp]
        L.conv2d_winograd_filter_transform.restype = i32
        L.conv2d_winograd_input_transform.argtypes = [vp, vp, dp, vp]
        L.conv2d_winograd_input_transform.restype = i32
        L.conv2d_status_string.argtypes = [i32]
        L.conv2d_status_string.restype = ctypes.c_char_p
        L.conv2d_algo_name.argtypes = [i32]
        L.conv2d_algo_name.restype = ctypes.c_char_p
        L.conv2d_algo_from_name.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_int)]
        L.conv2d_algo_from_name.restype = i32
        L.conv2d_probe_mfma.argtypes = [i32, i32, i32, vp, vp]
        L.conv2d_probe_mfma.restype = i32
        L.conv2d_probe_copy.argtypes = [vp, vp, ctypes.c_size_t, vp]
        L.conv2d_probe_copy.restype = i32
        # model executor (include/convsel_model.h)
        mp = ctypes.c_void_p
        i64 = ctypes.c_int64
        pi32 = ctypes.POINTER(ctypes.c_int32)
        L.convsel_model_create.argtypes = [i32, ctypes.POINTER(ctypes.c_void_p)]
        L.convsel_model_destroy.argtypes = [mp]
        L.convsel_model_destroy.restype = None
        L.convsel_model_conv.argtypes = [mp, i32, i64, i64, i64, i64, i32, i32, i32, i32, i32, i32, i32, i32, vp, vp,
                                         i32, pi32]
        L.convsel_model_linear.argtypes = [mp, i32, i64, i64, i32, vp, vp, i32, pi32]
        L.convsel_model_relu.argtypes = [mp, i32, pi32]
        L.convsel_model_pool.argtypes = [mp, i32, i32, i32, i32, i32, i32, i32, i32, pi32]
        L.convsel_model_global_avgpool.argtypes = [mp, i32, pi32]
        L.convsel_model_add.argtypes = [mp, i32, i32, i32, pi32]
        L.convsel_model_flatten.argtypes = [mp, i32, pi32]
        L.convsel_model_set_output.argtypes = [mp, i32]
        L.convsel_model_plan.argtypes = [mp, i64, i64, i64, i64, ctypes.POINTER(ctypes.c_size_t)]
        L.convsel_model_output_shape.argtypes = [mp, ctypes.POINTER(i64), pi32]
        L.convsel_model_value_placement.argtypes = [mp, i32, ctypes.POINTER(i64), ctypes.POINTER(i64)]
        L.convsel_model_bind.argtypes = [mp, vp, ctypes.c_size_t, vp]
        L.convsel_model_forward.argtypes = [mp, vp, vp, vp]
        L.convsel_model_describe.argtypes = [mp, ctypes.c_char_p, ctypes.c_size_t]
        for n in EXPORTED_MODEL:
            if n != "convsel_model_destroy":
                getattr(L, n).restype = i32
        _lib = L
    return _lib


def _pair(v):
    if isinstance(v, (tuple, list)):
        if len(v) != 2:
            raise ValueError("expected an int or a pair, got %r" % (v,))
        return int(v[0]), int(v[1])
    return int(v), int(v)


def make_desc(n, c, h, w, k, r, s, stride=1, padding=0, dilation=1, groups=1, dtype="f32", bias=False,
              relu=False):
    sh, sw = _pair(stride)
    ph, pw = _pair(padding)
    dh, dw = _pair(dilation)
    return Desc(n, c, h, w, k, r, s, sh, sw, ph, pw, dh, dw, int(groups), DTYPES[dtype], int(bool(bias)),
                int(bool(relu)))


def status_string(status):
    return lib().conv2d_status_string(int(status)).decode()


def algo_id(name):
    out = ctypes.c_int()
    st = lib().conv2d_algo_from_name(name.encode() if isinstance(name, str) else name, ctypes.byref(out))
    if st != CONV_OK:
        raise ValueError("unknown convolution algorithm %r" % (name,))
    return out.value


def algo_name(algo):
    return lib().conv2d_algo_name(int(algo)).decode()


def output_shape(desc):
    p, q = ctypes.c_int64(), ctypes.c_int64()
    st = lib().conv2d_output_shape(ctypes.byref(desc), ctypes.byref(p), ctypes.byref(q))
    if st != CONV_OK:
        raise Conv2dError(st, "conv2d_output_shape")
    return p.value, q.value


def check(desc, algo):
    """Status of conv2d_check (no exception)."""
    return lib().conv2d_check(ctypes.byref(desc), algo_id(algo) if isinstance(algo, str) else int(algo))


def workspace_bytes(desc, algo):
    out = ctypes.c_size_t()
    st = lib().conv2d_workspace_bytes(ctypes.byref(desc), algo_id(algo) if isinstance(algo, str) else int(algo),
                                      ctypes.byref(out))
    if st != CONV_OK:
        raise Conv2dError(st, "conv2d_workspace_bytes")
    return out.value


def packed_filter_bytes(desc, algo):
    out = ctypes.c_size_t()
    st = lib().conv2d_packed_filter_bytes(ctypes.byref(desc), algo_id(algo) if isinstance(algo, str) else int(algo),
                                          ctypes.byref(out))
    if st != CONV_OK:
        raise Conv2dError(st, "conv2d_packed_filter_bytes")
    return out.value


def probe_mfma(dtype, blocks, iters, sink_ptr, stream_ptr):
    """Launches the MFMA-rate probe (conv2d_probe_mfma); dtype "bf16" or "f32"."""
    st = lib().conv2d_probe_mfma(1 if dtype == "bf16" else 0, int(blocks), int(iters), ctypes.c_void_p(sink_ptr),
                                 ctypes.c_void_p(stream_ptr))
    if st != CONV_OK:
        raise Conv2dError(st, "conv2d_probe_mfma")


def probe_copy(src_ptr, dst_ptr, nbytes, stream_ptr):
    """Launches the 16-byte copy probe (conv2d_probe_copy)."""
    st = lib().conv2d_probe_copy(ctypes.c_void_p(src_ptr), ctypes.c_void_p(dst_ptr), ctypes.c_size_t(nbytes),
                                 ctypes.c_void_p(stream_ptr))
    if st != CONV_OK:
        raise Conv2dError(st, "conv2d_probe_copy")


def prepacked_workspace_bytes(desc, algo):
    out = ctypes.c_size_t()
    st = lib().conv2d_prepacked_workspace_bytes(ctypes.byref(desc),
                                                algo_id(algo) if isinstance(algo, str) else int(algo),
                                                ctypes.byref(out))
    if st != CONV_OK:
        raise Conv2dError(st, "conv2d_prepacked_workspace_bytes")
    return out.value


def describe(desc, algo):
    buf = ctypes.create_string_buffer(1024)
    st = lib().conv2d_describe(ctypes.byref(desc), algo_id(algo) if isinstance(algo, str) else int(algo), buf,
                               len(buf))
    if st != CONV_OK:
        raise Conv2dError(st, "conv2d_describe")
    return buf.value.decode()


def default_algo(desc):
    return ALGO_NAMES[lib().conv2d_default_algo(ctypes.byref(desc))]


def conv2d_raw(x_ptr, w_ptr, b_ptr, y_ptr, desc, algo, ws_ptr, ws_bytes, stream):
    """conv2d() on raw device addresses (ints); returns the status."""
    return lib().conv2d(x_ptr, w_ptr, b_ptr, y_ptr, ctypes.byref(desc),
                        algo_id(algo) if isinstance(algo, str) else int(algo), ws_ptr, ws_bytes, stream)


def conv2d_static_scratch_raw(x_ptr, w_ptr, b_ptr, y_ptr, desc, algo, stream):
    """conv2d_static_scratch() on raw device addresses (ints); returns the status."""
    return lib().conv2d_static_scratch(x_ptr, w_ptr, b_ptr, y_ptr, ctypes.byref(desc),
                                       algo_id(algo) if isinstance(algo, str) else int(algo), stream)


def static_scratch_capacity():
    return int(lib().conv2d_static_scratch_capacity())


def im2col_raw(x_ptr, col_ptr, desc, stream):
    return lib().conv2d_im2col(x_ptr, col_ptr, ctypes.byref(desc), stream)


def wino_filter_raw(w_ptr, u_ptr, desc, stream):
    return lib().conv2d_winograd_filter_transform(w_ptr, u_ptr, ctypes.byref(desc), stream)


def wino_input_raw(x_ptr, v_ptr, desc, stream):
    return lib().conv2d_winograd_input_transform(x_ptr, v_ptr, ctypes.byref(desc), stream)


class PreparedCall:
    """A conv2d() (or, with prepacked=True, conv2d_prepacked()) call with
    every argument converted once, for repeated launches with no per-call
    Python work beyond the foreign call itself."""

    def __init__(self, x_ptr, w_ptr, b_ptr, y_ptr, desc, algo, ws_ptr, ws_bytes, stream, prepacked=False):
        self._fn = lib().conv2d_prepacked if prepacked else lib().conv2d
        self._desc = desc  # keep alive: passed by reference
        self._args = (ctypes.c_void_p(x_ptr), ctypes.c_void_p(w_ptr), ctypes.c_void_p(b_ptr or 0),
                      ctypes.c_void_p(y_ptr), ctypes.byref(desc),
                      algo_id(algo) if isinstance(algo, str) else int(algo),
                      ctypes.c_void_p(ws_ptr or 0), ctypes.c_size_t(ws_bytes), ctypes.c_void_p(stream or 0))

    def __call__(self):
        st = self._fn(*self._args)
        if st != CONV_OK:
            raise Conv2dError(st, "conv2d")


class NativeModel:
    """Owner of one convsel_model_t (include/convsel_model.h): the calls
    marshal arguments only; every check and the planning run in the library."""

    def __init__(self, dtype):
        h = ctypes.c_void_p()
        st = lib().convsel_model_create(DTYPES[dtype], ctypes.byref(h))
        if st != CONV_OK:
            raise Conv2dError(st, "convsel_model_create")
        self._h = h
        self.dtype = dtype

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:
            _lib.convsel_model_destroy(h)
            self._h = None

    def _add(self, fn, *args):
        out = ctypes.c_int32()
        st = getattr(lib(), fn)(self._h, *args, ctypes.byref(out))
        if st != CONV_OK:
            raise Conv2dError(st, fn)
        return out.value

    def conv(self, v, c, k, r, s, stride, padding, dilation, groups, algo, w_ptr, b_ptr, relu):
        sh, sw = _pair(stride)
        ph, pw = _pair(padding)
        dh, dw = _pair(dilation)
        return self._add("convsel_model_conv", v, c, k, r, s, sh, sw, ph, pw, dh, dw, groups, algo_id(algo),
                         w_ptr, b_ptr or None, int(bool(relu)))

    def linear(self, v, in_features, out_features, algo, w_ptr, b_ptr, relu):
        return self._add("convsel_model_linear", v, in_features, out_features, algo_id(algo), w_ptr, b_ptr or None,
                         int(bool(relu)))

    def relu(self, v):
        return self._add("convsel_model_relu", v)

    def pool(self, v, kind, kernel, stride, padding):
        kh, kw = _pair(kernel)
        sh, sw = _pair(stride)
        ph, pw = _pair(padding)
        return self._add("convsel_model_pool", v, {"max": 0, "avg": 1}[kind], kh, kw, sh, sw, ph, pw)

    def global_avgpool(self, v):
        return self._add("convsel_model_global_avgpool", v)

    def add(self, a, b, relu):
        return self._add("convsel_model_add", a, b, int(bool(relu)))

    def flatten(self, v):
        return self._add("convsel_model_flatten", v)

    def set_output(self, v):
        st = lib().convsel_model_set_output(self._h, v)
        if st != CONV_OK:
            raise Conv2dError(st, "convsel_model_set_output")

    def plan(self, n, c, h, w):
        nb = ctypes.c_size_t()
        st = lib().convsel_model_plan(self._h, n, c, h, w, ctypes.byref(nb))
        if st != CONV_OK:
            raise Conv2dError(st, "convsel_model_plan")
        return nb.value

    def output_shape(self):
        dims = (ctypes.c_int64 * 4)()
        nd = ctypes.c_int32()
        st = lib().convsel_model_output_shape(self._h, dims, ctypes.byref(nd))
        if st != CONV_OK:
            raise Conv2dError(st, "convsel_model_output_shape")
        return tuple(dims[i] for i in range(nd.value))

    def placement(self, v):
        off, nb = ctypes.c_int64(), ctypes.c_int64()
        st = lib().convsel_model_value_placement(self._h, v, ctypes.byref(off), ctypes.byref(nb))
        if st != CONV_OK:
            raise Conv2dError(st, "convsel_model_value_placement")
        return off.value, nb.value

    def bind(self, arena_ptr, nbytes, stream):
        st = lib().convsel_model_bind(self._h, arena_ptr, nbytes, stream)
        if st != CONV_OK:
            raise Conv2dError(st, "convsel_model_bind")

    def forward(self, x_ptr, y_ptr, stream):
        st = lib().convsel_model_forward(self._h, x_ptr, y_ptr, stream)
        if st != CONV_OK:
            raise Conv2dError(st, "convsel_model_forward")

    def describe(self):
        buf = ctypes.create_string_buffer(1 << 16)
        st = lib().convsel_model_describe(self._h, buf, len(buf))
        if st != CONV_OK:
            raise Conv2dError(st, "convsel_model_describe")
        return buf.value.decode()
