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
            "conv2d_algo_from_name")


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
