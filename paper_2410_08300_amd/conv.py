"""Torch-facing convolution call: marshals tensors into the C ABI.

PyTorch supplies device memory (caching allocator) and the current stream;
the convolution itself runs in the HIP library.  Inputs must be CUDA (HIP)
tensors: there is no CPU path.
"""
import ctypes

import torch

from . import _lib

_TORCH_DTYPES = {torch.float32: "f32", torch.bfloat16: "bf16"}


def _desc_for(x, w, b, stride, padding, dilation, groups, relu):
    if x.dim() != 4 or w.dim() != 4:
        raise ValueError("conv2d expects a 4-D NCHW input and a 4-D KCRS weight")
    if x.dtype != w.dtype or (b is not None and b.dtype != x.dtype):
        raise ValueError("input, weight and bias must share one dtype")
    if x.dtype not in _TORCH_DTYPES:
        raise ValueError("unsupported dtype %s (float32 or bfloat16)" % x.dtype)
    N, C, H, W = x.shape
    K, Cg, R, S = w.shape
    if Cg * groups != C:
        raise ValueError("weight expects %d input channels per group but input has %d channels and groups=%d"
                         % (Cg, C, groups))
    if b is not None and (b.dim() != 1 or b.shape[0] != K):
        raise ValueError("bias must hold K=%d values" % K)
    return _lib.make_desc(N, C, H, W, K, R, S, stride, padding, dilation, groups, _TORCH_DTYPES[x.dtype],
                          b is not None, relu)


def conv2d(x, w, b=None, stride=1, padding=0, dilation=1, groups=1, algo="default", relu=False,
           out=None):
    """Forward 2-D convolution with the chosen algorithm.

    Same semantics as ``torch.nn.functional.conv2d`` (zero padding given as
    an int or a pair), plus ``algo`` ("default", "direct", "implicit_gemm",
    "im2col_gemm" / "gemm", "winograd") and an optional fused ReLU.  Raises
    ``Conv2dError`` for any non-OK library status.
    """
    if not (x.is_cuda and w.is_cuda and (b is None or b.is_cuda)):
        raise ValueError("conv2d runs on the GPU only: move input, weight and bias to a HIP device")
    desc = _desc_for(x, w, b, stride, padding, dilation, groups, relu)
    x = x.contiguous()
    w = w.contiguous()
    b = None if b is None else b.contiguous()
    P, Q = _lib.output_shape(desc)
    algo_i = _lib.algo_id(algo)
    with torch.cuda.device(x.device):
        if out is None:
            out = torch.empty((x.shape[0], w.shape[0], P, Q), device=x.device, dtype=x.dtype)
        elif (out.shape != (x.shape[0], w.shape[0], P, Q) or out.dtype != x.dtype or not out.is_contiguous()
              or out.device != x.device):
            raise ValueError("out must be a contiguous %s tensor of shape %s on %s"
                             % (x.dtype, (x.shape[0], w.shape[0], P, Q), x.device))
        nws = _lib.workspace_bytes(desc, algo_i)
        ws = torch.empty(nws, dtype=torch.uint8, device=x.device) if nws else None
        stream = torch.cuda.current_stream(x.device).cuda_stream
        st = _lib.conv2d_raw(x.data_ptr(), w.data_ptr(), None if b is None else b.data_ptr(), out.data_ptr(),
                             desc, algo_i, None if ws is None else ws.data_ptr(), nws, stream)
    if st != _lib.CONV_OK:
        raise _lib.Conv2dError(st, "conv2d(algo=%s)" % _lib.algo_name(algo_i))
    return out


def im2col(x, kernel_size, stride=1, padding=0, dilation=1, groups=1):
    """The column matrix of the IM2COL algorithm, [N][G][P*Q][Cg*R*S]."""
    R, S = _lib._pair(kernel_size)
    N, C, H, W = x.shape
    desc = _lib.make_desc(N, C, H, W, groups, R, S, stride, padding, dilation, groups,
                          _TORCH_DTYPES[x.dtype])
    P, Q = _lib.output_shape(desc)
    x = x.contiguous()
    with torch.cuda.device(x.device):
        col = torch.empty((N, groups, P * Q, (C // groups) * R * S), device=x.device, dtype=x.dtype)
        st = _lib.im2col_raw(x.data_ptr(), col.data_ptr(), desc, torch.cuda.current_stream(x.device).cuda_stream)
    if st != _lib.CONV_OK:
        raise _lib.Conv2dError(st, "conv2d_im2col")
    return col


def winograd_filter_transform(w):
    """U[16][K][C] of F(2x2,3x3) for 3x3 filters w[K][C][3][3]."""
    K, C, R, S = w.shape
    desc = _lib.make_desc(1, C, 4, 4, K, R, S, 1, 1, 1, 1, _TORCH_DTYPES[w.dtype])
    w = w.contiguous()
    with torch.cuda.device(w.device):
        u = torch.empty((16, K, C), device=w.device, dtype=w.dtype)
        st = _lib.wino_filter_raw(w.data_ptr(), u.data_ptr(), desc, torch.cuda.current_stream(w.device).cuda_stream)
    if st != _lib.CONV_OK:
        raise _lib.Conv2dError(st, "conv2d_winograd_filter_transform")
    return u


def winograd_input_transform(x, padding=1):
    """V[16][T][C] of F(2x2,3x3) for input x (3x3 filter, stride 1)."""
    N, C, H, W = x.shape
    desc = _lib.make_desc(N, C, H, W, 1, 3, 3, 1, padding, 1, 1, _TORCH_DTYPES[x.dtype])
    P, Q = _lib.output_shape(desc)
    T = N * ((P + 1) // 2) * ((Q + 1) // 2)
    x = x.contiguous()
    with torch.cuda.device(x.device):
        v = torch.empty((16, T, C), device=x.device, dtype=x.dtype)
        st = _lib.wino_input_raw(x.data_ptr(), v.data_ptr(), desc, torch.cuda.current_stream(x.device).cuda_stream)
    if st != _lib.CONV_OK:
        raise _lib.Conv2dError(st, "conv2d_winograd_input_transform")
    return v


def resolve_algo(x, w, b=None, stride=1, padding=0, dilation=1, groups=1, algo="default", relu=False):
    """The concrete algorithm name "default" stands for on this layer."""
    if algo != "default":
        return "im2col_gemm" if algo == "gemm" else algo
    return _lib.default_algo(_desc_for(x, w, b, stride, padding, dilation, groups, relu))


def pack_filters(w, x_shape, stride=1, padding=0, dilation=1, groups=1, algo="default", bias=False, relu=False):
    """The filter package of ``algo`` for a layer with input shape
    ``x_shape`` (uint8 tensor on w's device); see conv2d_prepacked()."""
    N, C, H, W = x_shape
    K, Cg, R, S = w.shape
    desc = _lib.make_desc(N, C, H, W, K, R, S, stride, padding, dilation, groups, _TORCH_DTYPES[w.dtype], bias,
                          relu)
    algo_i = _lib.algo_id(algo)
    nbytes = _lib.packed_filter_bytes(desc, algo_i)
    w = w.contiguous()
    with torch.cuda.device(w.device):
        pk = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=w.device)
        st = _lib.lib().conv2d_pack_filters(ctypes.c_void_p(w.data_ptr()), ctypes.c_void_p(pk.data_ptr()),
                                            ctypes.byref(desc), algo_i,
                                            ctypes.c_void_p(torch.cuda.current_stream(w.device).cuda_stream))
    if st != _lib.CONV_OK:
        raise _lib.Conv2dError(st, "conv2d_pack_filters(algo=%s)" % _lib.algo_name(algo_i))
    return pk


def conv2d_prepacked(x, packed, w_shape, b=None, stride=1, padding=0, dilation=1, groups=1, algo="default",
                     relu=False, out=None):
    """conv2d with a filter package from pack_filters() (same layer shape
    and algorithm) in place of the filters."""
    if not (x.is_cuda and packed.is_cuda and (b is None or b.is_cuda)):
        raise ValueError("conv2d runs on the GPU only")
    N, C, H, W = x.shape
    K, Cg, R, S = w_shape
    if x.dtype not in _TORCH_DTYPES or (b is not None and b.dtype != x.dtype):
        raise ValueError("input and bias must share a float32 or bfloat16 dtype")
    desc = _lib.make_desc(N, C, H, W, K, R, S, stride, padding, dilation, groups, _TORCH_DTYPES[x.dtype],
                          b is not None, relu)
    x = x.contiguous()
    b = None if b is None else b.contiguous()
    P, Q = _lib.output_shape(desc)
    algo_i = _lib.algo_id(algo)
    with torch.cuda.device(x.device):
        if out is None:
            out = torch.empty((N, K, P, Q), device=x.device, dtype=x.dtype)
        nws = _lib.prepacked_workspace_bytes(desc, algo_i)
        ws = torch.empty(nws, dtype=torch.uint8, device=x.device) if nws else None
        st = _lib.lib().conv2d_prepacked(ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(packed.data_ptr()),
                                         ctypes.c_void_p(0 if b is None else b.data_ptr()),
                                         ctypes.c_void_p(out.data_ptr()), ctypes.byref(desc), algo_i,
                                         ctypes.c_void_p(0 if ws is None else ws.data_ptr()), nws,
                                         ctypes.c_void_p(torch.cuda.current_stream(x.device).cuda_stream))
    if st != _lib.CONV_OK:
        raise _lib.Conv2dError(st, "conv2d_prepacked(algo=%s)" % _lib.algo_name(algo_i))
    return out


def prepare(x, w, b=None, stride=1, padding=0, dilation=1, groups=1, algo="default", relu=False, out=None,
            prepacked=False):
    """(callable, out): a conv2d launch with all arguments marshalled once
    (output, workspace and -- with prepacked=True -- the filter package
    allocated here), for timing and tight loops.  The tensors must stay
    alive and unmoved while the callable is used."""
    if not (x.is_cuda and w.is_cuda and (b is None or b.is_cuda)):
        raise ValueError("conv2d runs on the GPU only")
    desc = _desc_for(x, w, b, stride, padding, dilation, groups, relu)
    if not (x.is_contiguous() and w.is_contiguous() and (b is None or b.is_contiguous())):
        raise ValueError("prepare() needs contiguous tensors")
    P, Q = _lib.output_shape(desc)
    algo_i = _lib.algo_id(resolve_algo(x, w, b, stride, padding, dilation, groups, algo, relu))
    st = _lib.check(desc, algo_i)
    if st != _lib.CONV_OK:
        raise _lib.Conv2dError(st, "conv2d(algo=%s)" % _lib.algo_name(algo_i))
    if out is None:
        out = torch.empty((x.shape[0], w.shape[0], P, Q), device=x.device, dtype=x.dtype)
    pk = None
    if prepacked:
        pk = pack_filters(w, tuple(x.shape), stride, padding, dilation, groups, _lib.algo_name(algo_i),
                          b is not None, relu)
        nws = _lib.prepacked_workspace_bytes(desc, algo_i)
    else:
        nws = _lib.workspace_bytes(desc, algo_i)
    ws = torch.empty(nws, dtype=torch.uint8, device=x.device) if nws else None
    call = _lib.PreparedCall(x.data_ptr(), (pk if prepacked else w).data_ptr(),
                             None if b is None else b.data_ptr(), out.data_ptr(), desc, algo_i,
                             None if ws is None else ws.data_ptr(), nws,
                             torch.cuda.current_stream(x.device).cuda_stream, prepacked=prepacked)
    call.workspace = ws  # keep alive
    call.package = pk
    return call, out


def describe(x_shape, w_shape, stride=1, padding=0, dilation=1, groups=1, dtype=torch.float32, algo="default",
             bias=False, relu=False):
    """How the library runs this layer with ``algo`` (kernels, tiles,
    workspace), as one line of text."""
    N, C, H, W = x_shape
    K, Cg, R, S = w_shape
    desc = _lib.make_desc(N, C, H, W, K, R, S, stride, padding, dilation, groups, _TORCH_DTYPES[dtype], bias, relu)
    return _lib.describe(desc, algo)
