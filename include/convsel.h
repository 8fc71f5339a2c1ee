/*
 * convsel -- forward 2-D convolution for AMD MI355X (gfx950) with a per-call
 * choice of algorithm.
 *
 * The operation is the forward pass of a convolution layer as PyTorch's Conv2d
 * defines it (the paper, Sec. IV, requires every algorithm to reproduce that
 * output).  With G groups, Cg = C/G and Kg = K/G:
 *
 *   P = floor((H + 2*pad_h - dil_h*(R-1) - 1) / stride_h) + 1
 *   Q = floor((W + 2*pad_w - dil_w*(S-1) - 1) / stride_w) + 1
 *   y[n,k,p,q] = b[k] + sum_{c<Cg, r<R, s<S}
 *                x[n, (k/Kg)*Cg + c, p*stride_h - pad_h + r*dil_h,
 *                                    q*stride_w - pad_w + s*dil_w] * w[k,c,r,s]
 *
 * where x reads as zero outside the image (cross-correlation, no filter flip),
 * optionally followed by max(0, .) (the ReLU that follows convolutions in the
 * paper's example networks, Sec. IV Listing 1).
 *
 * The algorithms are those the paper lets a user pick per layer (Sec. II-B and
 * Sec. V-B): direct convolution, implicit GEMM (no column matrix is formed),
 * implicit precomputed-index GEMM (the same, with the gather offsets of every
 * reduction index and output pixel precomputed into tables), IM2COL + GEMM
 * (the column matrix is formed in a workspace, then multiplied), KN2ROW (one
 * GEMM of the tap-stacked filters with the input as it lies, then a
 * shift-and-add of the R*S partial planes), SMM (the input zero-padded once,
 * then every output plane accumulated as shifted input planes scaled by
 * single filter values), and Winograd minimal filtering F(2x2, 3x3) for 3x3
 * stride-1 layers.  All of them compute the same function; they differ in
 * speed and workspace.
 *
 * Conventions shared by every entry point:
 *  - Layouts: x is N x C x H x W, w is K x Cg x R x S, b is K values, y is
 *    N x K x P x Q; all dense row-major (NCHW / KCRS), device memory.
 *  - x, w, b and y share one element type (conv_dtype_t).  bf16 data is
 *    multiplied exactly and accumulated in fp32; outputs are rounded to the
 *    element type (round to nearest even for bf16).
 *  - Ownership: the caller owns every buffer (inputs, output, workspace).  The
 *    library allocates no device memory inside any entry point and keeps no
 *    per-call state; the only process state is a lazily filled, thread-safe
 *    table of device properties.
 *  - Streams: `stream` is a hipStream_t passed as void* (NULL = the default
 *    stream).  Work is enqueued and the call returns without synchronising.
 *  - Errors: status codes only.  Every argument, shape, support and workspace
 *    check runs on the host before the first HIP call, so those errors leave
 *    the device untouched.  A failed HIP call (no device, wrong architecture,
 *    launch failure) returns CONV_ERR_DEVICE with the HIP error cleared.
 *  - N == 0 is a valid no-op.  P < 1 or Q < 1 is CONV_ERR_INVALID_ARG.
 */
#ifndef CONVSEL_H
#define CONVSEL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum conv_status {
  CONV_OK = 0,
  CONV_ERR_INVALID_ARG = 1,  /* bad descriptor, NULL pointer, overlap, empty output */
  CONV_ERR_UNSUPPORTED = 2,  /* the algorithm is not defined for this layer */
  CONV_ERR_WORKSPACE = 3,    /* workspace smaller than conv2d_workspace_bytes() */
  CONV_ERR_DEVICE = 4        /* a HIP call failed */
} conv_status_t;

typedef enum conv_algo {
  CONV_ALGO_DEFAULT = 0,        /* the library's own pick, conv2d_default_algo() */
  CONV_ALGO_DIRECT = 1,         /* paper Sec. II-B item (d) */
  CONV_ALGO_IMPLICIT_GEMM = 2,  /* paper Sec. V-B item (b) */
  CONV_ALGO_IM2COL_GEMM = 3,    /* paper Sec. II-B item (a), Sec. V-B item (c) */
  CONV_ALGO_WINOGRAD = 4,       /* paper Sec. V-B item (d): F(2x2,3x3) */
  CONV_ALGO_IMPLICIT_PRECOMP_GEMM = 5,  /* paper Sec. V-B item (a) */
  CONV_ALGO_KN2ROW = 6,         /* paper Sec. II-B item (b) */
  CONV_ALGO_SMM = 7             /* paper Sec. II-B item (c): scalar MM with zero packing */
} conv_algo_t;

typedef enum conv_dtype {
  CONV_F32 = 0,
  CONV_BF16 = 1
} conv_dtype_t;

/* One layer.  Sizes are element counts; w holds K x (C/groups) x R x S. */
typedef struct conv2d_desc {
  int64_t n, c, h, w;
  int64_t k, r, s;
  int32_t stride_h, stride_w;
  int32_t pad_h, pad_w;
  int32_t dil_h, dil_w;
  int32_t groups;
  int32_t dtype;      /* conv_dtype_t */
  int32_t has_bias;   /* 0: b must be NULL; 1: b holds K values */
  int32_t fuse_relu;  /* 1: y = max(0, conv + bias) */
} conv2d_desc_t;

/* Output height and width of the layer (formula above).  INVALID_ARG for a
 * malformed descriptor (non-positive sizes, stride or dilation < 1, negative
 * padding, C or K not divisible by groups, unknown dtype) or an empty output. */
conv_status_t conv2d_output_shape(const conv2d_desc_t* desc, int64_t* p, int64_t* q);

/* OK if `algo` can run this layer; UNSUPPORTED if the algorithm is not defined
 * for it (Winograd needs R = S = 3, stride 1, dilation 1, groups 1; implicit
 * precomputed-index GEMM needs H + 2*pad_h and W + 2*pad_w below 16384, its
 * coordinates being packed as 16-bit halves; KN2ROW needs R*S*K/groups*H*W
 * below 2^31; SMM needs its zero-padded planes of one image below 2^31
 * elements and groups * ceil(K/groups / 16) <= 65535) or for which implicit
 * GEMM finds no tiling;
 * INVALID_ARG as conv2d_output_shape, or for an unknown algo value. */
conv_status_t conv2d_check(const conv2d_desc_t* desc, conv_algo_t algo);

/* Device workspace, in bytes, that conv2d() needs for this layer and algo.
 *  - direct: 0.
 *  - implicit GEMM: the filters repacked per call into the kernel's layout
 *    (K padded to the tile, channels padded to the chunk: at most a few MB
 *    for common layers), plus, for layers whose output tiles alone would
 *    leave compute units idle, S*N*K*P*Q fp32 partial sums of a channel
 *    split over S <= 8 workgroups (summed by a second, deterministic kernel).
 *  - implicit precomputed-index GEMM: its package (zero-padded filters, one
 *    8-byte table entry per reduction index and per output pixel of a launch).
 *  - IM2COL + GEMM and Winograd: the column matrix / transformed tiles, built
 *    for batches of images so the figure is capped near 1 GiB unless one
 *    image alone needs more.
 *  - KN2ROW: the tap-stacked filters plus R*S*K*H*W fp32 partial planes per
 *    image; SMM: the repacked filters plus the zero-padded input
 *    (C x ((P-1)*stride_h + (R-1)*dil_h + 1) x ((Q-1)*stride_w + (S-1)*dil_w + 1)
 *    per image); both batched over images with the same cap.
 * Same errors as conv2d_check. */
conv_status_t conv2d_workspace_bytes(const conv2d_desc_t* desc, conv_algo_t algo, size_t* bytes);

/* The concrete algorithm CONV_ALGO_DEFAULT resolves to for this layer: the
 * library's prediction of the fastest algorithm without timing anything (the
 * "default" selector of Sec. IV, playing the part of the heuristic "guess"
 * of Sec. V-B).  A decision tree over shape features (dtype, depthwise,
 * taps, stride, log2 of C/groups, K/groups, N*P*Q and P*Q, Winograd
 * eligibility, dilation, grouping), fitted offline to measured timings of
 * every algorithm on random layers, ranks the algorithms; the first one
 * that supports the layer is returned.  Host only, deterministic.  Returns
 * CONV_ALGO_DEFAULT itself only for an invalid descriptor. */
conv_algo_t conv2d_default_algo(const conv2d_desc_t* desc);

/* y = conv(x, w) (+ b) (then ReLU) with the chosen algorithm, enqueued on
 * `stream`.  x, w, y (and b when has_bias) must be non-NULL device pointers
 * (any element alignment); y must not overlap x, w, b or the workspace.  A
 * workspace, when one is needed, must be 256-byte aligned (INVALID_ARG
 * otherwise); it may be NULL when the required size is 0.  Returns
 * INVALID_ARG / UNSUPPORTED / WORKSPACE before touching the device, DEVICE
 * if a HIP call fails. */
conv_status_t conv2d(const void* x, const void* w, const void* b, void* y, const conv2d_desc_t* desc,
                     conv_algo_t algo, void* workspace, size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): conv2d()
 * without the workspace arguments.  Its workspace is a library-owned static
 * device array of conv2d_static_scratch_capacity() bytes (32 MiB), one per
 * GPU, held until the process ends; the call itself allocates nothing and
 * runs the same kernels as conv2d(), so the results are identical.
 * Returns WORKSPACE (before any HIP call) when conv2d_workspace_bytes() of
 * the layer and algo exceeds the capacity; otherwise as conv2d().  Every
 * call on one GPU shares that GPU's array: calls that may run at the same
 * time on one GPU (different streams, host threads) race and must be
 * serialised by the caller; nothing in the array needs to start at zero. */
conv_status_t conv2d_static_scratch(const void* x, const void* w, const void* b, void* y, const conv2d_desc_t* desc,
                                    conv_algo_t algo, void* stream);
size_t conv2d_static_scratch_capacity(void);

/* Filter packages.  Implicit GEMM and Winograd first rearrange the filters
 * (implicit GEMM: into its tile layout, zero-padded; implicit precomputed-
 * index GEMM: zero-padded filters plus its index tables; KN2ROW: the
 * tap-stacked filter matrix; SMM: blocks of 8 or 16 output channels with the
 * channels innermost; Winograd: the filter transform U below); conv2d()
 * redoes that in its workspace on every call.
 * An inference caller whose filters do not change can build the package
 * once and call conv2d_prepacked() instead, which then runs only the work
 * that depends on the input.  For direct and IM2COL + GEMM the package is a
 * copy of the filters.
 *  - conv2d_packed_filter_bytes: size of the package.
 *  - conv2d_pack_filters: writes it (`packed` 256-byte aligned, not
 *    overlapping w; enqueued on `stream`).  Same errors as conv2d_check,
 *    INVALID_ARG for NULL / misaligned / overlapping pointers.
 *  - conv2d_prepacked_workspace_bytes: workspace of conv2d_prepacked()
 *    (conv2d's workspace minus the package).
 *  - conv2d_prepacked: as conv2d() with the package (256-byte aligned) in
 *    place of w; same algorithm and descriptor as when the package was
 *    built. */
conv_status_t conv2d_packed_filter_bytes(const conv2d_desc_t* desc, conv_algo_t algo, size_t* bytes);
conv_status_t conv2d_pack_filters(const void* w, void* packed, const conv2d_desc_t* desc, conv_algo_t algo,
                                  void* stream);
conv_status_t conv2d_prepacked_workspace_bytes(const conv2d_desc_t* desc, conv_algo_t algo, size_t* bytes);
conv_status_t conv2d_prepacked(const void* x, const void* packed, const void* b, void* y,
                               const conv2d_desc_t* desc, conv_algo_t algo, void* workspace, size_t workspace_bytes,
                               void* stream);

/* One line describing how conv2d() runs this layer with `algo` (the kernels
 * it launches, tile and grid, workspace sizes), written NUL-terminated into
 * buf (truncated to len - 1 characters).  Host only. */
conv_status_t conv2d_describe(const conv2d_desc_t* desc, conv_algo_t algo, char* buf, size_t len);

/* The column matrix of the IM2COL + GEMM algorithm for all N images: col is
 * N x G x (P*Q) x (Cg*R*S), element [n][g][p*Q+q][(c*R + r)*S + s] =
 * x[n, g*Cg + c, p*stride_h - pad_h + r*dil_h, q*stride_w - pad_w + s*dil_w]
 * (zero outside the image), in the layer's dtype.  A pure gather: results
 * are bit-exact copies of input elements.  Same argument rules as conv2d. */
conv_status_t conv2d_im2col(const void* x, void* col, const conv2d_desc_t* desc, void* stream);

/* Winograd F(2x2,3x3) transforms (Lavin and Gray 2016, the algorithm the
 * paper's Winograd variant names, Sec. V-B item (d)).  Only for layers where
 * conv2d_check(desc, CONV_ALGO_WINOGRAD) is OK.
 *  - filter: U is 16 x K x C, U[xi*4+nu][k][c] = (G w[k,c] G^T)[xi][nu],
 *    computed in fp32 and stored in the layer's dtype.
 *  - input:  V is 16 x T x C with T = N*ceil(P/2)*ceil(Q/2) tiles,
 *    tile t = (n*ceil(P/2) + tp)*ceil(Q/2) + tq, V[xi*4+nu][t][c] =
 *    (B^T d B)[xi][nu] where d is the 4x4 input patch at row 2tp - pad_h,
 *    column 2tq - pad_w (zero outside the image); fp32 math, layer dtype. */
conv_status_t conv2d_winograd_filter_transform(const void* w, void* u, const conv2d_desc_t* desc,
                                               void* stream);
conv_status_t conv2d_winograd_input_transform(const void* x, void* v, const conv2d_desc_t* desc,
                                              void* stream);

/* Measurement probes for the roofline denominators (no convolution):
 *  - conv2d_probe_mfma launches `blocks` workgroups of four waves; every
 *    wave issues `iters` rounds of eight independent 32x32 MFMAs with the
 *    operands in registers (CONV_BF16: v_mfma_f32_32x32x16_bf16, 32768
 *    flops each; CONV_F32: v_mfma_f32_32x32x2_f32, 4096 flops each), then
 *    writes one float per lane to sink (device memory of blocks * 256
 *    floats, owned by the caller).  INVALID_ARG for a NULL sink, a
 *    non-positive count or another dtype.
 *  - conv2d_probe_copy copies `bytes` from src to dst (device memory, not
 *    overlapping) with 16-byte loads and stores when src is 16-byte aligned.
 * Both are asynchronous on `stream`: the caller times them with events. */
conv_status_t conv2d_probe_mfma(int32_t dtype, int32_t blocks, int32_t iters, float* sink, void* stream);
conv_status_t conv2d_probe_copy(const void* src, void* dst, size_t bytes, void* stream);

/* Static strings; never NULL ("unknown" for values outside the enums). */
const char* conv2d_status_string(conv_status_t status);
const char* conv2d_algo_name(conv_algo_t algo);

/* Parses "default", "direct", "implicit_gemm", "im2col_gemm" (alias "gemm"),
 * "winograd", "implicit_precomp_gemm", "kn2row", "smm".  INVALID_ARG for NULL
 * or any other name. */
conv_status_t conv2d_algo_from_name(const char* name, conv_algo_t* algo);

#ifdef __cplusplus
}
#endif

#endif /* CONVSEL_H */
