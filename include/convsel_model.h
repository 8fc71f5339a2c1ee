/*
 * convsel model executor -- a whole inference network run by the library
 * (the paper's swap_backend entry point, Sec. IV: every module of the model
 * is replaced and the result is a model the framework manages), built on
 * the convolution ABI of convsel.h.
 *
 * A model is a list of operations over numbered values.  Value 0 is the
 * network input (N x C x H x W); every convsel_model_* call that adds an
 * operation returns the number of the value it produces.  The operations
 * are the ones the paper's example networks use (Sec. IV, Listings 1-2):
 *
 *   conv     y = conv2d(x, w) + b (then ReLU), any algorithm of convsel.h;
 *   linear   y[n][o] = sum_i x[n][i] * w[o][i] + b[o] (then ReLU), run as a
 *            1 x 1 convolution of an N x I x 1 x 1 input;
 *   relu     y = max(0, x);
 *   pool     max or average over kh x kw windows with stride and zero
 *            padding (average: divided by kh*kw, padding included, as
 *            PyTorch's AvgPool2d by default; max: padding never wins);
 *   global average pool  N x C x H x W -> N x C x 1 x 1 (AdaptiveAvgPool2d
 *            to 1 x 1);
 *   add      y = a + b (then ReLU), same shapes (residual connections);
 *   flatten  N x C x H x W -> N x (C*H*W), no data movement.
 *
 * Life cycle:
 *   1. convsel_model_create, then the operations in order, then
 *      convsel_model_set_output.  Filter and bias pointers are device
 *      addresses read only during convsel_model_bind.
 *   2. convsel_model_plan(n, c, h, w): shapes of every value, the algorithm
 *      of every convolution (CONV_ALGO_DEFAULT resolved), and one device
 *      arena laid out for filter packages, biases, intermediate values and
 *      the largest convolution workspace.  Intermediate values share arena
 *      space when their lifetimes (producer to last reader) do not overlap.
 *      An add whose operand is the output of an implicit-GEMM convolution
 *      (read by nothing else, without a ReLU of its own) and whose other
 *      operand exists before that convolution runs is fused into it: the
 *      convolution's epilogue adds the other operand and applies the add's
 *      ReLU, y = relu(round(conv + b) + other), and the add launches
 *      nothing.  Host only.
 *   3. convsel_model_bind(arena): the caller provides the arena (at least the
 *      planned bytes, 256-byte aligned); the library packs every filter and
 *      copies every bias into it, on `stream`.
 *   4. convsel_model_forward(x, y): runs the network on `stream`; it
 *      allocates nothing and makes no host synchronisation, so it can be
 *      captured into a HIP graph.  x is read only; y receives the output
 *      value (its shape from convsel_model_output_shape).  Calls on one
 *      model must not overlap: they share the arena.
 *   Planning again (another input shape) invalidates the binding.
 *
 * Element type: one per model (conv_dtype_t), shared by x, y, filters and
 * biases.  Errors: status codes of convsel.h; INVALID_ARG for bad value
 * numbers, shapes that do not chain, calls out of order or a NULL model.
 */
#ifndef CONVSEL_MODEL_H
#define CONVSEL_MODEL_H

#include <stddef.h>
#include <stdint.h>

#include "convsel.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct convsel_model convsel_model_t;

conv_status_t convsel_model_create(int32_t dtype, convsel_model_t** model);
void convsel_model_destroy(convsel_model_t* model);

/* c: the input's channel count (checked against the input value at
 * planning); w: K x (c/groups) x R x S device filters; b: K values or NULL. */
conv_status_t convsel_model_conv(convsel_model_t* model, int32_t in, int64_t c, int64_t k, int64_t r, int64_t s,
                                 int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w, int32_t dil_h,
                                 int32_t dil_w, int32_t groups, conv_algo_t algo, const void* w, const void* b,
                                 int32_t fuse_relu, int32_t* out);
/* w: O x I device weights (I = in_features, checked against the flattened
 * input at planning); b: O values or NULL. */
conv_status_t convsel_model_linear(convsel_model_t* model, int32_t in, int64_t in_features, int64_t out_features,
                                   conv_algo_t algo, const void* w, const void* b, int32_t fuse_relu, int32_t* out);
conv_status_t convsel_model_relu(convsel_model_t* model, int32_t in, int32_t* out);
/* kind 0 = max, 1 = average. */
conv_status_t convsel_model_pool(convsel_model_t* model, int32_t in, int32_t kind, int32_t kh, int32_t kw,
                                 int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w, int32_t* out);
conv_status_t convsel_model_global_avgpool(convsel_model_t* model, int32_t in, int32_t* out);
conv_status_t convsel_model_add(convsel_model_t* model, int32_t a, int32_t b, int32_t fuse_relu, int32_t* out);
conv_status_t convsel_model_flatten(convsel_model_t* model, int32_t in, int32_t* out);
conv_status_t convsel_model_set_output(convsel_model_t* model, int32_t value);

/* Plans for an N x C x H x W input; *arena_bytes receives the device bytes
 * convsel_model_bind needs. */
conv_status_t convsel_model_plan(convsel_model_t* model, int64_t n, int64_t c, int64_t h, int64_t w,
                                 size_t* arena_bytes);
/* Output shape after planning: dims[0..*ndim-1] (4 for images, 2 after a
 * flatten or linear). */
conv_status_t convsel_model_output_shape(const convsel_model_t* model, int64_t dims[4], int32_t* ndim);
/* Arena offset and size of value `v` after planning (-1 offset: the value is
 * the caller's input or output, or an alias of one). For tests and tools. */
conv_status_t convsel_model_value_placement(const convsel_model_t* model, int32_t v, int64_t* offset,
                                            int64_t* bytes);
conv_status_t convsel_model_bind(convsel_model_t* model, void* arena, size_t arena_bytes, void* stream);
conv_status_t convsel_model_forward(convsel_model_t* model, const void* x, void* y, void* stream);
/* One line per operation (kind, shapes, algorithm, arena offsets). */
conv_status_t convsel_model_describe(const convsel_model_t* model, char* buf, size_t len);

#ifdef __cplusplus
}
#endif

#endif /* CONVSEL_MODEL_H */
