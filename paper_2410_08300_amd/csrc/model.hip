// Model executor (declared in include/convsel_model.h): a network of
// convolutions, linear layers, ReLU, pooling, residual adds and flattens run
// from one caller-provided device arena.  Planning is host-only: value shapes,
// resolved algorithms, filter packages, the largest convolution workspace,
// and an arena offset for every intermediate value, shared between values
// whose lifetimes do not overlap (greedy by size: each value goes to the
// lowest offset that no already-placed, simultaneously live value covers).
// The forward pass launches the library's convolution entry points and the
// small elementwise / pooling kernels below, and allocates nothing.
#include <algorithm>
#include <stdio.h>
#include <string>
#include <vector>

#include "../../include/convsel_model.h"
#include "common.hpp"

using convsel::bf16_t;
using convsel::elem;

namespace convsel {
conv_status_t conv2d_prepacked_residual(const void* x, const void* packed, const void* b, const void* res, void* y,
                                        const conv2d_desc_t* desc, conv_algo_t algo, void* workspace,
                                        size_t workspace_bytes, void* stream);
}

namespace {

// ---- kernels -------------------------------------------------------------

template <typename T>
__global__ __launch_bounds__(256) void relu_kernel(const T* __restrict__ x, T* __restrict__ y, int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) elem<T>::store(y + i, fmaxf(elem<T>::load(x + i), 0.f));
}

template <typename T>
__global__ __launch_bounds__(256) void add_kernel(const T* __restrict__ a, const T* __restrict__ b, T* __restrict__ y,
                                                  int64_t n, int relu) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= n) return;
  float v = elem<T>::load(a + i) + elem<T>::load(b + i);
  if (relu) v = fmaxf(v, 0.f);
  elem<T>::store(y + i, v);
}

// One output element per thread; consecutive threads take consecutive q.
// A workgroup covers 256 outputs of one plane (`tiles` workgroups per
// plane), so the plane is a per-workgroup quantity and the per-thread index
// arithmetic stays in 32 bits.  Max: padding never contributes.  Average:
// the window sum over the padded input divided by kh*kw.
template <typename T, bool MAX>
__global__ __launch_bounds__(256) void pool_kernel(const T* __restrict__ x, T* __restrict__ y, int tiles, int H,
                                                   int W, int P, int Q, int kh, int kw, int sh, int sw, int ph,
                                                   int pw) {
  const int plane = blockIdx.x / tiles;
  const int j = (blockIdx.x - plane * tiles) * 256 + threadIdx.x;
  if (j >= P * Q) return;
  const int p = j / Q, q = j - p * Q;
  const T* xp = x + static_cast<int64_t>(plane) * H * W;
  float acc = MAX ? -INFINITY : 0.f;
  const int ih0 = p * sh - ph, iw0 = q * sw - pw;
  if (kh <= 3 && kw <= 3) {  // uniform: all taps' loads issued together, then one wait
    float v[9];
#pragma unroll
    for (int t = 0; t < 9; ++t) {
      const int ih = ih0 + t / 3, iw = iw0 + t % 3;
      const bool ok = t / 3 < kh && t % 3 < kw && ih >= 0 && ih < H && iw >= 0 && iw < W;
      v[t] = elem<T>::load(xp + (ok ? ih * W + iw : 0));
      v[t] = ok ? v[t] : (MAX ? -INFINITY : 0.f);
    }
#pragma unroll
    for (int t = 0; t < 9; ++t) acc = MAX ? fmaxf(acc, v[t]) : acc + v[t];
    if (!MAX) acc /= static_cast<float>(kh * kw);
    elem<T>::store(y + static_cast<int64_t>(plane) * P * Q + j, acc);
    return;
  }
  for (int r = 0; r < kh; ++r) {
    const int ih = ih0 + r;
    if (ih < 0 || ih >= H) continue;
    const T* row = xp + ih * W;
    for (int s = 0; s < kw; ++s) {
      const int iw = iw0 + s;
      if (iw < 0 || iw >= W) continue;
      const float v = elem<T>::load(row + iw);
      acc = MAX ? fmaxf(acc, v) : acc + v;
    }
  }
  if (!MAX) acc /= static_cast<float>(kh * kw);
  elem<T>::store(y + static_cast<int64_t>(plane) * P * Q + j, acc);
}

// Global average: one wave per plane, lanes stride the plane, then a fixed
// butterfly over the 64 lanes (deterministic order).
template <typename T>
__global__ __launch_bounds__(256) void global_avgpool_kernel(const T* __restrict__ x, T* __restrict__ y, int64_t planes,
                                                             int HW) {
  const int64_t plane = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (plane >= planes) return;
  const T* xp = x + plane * HW;
  float acc = 0.f;
  for (int i = lane; i < HW; i += 64) acc += elem<T>::load(xp + i);
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, 64);
  if (lane == 0) elem<T>::store(y + plane, acc / static_cast<float>(HW));
}

unsigned blocks_for(int64_t n, int per = 256) { return static_cast<unsigned>((n + per - 1) / per); }

// ---- model ----------------------------------------------------------------

enum OpKind { OP_CONV, OP_RELU, OP_POOL, OP_GAP, OP_ADD, OP_FLATTEN };

struct Value {
  int ndim = 0;
  int64_t d[4] = {0, 0, 0, 0};
  int producer = -1;  // op index; -1 for the input
  int alias = -1;     // flatten: the value whose storage this one shares
  int falias = -1;    // planned: a fused add's output shares its convolution's storage
  int64_t offset = -1;
  int64_t bytes = 0;
  int64_t elems() const {
    int64_t e = 1;
    for (int i = 0; i < ndim; ++i) e *= d[i];
    return e;
  }
};

struct Op {
  OpKind kind;
  int in = -1, in2 = -1, out = -1;
  // convolution / linear
  bool linear = false;
  int64_t c = 0, k = 0, r = 1, s = 1;
  int32_t sh = 1, sw = 1, ph = 0, pw = 0, dh = 1, dw = 1, groups = 1;
  conv_algo_t algo = CONV_ALGO_DEFAULT, algo_run = CONV_ALGO_DEFAULT;
  const void* w = nullptr;
  const void* b = nullptr;
  int relu = 0;
  // planned: residual value added in this convolution's epilogue (an add
  // fused into it; -1: none), the ReLU that then follows it, and whether this
  // op (a fused add) is skipped
  int res = -1;
  int relu_eff = 0;
  bool skip = false;
  conv2d_desc_t desc{};
  int64_t pk_off = -1, pk_bytes = 0, bias_off = -1, ws_bytes = 0;
  // pooling
  int pool_kind = 0, kh = 1, kw = 1;
};

constexpr int64_t kAlign = 256;
int64_t align_up(int64_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

}  // namespace

struct convsel_model {
  int32_t dtype = CONV_F32;
  std::vector<Op> ops;
  std::vector<Value> vals;  // vals[0] is the input
  int output = -1;
  bool planned = false, bound = false;
  char* arena = nullptr;
  int64_t arena_bytes = 0, ws_off = 0, ws_bytes = 0;
  int64_t esize() const { return dtype == CONV_F32 ? 4 : 2; }
  int root(int v) const {
    for (;;) {
      if (vals[v].alias >= 0) v = vals[v].alias;
      else if (vals[v].falias >= 0) v = vals[v].falias;
      else return v;
    }
  }
};

namespace {

conv_status_t add_op(convsel_model_t* m, Op op, int32_t* out) {
  if (!m || !out) return CONV_ERR_INVALID_ARG;
  const int nv = (int)m->vals.size();
  if (op.in < 0 || op.in >= nv || (op.kind == OP_ADD && (op.in2 < 0 || op.in2 >= nv))) return CONV_ERR_INVALID_ARG;
  Value v;
  v.producer = (int)m->ops.size();
  op.out = nv;
  m->vals.push_back(v);
  m->ops.push_back(op);
  m->planned = m->bound = false;
  *out = op.out;
  return CONV_OK;
}

conv_status_t from_hip(hipError_t e) {
  if (e == hipSuccess) return CONV_OK;
  (void)hipGetLastError();
  return CONV_ERR_DEVICE;
}

template <typename T>
hipError_t launch_elementwise(const Op& op, const void* a, const void* b, void* y, const Value& vin, const Value& vout,
                              hipStream_t st) {
  switch (op.kind) {
    case OP_RELU:
      hipLaunchKernelGGL(relu_kernel<T>, dim3(blocks_for(vout.elems())), dim3(256), 0, st,
                         reinterpret_cast<const T*>(a), reinterpret_cast<T*>(y), vout.elems());
      break;
    case OP_ADD:
      hipLaunchKernelGGL(add_kernel<T>, dim3(blocks_for(vout.elems())), dim3(256), 0, st,
                         reinterpret_cast<const T*>(a), reinterpret_cast<const T*>(b), reinterpret_cast<T*>(y),
                         vout.elems(), op.relu);
      break;
    case OP_POOL: {
      // Planning keeps planes * tiles and every plane's size below 2^31.
      const int tiles = (int)blocks_for(vout.d[2] * vout.d[3]);
      const dim3 grid((unsigned)(vout.d[0] * vout.d[1] * tiles));
      if (op.pool_kind == 0)
        hipLaunchKernelGGL((pool_kernel<T, true>), grid, dim3(256), 0, st, reinterpret_cast<const T*>(a),
                           reinterpret_cast<T*>(y), tiles, (int)vin.d[2], (int)vin.d[3], (int)vout.d[2],
                           (int)vout.d[3], op.kh, op.kw, op.sh, op.sw, op.ph, op.pw);
      else
        hipLaunchKernelGGL((pool_kernel<T, false>), grid, dim3(256), 0, st, reinterpret_cast<const T*>(a),
                           reinterpret_cast<T*>(y), tiles, (int)vin.d[2], (int)vin.d[3], (int)vout.d[2],
                           (int)vout.d[3], op.kh, op.kw, op.sh, op.sw, op.ph, op.pw);
      break;
    }
    case OP_GAP:
      hipLaunchKernelGGL(global_avgpool_kernel<T>, dim3(blocks_for(vin.d[0] * vin.d[1], 4)), dim3(256), 0, st,
                         reinterpret_cast<const T*>(a), reinterpret_cast<T*>(y), vin.d[0] * vin.d[1],
                         (int)(vin.d[2] * vin.d[3]));
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

extern "C" {

conv_status_t convsel_model_create(int32_t dtype, convsel_model_t** model) {
  if (!model || (dtype != CONV_F32 && dtype != CONV_BF16)) return CONV_ERR_INVALID_ARG;
  convsel_model_t* m = new convsel_model_t();
  m->dtype = dtype;
  m->vals.push_back(Value());  // the input
  *model = m;
  return CONV_OK;
}

void convsel_model_destroy(convsel_model_t* model) { delete model; }

conv_status_t convsel_model_conv(convsel_model_t* model, int32_t in, int64_t c, int64_t k, int64_t r, int64_t s,
                                 int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w, int32_t dil_h,
                                 int32_t dil_w, int32_t groups, conv_algo_t algo, const void* w, const void* b,
                                 int32_t fuse_relu, int32_t* out) {
  if (!w || c < 1 || k < 1 || r < 1 || s < 1 || groups < 1 || (fuse_relu != 0 && fuse_relu != 1))
    return CONV_ERR_INVALID_ARG;
  if (conv2d_algo_name(algo)[0] == 'u') return CONV_ERR_INVALID_ARG;  // "unknown"
  Op op;
  op.kind = OP_CONV;
  op.in = in;
  op.c = c; op.k = k; op.r = r; op.s = s;
  op.sh = stride_h; op.sw = stride_w; op.ph = pad_h; op.pw = pad_w; op.dh = dil_h; op.dw = dil_w;
  op.groups = groups;
  op.algo = algo;
  op.w = w;
  op.b = b;
  op.relu = fuse_relu;
  return add_op(model, op, out);
}

conv_status_t convsel_model_linear(convsel_model_t* model, int32_t in, int64_t in_features, int64_t out_features,
                                   conv_algo_t algo, const void* w, const void* b, int32_t fuse_relu, int32_t* out) {
  if (!w || in_features < 1 || out_features < 1 || (fuse_relu != 0 && fuse_relu != 1)) return CONV_ERR_INVALID_ARG;
  if (conv2d_algo_name(algo)[0] == 'u') return CONV_ERR_INVALID_ARG;
  Op op;
  op.kind = OP_CONV;
  op.linear = true;
  op.in = in;
  op.c = in_features;
  op.k = out_features;
  op.algo = algo;
  op.w = w;
  op.b = b;
  op.relu = fuse_relu;
  return add_op(model, op, out);
}

conv_status_t convsel_model_relu(convsel_model_t* model, int32_t in, int32_t* out) {
  Op op;
  op.kind = OP_RELU;
  op.in = in;
  return add_op(model, op, out);
}

conv_status_t convsel_model_pool(convsel_model_t* model, int32_t in, int32_t kind, int32_t kh, int32_t kw,
                                 int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w, int32_t* out) {
  if ((kind != 0 && kind != 1) || kh < 1 || kw < 1 || stride_h < 1 || stride_w < 1 || pad_h < 0 || pad_w < 0 ||
      2 * pad_h > kh || 2 * pad_w > kw)
    return CONV_ERR_INVALID_ARG;
  Op op;
  op.kind = OP_POOL;
  op.in = in;
  op.pool_kind = kind;
  op.kh = kh; op.kw = kw; op.sh = stride_h; op.sw = stride_w; op.ph = pad_h; op.pw = pad_w;
  return add_op(model, op, out);
}

conv_status_t convsel_model_global_avgpool(convsel_model_t* model, int32_t in, int32_t* out) {
  Op op;
  op.kind = OP_GAP;
  op.in = in;
  return add_op(model, op, out);
}

conv_status_t convsel_model_add(convsel_model_t* model, int32_t a, int32_t b, int32_t fuse_relu, int32_t* out) {
  if (fuse_relu != 0 && fuse_relu != 1) return CONV_ERR_INVALID_ARG;
  Op op;
  op.kind = OP_ADD;
  op.in = a;
  op.in2 = b;
  op.relu = fuse_relu;
  return add_op(model, op, out);
}

conv_status_t convsel_model_flatten(convsel_model_t* model, int32_t in, int32_t* out) {
  Op op;
  op.kind = OP_FLATTEN;
  op.in = in;
  const conv_status_t st = add_op(model, op, out);
  if (st == CONV_OK) model->vals[*out].alias = in;
  return st;
}

conv_status_t convsel_model_set_output(convsel_model_t* model, int32_t value) {
  if (!model || value <= 0 || value >= (int32_t)model->vals.size()) return CONV_ERR_INVALID_ARG;
  model->output = value;
  model->planned = model->bound = false;
  return CONV_OK;
}

conv_status_t convsel_model_plan(convsel_model_t* model, int64_t n, int64_t c, int64_t h, int64_t w,
                                 size_t* arena_bytes) {
  if (!model || !arena_bytes || n < 1 || c < 1 || h < 1 || w < 1 || model->output < 0) return CONV_ERR_INVALID_ARG;
  convsel_model_t& m = *model;
  m.planned = m.bound = false;
  const int64_t es = m.esize();
  for (Op& op : m.ops) {
    op.res = -1;
    op.relu_eff = op.relu;
    op.skip = false;
  }
  for (Value& v : m.vals) v.falias = -1;
  Value& in = m.vals[0];
  in.ndim = 4;
  in.d[0] = n; in.d[1] = c; in.d[2] = h; in.d[3] = w;
  // Shapes, algorithms, packages and workspaces, in operation order.
  int64_t off = 0;
  m.ws_bytes = 0;
  for (Op& op : m.ops) {
    const Value& a = m.vals[op.in];
    Value& o = m.vals[op.out];
    o.offset = -1;
    switch (op.kind) {
      case OP_CONV: {
        conv2d_desc_t& d = op.desc;
        if (op.linear) {
          const int64_t feat = a.ndim == 2 ? a.d[1] : (a.ndim == 4 ? a.d[1] * a.d[2] * a.d[3] : -1);
          if (feat != op.c || (a.ndim == 4 && a.d[2] * a.d[3] != 1)) return CONV_ERR_INVALID_ARG;
          d = conv2d_desc_t{a.d[0], op.c, 1, 1, op.k, 1, 1, 1, 1, 0, 0, 1, 1, 1, m.dtype, op.b != nullptr, op.relu};
        } else {
          if (a.ndim != 4 || a.d[1] != op.c) return CONV_ERR_INVALID_ARG;
          d = conv2d_desc_t{a.d[0], a.d[1], a.d[2], a.d[3], op.k, op.r, op.s, op.sh, op.sw, op.ph, op.pw,
                            op.dh, op.dw, op.groups, m.dtype, op.b != nullptr, op.relu};
        }
        conv_algo_t al = op.algo == CONV_ALGO_DEFAULT ? conv2d_default_algo(&d) : op.algo;
        const conv_status_t st = conv2d_check(&d, al);
        if (st != CONV_OK) return st;
        op.algo_run = al;
        size_t pk = 0, ws = 0;
        if (conv2d_packed_filter_bytes(&d, al, &pk) != CONV_OK || conv2d_prepacked_workspace_bytes(&d, al, &ws) != CONV_OK)
          return CONV_ERR_INVALID_ARG;
        op.pk_off = off;
        op.pk_bytes = (int64_t)pk;
        off = align_up(off + (int64_t)pk);
        op.bias_off = -1;
        if (op.b) {
          op.bias_off = off;
          off = align_up(off + op.k * es);
        }
        op.ws_bytes = (int64_t)ws;
        m.ws_bytes = std::max(m.ws_bytes, (int64_t)ws);
        if (op.linear) {
          o.ndim = 2;
          o.d[0] = a.d[0]; o.d[1] = op.k; o.d[2] = o.d[3] = 0;
        } else {
          int64_t P = 0, Q = 0;
          conv2d_output_shape(&d, &P, &Q);
          o.ndim = 4;
          o.d[0] = a.d[0]; o.d[1] = op.k; o.d[2] = P; o.d[3] = Q;
        }
        break;
      }
      case OP_RELU:
        o.ndim = a.ndim;
        for (int i = 0; i < 4; ++i) o.d[i] = a.d[i];
        break;
      case OP_ADD: {
        const Value& b = m.vals[op.in2];
        if (a.ndim != b.ndim) return CONV_ERR_INVALID_ARG;
        for (int i = 0; i < a.ndim; ++i)
          if (a.d[i] != b.d[i]) return CONV_ERR_INVALID_ARG;
        o.ndim = a.ndim;
        for (int i = 0; i < 4; ++i) o.d[i] = a.d[i];
        break;
      }
      case OP_POOL: {
        if (a.ndim != 4 || a.elems() >= ((int64_t)1 << 31)) return CONV_ERR_INVALID_ARG;  // 32-bit plane offsets
        const int64_t P = (a.d[2] + 2 * op.ph - op.kh) / op.sh + 1;
        const int64_t Q = (a.d[3] + 2 * op.pw - op.kw) / op.sw + 1;
        if (a.d[2] + 2 * op.ph < op.kh || a.d[3] + 2 * op.pw < op.kw || P < 1 || Q < 1) return CONV_ERR_INVALID_ARG;
        o.ndim = 4;
        o.d[0] = a.d[0]; o.d[1] = a.d[1]; o.d[2] = P; o.d[3] = Q;
        break;
      }
      case OP_GAP:
        if (a.ndim != 4) return CONV_ERR_INVALID_ARG;
        o.ndim = 4;
        o.d[0] = a.d[0]; o.d[1] = a.d[1]; o.d[2] = o.d[3] = 1;
        break;
      case OP_FLATTEN:
        if (a.ndim != 4) return CONV_ERR_INVALID_ARG;
        o.ndim = 2;
        o.d[0] = a.d[0]; o.d[1] = a.d[1] * a.d[2] * a.d[3]; o.d[2] = o.d[3] = 0;
        break;
    }
    if (o.elems() >= ((int64_t)1 << 31)) return CONV_ERR_INVALID_ARG;
    o.bytes = o.elems() * es;
  }
  // Residual adds into implicit GEMM convolutions: an add of a convolution's
  // output X (read by nothing else, no ReLU of its own) and a value Y that
  // exists before that convolution runs becomes that convolution's epilogue
  // residual, y = relu(conv + b + Y); the add's output then shares X's storage.
  {
    const int nv0 = (int)m.vals.size();
    std::vector<int> uses(nv0, 0);
    for (const Op& op : m.ops) {
      ++uses[op.in];
      if (op.kind == OP_ADD) ++uses[op.in2];
    }
    ++uses[m.output];
    for (int i = 0; i < (int)m.ops.size(); ++i) {
      Op& add = m.ops[i];
      if (add.kind != OP_ADD) continue;
      int best = -1, other = -1;
      for (int side = 0; side < 2; ++side) {
        const int X = side == 0 ? add.in : add.in2, Y = side == 0 ? add.in2 : add.in;
        const int p = m.vals[X].producer;
        if (p < 0 || m.vals[X].alias >= 0 || uses[X] != 1) continue;
        const Op& c = m.ops[p];
        if (c.kind != OP_CONV || c.algo_run != CONV_ALGO_IMPLICIT_GEMM || c.relu_eff || c.res >= 0) continue;
        if (m.vals[m.root(Y)].producer >= p) continue;  // Y must exist when the convolution runs
        if (best < 0 || p > m.vals[best].producer) {
          best = X;
          other = Y;
        }
      }
      if (best < 0) continue;
      Op& c = m.ops[m.vals[best].producer];
      c.res = other;
      c.relu_eff = add.relu;
      c.desc.fuse_relu = add.relu;
      add.skip = true;
      m.vals[add.out].falias = best;
    }
  }
  // The output must come out of an operation, not be the input itself.
  const int out_root = m.root(m.output);
  if (out_root == 0) return CONV_ERR_UNSUPPORTED;
  // Lifetimes of the storage roots: [producer, last reader].
  const int nv = (int)m.vals.size();
  std::vector<int> last(nv, -1), first(nv, -1);
  for (int i = 0; i < nv; ++i)
    if (m.vals[i].alias < 0 && m.vals[i].falias < 0) first[i] = last[i] = m.vals[i].producer;
  for (int i = 0; i < (int)m.ops.size(); ++i) {
    const Op& op = m.ops[i];
    if (op.skip) continue;
    last[m.root(op.in)] = std::max(last[m.root(op.in)], i);
    if (op.kind == OP_ADD) last[m.root(op.in2)] = std::max(last[m.root(op.in2)], i);
    if (op.res >= 0) last[m.root(op.res)] = std::max(last[m.root(op.res)], i);
  }
  // The workspace, then the activations.
  m.ws_off = off;
  off = align_up(off + m.ws_bytes);
  const int64_t act_base = off;
  std::vector<int> order;
  for (int i = 1; i < nv; ++i)
    if (m.vals[i].alias < 0 && m.vals[i].falias < 0 && i != out_root) order.push_back(i);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return m.vals[a].bytes > m.vals[b].bytes; });
  std::vector<int> placed;
  int64_t act_top = 0;
  for (int v : order) {
    // Intervals [offset, offset + bytes) of placed values live at the same time, sorted by offset.
    std::vector<std::pair<int64_t, int64_t>> busy;
    for (int u : placed)
      if (first[u] <= last[v] && first[v] <= last[u])
        busy.push_back({m.vals[u].offset, m.vals[u].offset + align_up(m.vals[u].bytes)});
    std::sort(busy.begin(), busy.end());
    int64_t cand = 0;
    const int64_t need = align_up(m.vals[v].bytes);
    for (const auto& iv : busy) {
      if (cand + need <= iv.first) break;
      cand = std::max(cand, iv.second);
    }
    m.vals[v].offset = cand;
    act_top = std::max(act_top, cand + need);
    placed.push_back(v);
  }
  for (int v : order) m.vals[v].offset += act_base;
  m.arena_bytes = act_base + act_top;
  *arena_bytes = (size_t)m.arena_bytes;
  m.planned = true;
  return CONV_OK;
}

conv_status_t convsel_model_output_shape(const convsel_model_t* model, int64_t dims[4], int32_t* ndim) {
  if (!model || !dims || !ndim || !model->planned) return CONV_ERR_INVALID_ARG;
  const Value& v = model->vals[model->output];
  *ndim = v.ndim;
  for (int i = 0; i < 4; ++i) dims[i] = i < v.ndim ? v.d[i] : 0;
  return CONV_OK;
}

conv_status_t convsel_model_value_placement(const convsel_model_t* model, int32_t v, int64_t* offset,
                                            int64_t* bytes) {
  if (!model || !offset || !bytes || !model->planned || v < 0 || v >= (int32_t)model->vals.size())
    return CONV_ERR_INVALID_ARG;
  const int r = model->root(v);
  *offset = (r == 0 || r == model->root(model->output)) ? -1 : model->vals[r].offset;
  *bytes = model->vals[v].bytes;
  return CONV_OK;
}

conv_status_t convsel_model_bind(convsel_model_t* model, void* arena, size_t arena_bytes, void* stream) {
  if (!model || !model->planned) return CONV_ERR_INVALID_ARG;
  convsel_model_t& m = *model;
  if ((int64_t)arena_bytes < m.arena_bytes || (m.arena_bytes > 0 && !arena) ||
      reinterpret_cast<uintptr_t>(arena) % kAlign != 0)
    return CONV_ERR_INVALID_ARG;
  m.bound = false;
  char* base = reinterpret_cast<char*>(arena);
  const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  for (Op& op : m.ops) {
    if (op.kind != OP_CONV) continue;
    conv_status_t s = conv2d_pack_filters(op.w, base + op.pk_off, &op.desc, op.algo_run, stream);
    if (s != CONV_OK) return s;
    if (op.b) {
      s = from_hip(hipMemcpyAsync(base + op.bias_off, op.b, (size_t)(op.k * m.esize()), hipMemcpyDeviceToDevice, st));
      if (s != CONV_OK) return s;
    }
  }
  m.arena = base;
  m.bound = true;
  return CONV_OK;
}

conv_status_t convsel_model_forward(convsel_model_t* model, const void* x, void* y, void* stream) {
  if (!model || !model->bound || !x || !y) return CONV_ERR_INVALID_ARG;
  convsel_model_t& m = *model;
  const int out_root = m.root(m.output);
  const hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  auto ptr = [&](int v) -> char* {
    const int r = m.root(v);
    if (r == 0) return const_cast<char*>(reinterpret_cast<const char*>(x));
    if (r == out_root) return reinterpret_cast<char*>(y);
    return m.arena + m.vals[r].offset;
  };
  for (const Op& op : m.ops) {
    const Value& vin = m.vals[op.in];
    const Value& vout = m.vals[op.out];
    conv_status_t s = CONV_OK;
    if (op.skip) continue;  // an add fused into its convolution
    switch (op.kind) {
      case OP_CONV:
        if (op.res >= 0)
          s = convsel::conv2d_prepacked_residual(
              ptr(op.in), m.arena + op.pk_off, op.b ? m.arena + op.bias_off : nullptr, ptr(op.res), ptr(op.out),
              &op.desc, op.algo_run, op.ws_bytes ? m.arena + m.ws_off : nullptr, (size_t)op.ws_bytes, stream);
        else
          s = conv2d_prepacked(ptr(op.in), m.arena + op.pk_off, op.b ? m.arena + op.bias_off : nullptr, ptr(op.out),
                               &op.desc, op.algo_run, op.ws_bytes ? m.arena + m.ws_off : nullptr, (size_t)op.ws_bytes,
                               stream);
        break;
      case OP_FLATTEN:
        break;
      default:
        s = from_hip(m.dtype == CONV_F32
                         ? launch_elementwise<float>(op, ptr(op.in), op.in2 >= 0 ? ptr(op.in2) : nullptr,
                                                     ptr(op.out), vin, vout, st)
                         : launch_elementwise<bf16_t>(op, ptr(op.in), op.in2 >= 0 ? ptr(op.in2) : nullptr,
                                                      ptr(op.out), vin, vout, st));
        break;
    }
    if (s != CONV_OK) return s;
  }
  return CONV_OK;
}

conv_status_t convsel_model_describe(const convsel_model_t* model, char* buf, size_t len) {
  if (!model || !buf || len == 0) return CONV_ERR_INVALID_ARG;
  static const char* names[] = {"conv", "relu", "pool", "global_avgpool", "add", "flatten"};
  std::string d;
  char line[256];
  for (size_t i = 0; i < model->ops.size(); ++i) {
    const Op& op = model->ops[i];
    const Value& o = model->vals[op.out];
    const char* nm = op.kind == OP_CONV && op.linear ? "linear" : names[op.kind];
    snprintf(line, sizeof(line), "%zu %s v%d%s -> v%d [%lld %lld %lld %lld]", i, nm, op.in,
             op.kind == OP_ADD ? (std::string(" + v") + std::to_string(op.in2)).c_str() : "", op.out,
             (long long)o.d[0], (long long)o.d[1], (long long)o.d[2], (long long)o.d[3]);
    d += line;
    if (op.kind == OP_CONV) d += std::string(" algo=") + conv2d_algo_name(model->planned ? op.algo_run : op.algo);
    if (model->planned && op.res >= 0) d += " + v" + std::to_string(op.res);
    if (model->planned ? (op.kind == OP_CONV ? op.relu_eff : op.relu) : op.relu) d += " relu";
    if (model->planned && op.skip) d += " fused";
    if (model->planned) {
      snprintf(line, sizeof(line), " offset=%lld", (long long)(model->root(op.out) == model->root(model->output)
                                                                     ? -1
                                                                     : model->vals[model->root(op.out)].offset));
      d += line;
    }
    d += "\n";
  }
  if (model->planned) {
    snprintf(line, sizeof(line), "arena=%lld workspace=%lld@%lld", (long long)model->arena_bytes,
             (long long)model->ws_bytes, (long long)model->ws_off);
    d += line;
  }
  snprintf(buf, len, "%s", d.c_str());
  return CONV_OK;
}

}  // extern "C"
