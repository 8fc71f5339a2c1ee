// C ABI of the library (declared in include/convsel.h): descriptor
// validation, algorithm support, workspace sizes, the default-algorithm rule
// and dispatch to the kernel launchers.  All checks run on the host before
// the first HIP call.
#include <math.h>
#include <mutex>
#include <stdio.h>
#include <string.h>
#include <string>

#include "../../include/convsel.h"
#include "kernels.hpp"

using convsel::Shape;

namespace {

constexpr int64_t kInt31 = (int64_t)1 << 31;
constexpr size_t kWorkspaceCap = (size_t)1 << 30;  // batch the column matrix / Winograd buffers near 1 GiB

int64_t out_extent(int64_t in, int64_t pad, int64_t dil, int64_t ker, int64_t stride) {
  const int64_t span = in + 2 * pad - dil * (ker - 1) - 1;
  if (span < 0) return 0;
  return span / stride + 1;
}

conv_status_t validate(const conv2d_desc_t* d, Shape* s) {
  if (!d) return CONV_ERR_INVALID_ARG;
  if (d->n < 0 || d->c < 1 || d->h < 1 || d->w < 1 || d->k < 1 || d->r < 1 || d->s < 1) return CONV_ERR_INVALID_ARG;
  if (d->stride_h < 1 || d->stride_w < 1 || d->dil_h < 1 || d->dil_w < 1) return CONV_ERR_INVALID_ARG;
  if (d->pad_h < 0 || d->pad_w < 0 || d->groups < 1) return CONV_ERR_INVALID_ARG;
  if (d->c % d->groups != 0 || d->k % d->groups != 0) return CONV_ERR_INVALID_ARG;
  if (d->dtype != CONV_F32 && d->dtype != CONV_BF16) return CONV_ERR_INVALID_ARG;
  if ((d->has_bias != 0 && d->has_bias != 1) || (d->fuse_relu != 0 && d->fuse_relu != 1)) return CONV_ERR_INVALID_ARG;
  const int64_t P = out_extent(d->h, d->pad_h, d->dil_h, d->r, d->stride_h);
  const int64_t Q = out_extent(d->w, d->pad_w, d->dil_w, d->s, d->stride_w);
  if (P < 1 || Q < 1) return CONV_ERR_INVALID_ARG;
  // Every tensor, and the pixel count N*P*Q, must stay below 2^31 elements
  // (the kernels index within a tensor in 32 bits where it is cheaper).
  if (d->c > kInt31 / d->h || d->c * d->h > kInt31 / d->w) return CONV_ERR_INVALID_ARG;
  const int64_t chw = d->c * d->h * d->w;
  if (d->n > 0 && d->n > (kInt31 - 1) / chw) return CONV_ERR_INVALID_ARG;
  const int64_t Cg = d->c / d->groups;
  if (d->r > kInt31 / d->s || Cg > kInt31 / (d->r * d->s) || d->k > kInt31 / (Cg * d->r * d->s))
    return CONV_ERR_INVALID_ARG;
  if (P > kInt31 / Q || d->k > kInt31 / (P * Q)) return CONV_ERR_INVALID_ARG;
  if (d->n > 0 && d->n > (kInt31 - 1) / (d->k * P * Q)) return CONV_ERR_INVALID_ARG;
  if (s) {
    s->N = d->n; s->C = d->c; s->H = d->h; s->W = d->w; s->K = d->k; s->R = d->r; s->S = d->s;
    s->P = P; s->Q = Q;
    s->G = d->groups; s->Cg = Cg; s->Kg = d->k / d->groups;
    s->sh = d->stride_h; s->sw = d->stride_w; s->ph = d->pad_h; s->pw = d->pad_w;
    s->dh = d->dil_h; s->dw = d->dil_w;
    s->dtype = d->dtype == CONV_F32 ? convsel::DT_F32 : convsel::DT_BF16;
    s->bias = d->has_bias != 0;
    s->relu = d->fuse_relu != 0;
  }
  return CONV_OK;
}

bool winograd_ok(const Shape& s) {
  return s.R == 3 && s.S == 3 && s.sh == 1 && s.sw == 1 && s.dh == 1 && s.dw == 1 && s.G == 1;
}

conv_status_t support(const Shape& s, conv_algo_t algo) {
  switch (algo) {
    case CONV_ALGO_DIRECT:
    case CONV_ALGO_IM2COL_GEMM:
      return CONV_OK;
    case CONV_ALGO_IMPLICIT_GEMM:
      return convsel::implicit_gemm_fits(s) ? CONV_OK : CONV_ERR_UNSUPPORTED;
    case CONV_ALGO_WINOGRAD:
      return winograd_ok(s) ? CONV_OK : CONV_ERR_UNSUPPORTED;
    case CONV_ALGO_IMPLICIT_PRECOMP_GEMM:
      return convsel::precomp_applies(s) ? CONV_OK : CONV_ERR_UNSUPPORTED;
    case CONV_ALGO_KN2ROW:
      return convsel::kn2row_applies(s) ? CONV_OK : CONV_ERR_UNSUPPORTED;
    case CONV_ALGO_SMM:
      return convsel::smm_applies(s) ? CONV_OK : CONV_ERR_UNSUPPORTED;
    default:
      return CONV_ERR_INVALID_ARG;
  }
}

// The default choice: a decision tree over shape features, fitted offline to
// measured per-layer timings of every algorithm (the heuristic "guess" of the
// paper's comparison, Sec. V-B); a leaf ranks the algorithms and the first
// one that supports the layer is taken.
struct GuessNode {
  int feature;
  double threshold;
  int left, right, leaf;
};
#include "guess_tree.inc"

// Features in the fitted order: bf16, depthwise, taps, stride, log2(C/G),
// log2(K/G), log2(N*P*Q), log2(P*Q), Winograd-eligible, dilated, grouped.
void guess_features(const Shape& s, double f[11]) {
  f[0] = s.dtype == convsel::DT_BF16 ? 1.0 : 0.0;
  f[1] = s.Cg == 1 ? 1.0 : 0.0;
  f[2] = (double)(s.R * s.S);
  f[3] = (double)(s.sh > s.sw ? s.sh : s.sw);
  f[4] = log2((double)s.Cg);
  f[5] = log2((double)s.Kg);
  f[6] = log2((double)(s.N > 0 ? s.N : 1) * (double)(s.P * s.Q));
  f[7] = log2((double)(s.P * s.Q));
  f[8] = winograd_ok(s) ? 1.0 : 0.0;
  f[9] = (s.dh > 1 || s.dw > 1) ? 1.0 : 0.0;
  f[10] = (s.G > 1 && s.Cg > 1) ? 1.0 : 0.0;
}

conv_algo_t default_rule(const Shape& s) {
  double f[11];
  guess_features(s, f);
  int i = 0;
  while (kGuessNodes[i].feature >= 0)
    i = f[kGuessNodes[i].feature] <= kGuessNodes[i].threshold ? kGuessNodes[i].left : kGuessNodes[i].right;
  for (int a : kGuessRank[kGuessNodes[i].leaf])
    if (support(s, (conv_algo_t)a) == CONV_OK) return (conv_algo_t)a;
  return CONV_ALGO_DIRECT;  // defined for every valid layer
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// Images per batch of the column matrix.
int64_t im2col_batch(const Shape& s, size_t* bytes) {
  const size_t per_img = (size_t)s.G * s.P * s.Q * s.Cg * s.R * s.S * s.esize();
  int64_t nb = (int64_t)(kWorkspaceCap / per_img);
  if (nb < 1) nb = 1;
  if (nb > s.N) nb = s.N;
  if (bytes) *bytes = (size_t)nb * per_img;
  return nb;
}

size_t wino_u_bytes(const Shape& s) { return (size_t)16 * s.K * s.C * s.esize(); }

// Winograd workspace: [U (unless prepacked)] [V for nb images] [M for nb images].
struct WinoLayout {
  int64_t nb, TPQ;
  size_t v_off, m_off, total;
};

WinoLayout wino_layout(const Shape& s, bool with_u) {
  WinoLayout L;
  L.TPQ = ((s.P + 1) / 2) * ((s.Q + 1) / 2);
  const size_t v_img = (size_t)16 * L.TPQ * s.C * s.esize();
  const size_t m_img = (size_t)16 * s.K * L.TPQ * 4;
  int64_t nb = (int64_t)(kWorkspaceCap / (v_img + m_img));
  if (nb < 1) nb = 1;
  if (nb > s.N) nb = s.N;
  L.nb = nb;
  L.v_off = with_u ? align256(wino_u_bytes(s)) : 0;
  L.m_off = align256(L.v_off + nb * v_img);
  L.total = L.m_off + nb * m_img;
  return L;
}

// Workspace of conv2d() (prepacked = false) or conv2d_prepacked().
size_t workspace_for(const Shape& s, conv_algo_t algo, bool prepacked = false) {
  if (s.N == 0) return 0;
  if (algo == CONV_ALGO_IM2COL_GEMM) {
    size_t b = 0;
    im2col_batch(s, &b);
    return b;
  }
  if (algo == CONV_ALGO_WINOGRAD) return wino_layout(s, !prepacked).total;
  if (algo == CONV_ALGO_IMPLICIT_GEMM)
    return prepacked ? convsel::implicit_gemm_split_bytes(s) : convsel::implicit_gemm_workspace(s);
  if (algo == CONV_ALGO_IMPLICIT_PRECOMP_GEMM) return prepacked ? 0 : convsel::precomp_packed_bytes(s);
  if (algo == CONV_ALGO_KN2ROW)
    return (prepacked ? 0 : align256(convsel::kn2row_packed_bytes(s))) + convsel::kn2row_z_bytes(s);
  if (algo == CONV_ALGO_SMM)
    return (prepacked ? 0 : align256(convsel::smm_packed_bytes(s))) + convsel::smm_zero_pack_bytes(s);
  return 0;
}

// Size of the filter package of conv2d_pack_filters().
size_t packed_filter_bytes(const Shape& s, conv_algo_t algo) {
  if (algo == CONV_ALGO_IMPLICIT_GEMM) return convsel::implicit_gemm_packed_bytes(s);
  if (algo == CONV_ALGO_WINOGRAD) return wino_u_bytes(s);
  if (algo == CONV_ALGO_IMPLICIT_PRECOMP_GEMM) return convsel::precomp_packed_bytes(s);
  if (algo == CONV_ALGO_KN2ROW) return convsel::kn2row_packed_bytes(s);
  if (algo == CONV_ALGO_SMM) return convsel::smm_packed_bytes(s);
  return (size_t)s.K * s.Cg * s.R * s.S * s.esize();  // the filters themselves
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + nb && b0 < a0 + na;
}

// Device readiness: a current device that is gfx950.  Cached per device.
std::mutex g_dev_mu;
int g_dev_state[64];  // 0 unknown, 1 ok, 2 unusable

conv_status_t ensure_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    (void)hipGetLastError();
    return CONV_ERR_DEVICE;
  }
  std::lock_guard<std::mutex> lock(g_dev_mu);
  if (g_dev_state[dev] == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) {
      (void)hipGetLastError();
      return CONV_ERR_DEVICE;
    }
    g_dev_state[dev] = strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 2;
  }
  return g_dev_state[dev] == 1 ? CONV_OK : CONV_ERR_DEVICE;
}

// Scratch of conv2d_static_scratch(): the workspace of callers that cannot
// allocate.  A device global, so every GPU the library runs on holds its own
// copy (from module load until the process ends).  Host code must not use
// the array's name as an address: the per-device address comes from
// hipGetSymbolAddress, taken once per device with that device current.
constexpr size_t kScratchBytes = (size_t)32 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
void* g_scratch_ptr[64];

// This device's scratch address, or nullptr if it cannot be found (the
// caller's device is already checked by ensure_device()).
void* scratch_for_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    (void)hipGetLastError();
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_dev_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
      (void)hipGetLastError();
      return nullptr;
    }
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

conv_status_t from_hip(hipError_t e) {
  if (e == hipSuccess) return CONV_OK;
  (void)hipGetLastError();
  return CONV_ERR_DEVICE;
}

// Runs the algorithm.  `wpk` is the filter package of conv2d_pack_filters()
// (prepacked calls) or NULL, in which case the package is built in the
// workspace first (implicit GEMM, Winograd) or the filters are used as they
// are (direct, IM2COL + GEMM).
conv_status_t run(const Shape& s, conv_algo_t algo, const void* x, const void* w, const void* wpk, const void* b,
                  void* y, void* ws, hipStream_t st) {
  using namespace convsel;
  const void* filt = wpk ? wpk : w;
  switch (algo) {
    case CONV_ALGO_DIRECT:
      return from_hip(launch_direct(s, x, filt, b, y, st));
    case CONV_ALGO_IMPLICIT_GEMM:
      if (wpk) return from_hip(launch_implicit_main(s, x, wpk, b, y, ws, st));
      return from_hip(launch_implicit_gemm(s, x, w, b, y, ws, st));
    case CONV_ALGO_IM2COL_GEMM: {
      const int64_t nb = im2col_batch(s, nullptr);
      const int64_t crs = s.Cg * s.R * s.S, PQ = s.P * s.Q;
      for (int64_t n0 = 0; n0 < s.N; n0 += nb) {
        const int64_t cnt = s.N - n0 < nb ? s.N - n0 : nb;
        hipError_t e = launch_im2col(s, x, ws, n0, cnt, st);
        if (e != hipSuccess) return from_hip(e);
        GemmArgs g;
        g.A = filt;
        g.B = ws;
        g.C = (char*)y + (size_t)n0 * s.K * PQ * s.esize();
        g.bias = b;
        g.M = (int)s.Kg; g.N = (int)PQ; g.Kred = (int)crs;
        g.lda = crs; g.ldb = crs; g.ldc = PQ;
        g.batch = (int)(cnt * s.G); g.bdiv = s.G;
        g.sA0 = 0; g.sA1 = s.Kg * crs;                 // group g's filters
        g.sB0 = s.G * PQ * crs; g.sB1 = PQ * crs;      // image, group rows of col
        g.sC0 = s.K * PQ; g.sC1 = s.Kg * PQ;           // image, group planes of y
        g.sBias1 = s.Kg;                               // group g's biases
        g.relu = s.relu ? 1 : 0;
        g.out_f32 = 0;
        g.b_kmajor = 0;
        e = launch_gemm_nt(s.dtype, g, st);
        if (e != hipSuccess) return from_hip(e);
      }
      return CONV_OK;
    }
    case CONV_ALGO_WINOGRAD: {
      const WinoLayout L = wino_layout(s, wpk == nullptr);
      char* base = (char*)ws;
      const void* U = wpk;
      if (!wpk) {
        const hipError_t e = launch_wino_filter(s, w, base, st);
        if (e != hipSuccess) return from_hip(e);
        U = base;
      }
      void* V = base + L.v_off;
      float* M = (float*)(base + L.m_off);
      for (int64_t n0 = 0; n0 < s.N; n0 += L.nb) {
        const int64_t cnt = s.N - n0 < L.nb ? s.N - n0 : L.nb;
        const int64_t Tc = cnt * L.TPQ;
        hipError_t e = launch_wino_input(s, x, V, n0, cnt, st);
        if (e != hipSuccess) return from_hip(e);
        GemmArgs g;
        g.A = U; g.B = V; g.C = M; g.bias = nullptr;
        g.M = (int)s.K; g.N = (int)Tc; g.Kred = (int)s.C;
        g.lda = s.C; g.ldb = s.C; g.ldc = Tc;
        g.batch = 16; g.bdiv = 1;
        g.sA0 = s.K * s.C; g.sA1 = 0;
        g.sB0 = Tc * s.C; g.sB1 = 0;
        g.sC0 = s.K * Tc; g.sC1 = 0;
        g.sBias1 = 0;
        g.relu = 0;
        g.out_f32 = 1;
        g.b_kmajor = 0;
        e = launch_gemm_nt(s.dtype, g, st);
        if (e != hipSuccess) return from_hip(e);
        e = launch_wino_output(s, M, b, (char*)y + (size_t)n0 * s.K * s.P * s.Q * s.esize(), 0, cnt, st);
        if (e != hipSuccess) return from_hip(e);
      }
      return CONV_OK;
    }
    case CONV_ALGO_IMPLICIT_PRECOMP_GEMM: {
      if (!wpk) {
        const hipError_t e = precomp_pack(s, w, ws, st);
        if (e != hipSuccess) return from_hip(e);
      }
      return from_hip(precomp_main(s, x, wpk ? wpk : ws, b, y, st));
    }
    case CONV_ALGO_KN2ROW:
    case CONV_ALGO_SMM: {
      const bool kn = algo == CONV_ALGO_KN2ROW;
      char* base = (char*)ws;
      const void* pk = wpk;
      if (!wpk) {
        const hipError_t e = kn ? kn2row_pack(s, w, base, st) : smm_pack(s, w, base, st);
        if (e != hipSuccess) return from_hip(e);
        pk = base;
        base += align256(kn ? kn2row_packed_bytes(s) : smm_packed_bytes(s));
      }
      return from_hip(kn ? kn2row_main(s, x, pk, b, y, base, st) : smm_main(s, x, pk, b, y, base, st));
    }
    default:
      return CONV_ERR_INVALID_ARG;
  }
}

// Shared checks of conv2d() and conv2d_prepacked() up to the device call.
conv_status_t prepare_call(const conv2d_desc_t* desc, conv_algo_t* algo, Shape* s, const void* x, const void* w,
                           const void* b, void* y, void* workspace, size_t workspace_bytes, bool prepacked) {
  conv_status_t st = validate(desc, s);
  if (st != CONV_OK) return st;
  if (*algo == CONV_ALGO_DEFAULT) *algo = default_rule(*s);
  st = support(*s, *algo);
  if (st != CONV_OK) return st;
  if (s->N == 0) return CONV_OK;
  if (!x || !w || !y || (s->bias != (b != nullptr))) return CONV_ERR_INVALID_ARG;
  const size_t need = workspace_for(*s, *algo, prepacked);
  if (workspace_bytes < need || (need > 0 && !workspace)) return CONV_ERR_WORKSPACE;
  if (need > 0 && reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return CONV_ERR_INVALID_ARG;
  const size_t es = (size_t)s->esize();
  const size_t ybytes = (size_t)s->N * s->K * s->P * s->Q * es;
  const size_t wbytes = prepacked ? packed_filter_bytes(*s, *algo) : (size_t)s->K * s->Cg * s->R * s->S * es;
  if (prepacked && reinterpret_cast<uintptr_t>(w) % 256 != 0) return CONV_ERR_INVALID_ARG;
  if (overlaps(y, ybytes, x, (size_t)s->N * s->C * s->H * s->W * es) || overlaps(y, ybytes, w, wbytes) ||
      overlaps(y, ybytes, b, s->bias ? (size_t)s->K * es : 0) || overlaps(y, ybytes, workspace, need))
    return CONV_ERR_INVALID_ARG;
  return ensure_device();
}

}  // namespace

namespace convsel {

// Byte copy (filter packages of the algorithms that use the filters as they
// are): 16-byte units when the source is 16-byte aligned, then the remaining
// bytes one per thread.
namespace {
__global__ void copy16_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst, int64_t n16) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n16) dst[i] = src[i];
}
__global__ void copy1_kernel(const unsigned char* __restrict__ src, unsigned char* __restrict__ dst, int64_t from,
                             int64_t to) {
  const int64_t i = from + static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < to) dst[i] = src[i];
}

}  // namespace

hipError_t launch_copy(const void* w, void* dst, size_t bytes, hipStream_t st) {
  const bool aligned = reinterpret_cast<uintptr_t>(w) % 16 == 0;
  const int64_t n16 = aligned ? (int64_t)(bytes / 16) : 0;
  if (n16 > 0)
    hipLaunchKernelGGL(copy16_kernel, dim3((unsigned)((n16 + 255) / 256)), dim3(256), 0, st, (const uint4*)w,
                       (uint4*)dst, n16);
  const int64_t from = n16 * 16, rest = (int64_t)bytes - from;
  if (rest > 0)
    hipLaunchKernelGGL(copy1_kernel, dim3((unsigned)((rest + 255) / 256)), dim3(256), 0, st,
                       (const unsigned char*)w, (unsigned char*)dst, from, (int64_t)bytes);
  return hipGetLastError();
}

}  // namespace convsel

extern "C" {

conv_status_t conv2d_output_shape(const conv2d_desc_t* desc, int64_t* p, int64_t* q) {
  Shape s;
  const conv_status_t st = validate(desc, &s);
  if (st != CONV_OK) return st;
  if (!p || !q) return CONV_ERR_INVALID_ARG;
  *p = s.P;
  *q = s.Q;
  return CONV_OK;
}

conv_status_t conv2d_check(const conv2d_desc_t* desc, conv_algo_t algo) {
  Shape s;
  const conv_status_t st = validate(desc, &s);
  if (st != CONV_OK) return st;
  if (algo == CONV_ALGO_DEFAULT) algo = default_rule(s);
  return support(s, algo);
}

conv_status_t conv2d_workspace_bytes(const conv2d_desc_t* desc, conv_algo_t algo, size_t* bytes) {
  Shape s;
  conv_status_t st = validate(desc, &s);
  if (st != CONV_OK) return st;
  if (!bytes) return CONV_ERR_INVALID_ARG;
  if (algo == CONV_ALGO_DEFAULT) algo = default_rule(s);
  st = support(s, algo);
  if (st != CONV_OK) return st;
  *bytes = workspace_for(s, algo);
  return CONV_OK;
}

conv_algo_t conv2d_default_algo(const conv2d_desc_t* desc) {
  Shape s;
  if (validate(desc, &s) != CONV_OK) return CONV_ALGO_DEFAULT;
  return default_rule(s);
}

conv_status_t conv2d(const void* x, const void* w, const void* b, void* y, const conv2d_desc_t* desc,
                     conv_algo_t algo, void* workspace, size_t workspace_bytes, void* stream) {
  Shape s;
  const conv_status_t st = prepare_call(desc, &algo, &s, x, w, b, y, workspace, workspace_bytes, false);
  if (st != CONV_OK || s.N == 0) return st;
  return run(s, algo, x, w, nullptr, b, y, workspace, (hipStream_t)stream);
}

conv_status_t conv2d_static_scratch(const void* x, const void* w, const void* b, void* y, const conv2d_desc_t* desc,
                                    conv_algo_t algo, void* stream) {
  Shape s;
  conv_status_t st = validate(desc, &s);
  if (st != CONV_OK) return st;
  if (algo == CONV_ALGO_DEFAULT) algo = default_rule(s);
  st = support(s, algo);
  if (st != CONV_OK) return st;
  if (workspace_for(s, algo) > kScratchBytes) return CONV_ERR_WORKSPACE;
  if (s.N == 0) return CONV_OK;
  st = ensure_device();
  if (st != CONV_OK) return st;
  void* ws = scratch_for_current_device();
  if (!ws) return CONV_ERR_DEVICE;
  st = prepare_call(desc, &algo, &s, x, w, b, y, ws, kScratchBytes, false);
  if (st != CONV_OK) return st;
  return run(s, algo, x, w, nullptr, b, y, ws, (hipStream_t)stream);
}

size_t conv2d_static_scratch_capacity(void) { return kScratchBytes; }

conv_status_t conv2d_packed_filter_bytes(const conv2d_desc_t* desc, conv_algo_t algo, size_t* bytes) {
  Shape s;
  conv_status_t st = validate(desc, &s);
  if (st != CONV_OK) return st;
  if (!bytes) return CONV_ERR_INVALID_ARG;
  if (algo == CONV_ALGO_DEFAULT) algo = default_rule(s);
  st = support(s, algo);
  if (st != CONV_OK) return st;
  *bytes = packed_filter_bytes(s, algo);
  return CONV_OK;
}

conv_status_t conv2d_prepacked_workspace_bytes(const conv2d_desc_t* desc, conv_algo_t algo, size_t* bytes) {
  Shape s;
  conv_status_t st = validate(desc, &s);
  if (st != CONV_OK) return st;
  if (!bytes) return CONV_ERR_INVALID_ARG;
  if (algo == CONV_ALGO_DEFAULT) algo = default_rule(s);
  st = support(s, algo);
  if (st != CONV_OK) return st;
  *bytes = workspace_for(s, algo, true);
  return CONV_OK;
}

conv_status_t conv2d_pack_filters(const void* w, void* packed, const conv2d_desc_t* desc, conv_algo_t algo,
                                  void* stream) {
  Shape s;
  conv_status_t st = validate(desc, &s);
  if (st != CONV_OK) return st;
  if (algo == CONV_ALGO_DEFAULT) algo = default_rule(s);
  st = support(s, algo);
  if (st != CONV_OK) return st;
  if (!w || !packed) return CONV_ERR_INVALID_ARG;
  if (reinterpret_cast<uintptr_t>(packed) % 256 != 0) return CONV_ERR_INVALID_ARG;
  const size_t pbytes = packed_filter_bytes(s, algo);
  const size_t wbytes = (size_t)s.K * s.Cg * s.R * s.S * s.esize();
  if (overlaps(packed, pbytes, w, wbytes)) return CONV_ERR_INVALID_ARG;
  st = ensure_device();
  if (st != CONV_OK) return st;
  const hipStream_t hs = (hipStream_t)stream;
  if (algo == CONV_ALGO_IMPLICIT_GEMM) return from_hip(convsel::launch_implicit_pack(s, w, packed, hs));
  if (algo == CONV_ALGO_WINOGRAD) return from_hip(convsel::launch_wino_filter(s, w, packed, hs));
  if (algo == CONV_ALGO_IMPLICIT_PRECOMP_GEMM) return from_hip(convsel::precomp_pack(s, w, packed, hs));
  if (algo == CONV_ALGO_KN2ROW) return from_hip(convsel::kn2row_pack(s, w, packed, hs));
  if (algo == CONV_ALGO_SMM) return from_hip(convsel::smm_pack(s, w, packed, hs));
  return from_hip(convsel::launch_copy(w, packed, wbytes, hs));
}

conv_status_t conv2d_prepacked(const void* x, const void* packed, const void* b, void* y,
                               const conv2d_desc_t* desc, conv_algo_t algo, void* workspace, size_t workspace_bytes,
                               void* stream) {
  Shape s;
  const conv_status_t st = prepare_call(desc, &algo, &s, x, packed, b, y, workspace, workspace_bytes, true);
  if (st != CONV_OK || s.N == 0) return st;
  return run(s, algo, x, nullptr, packed, b, y, workspace, (hipStream_t)stream);
}

conv_status_t conv2d_describe(const conv2d_desc_t* desc, conv_algo_t algo, char* buf, size_t len) {
  Shape s;
  conv_status_t st = validate(desc, &s);
  if (st != CONV_OK) return st;
  if (!buf || len == 0) return CONV_ERR_INVALID_ARG;
  if (algo == CONV_ALGO_DEFAULT) algo = default_rule(s);
  st = support(s, algo);
  if (st != CONV_OK) return st;
  std::string d;
  switch (algo) {
    case CONV_ALGO_DIRECT:
      d = direct_describe(s);
      break;
    case CONV_ALGO_IMPLICIT_GEMM:
      d = convsel::implicit_gemm_describe(s);
      break;
    case CONV_ALGO_IM2COL_GEMM: {
      const int64_t nb = im2col_batch(s, nullptr);
      d = "im2col_gemm kernels=im2col_kernel;gemm_nt_kernel images_per_batch=" + std::to_string(nb);
      break;
    }
    case CONV_ALGO_WINOGRAD: {
      const WinoLayout L = wino_layout(s, true);
      d = "winograd kernels=wino_filter_kernel;wino_input_kernel;gemm_nt_kernel;wino_output_kernel "
          "images_per_batch=" + std::to_string(L.nb);
      break;
    }
    case CONV_ALGO_IMPLICIT_PRECOMP_GEMM:
      d = convsel::precomp_describe(s);
      break;
    case CONV_ALGO_KN2ROW:
      d = convsel::kn2row_describe(s);
      break;
    case CONV_ALGO_SMM:
      d = convsel::smm_describe(s);
      break;
    default:
      return CONV_ERR_INVALID_ARG;
  }
  d += " workspace=" + std::to_string(workspace_for(s, algo)) +
       " prepacked_workspace=" + std::to_string(workspace_for(s, algo, true)) +
       " packed_filters=" + std::to_string(packed_filter_bytes(s, algo));
  snprintf(buf, len, "%s", d.c_str());
  return CONV_OK;
}

conv_status_t conv2d_im2col(const void* x, void* col, const conv2d_desc_t* desc, void* stream) {
  Shape s;
  conv_status_t st = validate(desc, &s);
  if (st != CONV_OK) return st;
  if (s.N == 0) return CONV_OK;
  if (!x || !col) return CONV_ERR_INVALID_ARG;
  const size_t es = (size_t)s.esize();
  if (overlaps(col, (size_t)s.N * s.G * s.P * s.Q * s.Cg * s.R * s.S * es, x, (size_t)s.N * s.C * s.H * s.W * es))
    return CONV_ERR_INVALID_ARG;
  st = ensure_device();
  if (st != CONV_OK) return st;
  return from_hip(convsel::launch_im2col(s, x, col, 0, s.N, (hipStream_t)stream));
}

conv_status_t conv2d_winograd_filter_transform(const void* w, void* u, const conv2d_desc_t* desc, void* stream) {
  Shape s;
  conv_status_t st = validate(desc, &s);
  if (st != CONV_OK) return st;
  if (!winograd_ok(s)) return CONV_ERR_UNSUPPORTED;
  if (!w || !u) return CONV_ERR_INVALID_ARG;
  const size_t es = (size_t)s.esize();
  if (overlaps(u, (size_t)16 * s.K * s.C * es, w, (size_t)s.K * s.C * 9 * es)) return CONV_ERR_INVALID_ARG;
  st = ensure_device();
  if (st != CONV_OK) return st;
  return from_hip(convsel::launch_wino_filter(s, w, u, (hipStream_t)stream));
}

conv_status_t conv2d_winograd_input_transform(const void* x, void* v, const conv2d_desc_t* desc, void* stream) {
  Shape s;
  conv_status_t st = validate(desc, &s);
  if (st != CONV_OK) return st;
  if (!winograd_ok(s)) return CONV_ERR_UNSUPPORTED;
  if (s.N == 0) return CONV_OK;
  if (!x || !v) return CONV_ERR_INVALID_ARG;
  const size_t es = (size_t)s.esize();
  const int64_t T = s.N * ((s.P + 1) / 2) * ((s.Q + 1) / 2);
  if (T > kInt31 / s.C / 16) return CONV_ERR_INVALID_ARG;
  if (overlaps(v, (size_t)16 * T * s.C * es, x, (size_t)s.N * s.C * s.H * s.W * es)) return CONV_ERR_INVALID_ARG;
  st = ensure_device();
  if (st != CONV_OK) return st;
  return from_hip(convsel::launch_wino_input(s, x, v, 0, s.N, (hipStream_t)stream));
}

const char* conv2d_status_string(conv_status_t status) {
  switch (status) {
    case CONV_OK: return "ok";
    case CONV_ERR_INVALID_ARG: return "invalid argument";
    case CONV_ERR_UNSUPPORTED: return "algorithm not supported for this layer";
    case CONV_ERR_WORKSPACE: return "workspace too small";
    case CONV_ERR_DEVICE: return "device error";
    default: return "unknown";
  }
}

const char* conv2d_algo_name(conv_algo_t algo) {
  switch (algo) {
    case CONV_ALGO_DEFAULT: return "default";
    case CONV_ALGO_DIRECT: return "direct";
    case CONV_ALGO_IMPLICIT_GEMM: return "implicit_gemm";
    case CONV_ALGO_IM2COL_GEMM: return "im2col_gemm";
    case CONV_ALGO_WINOGRAD: return "winograd";
    case CONV_ALGO_IMPLICIT_PRECOMP_GEMM: return "implicit_precomp_gemm";
    case CONV_ALGO_KN2ROW: return "kn2row";
    case CONV_ALGO_SMM: return "smm";
    default: return "unknown";
  }
}

conv_status_t conv2d_algo_from_name(const char* name, conv_algo_t* algo) {
  if (!name || !algo) return CONV_ERR_INVALID_ARG;
  static const struct {
    const char* name;
    conv_algo_t algo;
  } table[] = {{"default", CONV_ALGO_DEFAULT},         {"direct", CONV_ALGO_DIRECT},
               {"implicit_gemm", CONV_ALGO_IMPLICIT_GEMM}, {"im2col_gemm", CONV_ALGO_IM2COL_GEMM},
               {"gemm", CONV_ALGO_IM2COL_GEMM},         {"winograd", CONV_ALGO_WINOGRAD},
               {"implicit_precomp_gemm", CONV_ALGO_IMPLICIT_PRECOMP_GEMM},
               {"kn2row", CONV_ALGO_KN2ROW},            {"smm", CONV_ALGO_SMM}};
  for (const auto& e : table)
    if (strcmp(name, e.name) == 0) {
      *algo = e.algo;
      return CONV_OK;
    }
  return CONV_ERR_INVALID_ARG;
}

}  // extern "C"

namespace convsel {

// For the model executor (not part of the public ABI): conv2d_prepacked() of
// an implicit GEMM layer whose epilogue also adds `res` (N x K x P x Q, the
// layer's dtype) before the ReLU.
conv_status_t conv2d_prepacked_residual(const void* x, const void* packed, const void* b, const void* res, void* y,
                                        const conv2d_desc_t* desc, conv_algo_t algo, void* workspace,
                                        size_t workspace_bytes, void* stream) {
  Shape s;
  const conv_status_t st = prepare_call(desc, &algo, &s, x, packed, b, y, workspace, workspace_bytes, true);
  if (st != CONV_OK || s.N == 0) return st;
  if (algo != CONV_ALGO_IMPLICIT_GEMM) return CONV_ERR_UNSUPPORTED;
  const size_t ybytes = (size_t)s.N * s.K * s.P * s.Q * s.esize();
  if (!res || overlaps(y, ybytes, res, ybytes)) return CONV_ERR_INVALID_ARG;
  return from_hip(launch_implicit_main(s, x, packed, b, y, workspace, (hipStream_t)stream, res));
}

}  // namespace convsel
