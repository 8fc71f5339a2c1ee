// KN2ROW (paper, Sec. II-B item (b)): the filter, not the input, is turned
// into matrix rows.  Each tap (r, s) of the filter is a 1x1 convolution, and
// the R*S of them share one input, so stacking the taps' filter matrices
//   Wst[g][(r*S + s)*Kg + k][c] = w[g*Kg + k][c][r][s]
// turns the whole layer into ONE GEMM per image and group over the input as
// it lies in memory (channels x pixels, no column matrix):
//   Z[n][g][(r, s, k)][h*W + w] = sum_c Wst[g][(r, s, k)][c] * x[n][g*Cg + c][h][w],
// followed by a shift-and-add of the R*S partial planes into the output:
//   y[n][g*Kg + k][p][q] = b + sum_{r,s} Z[n][g][(r, s, k)][p*sh - ph + r*dh][q*sw - pw + s*dw]
// over the taps whose input position lies inside the image (the others read
// padding, i.e. zero).
//
// The GEMM is the library's MFMA GEMM with its B operand read column-major
// (an NCHW image is channels x pixels); Z is kept in fp32 so that the sum of
// the R*S partial products is rounded once, in the output.  The shift-add
// kernel gives each thread one output element: consecutive threads take
// consecutive q, so each partial plane is read along its rows, once.
#include <stdio.h>
#include <string>

#include "common.hpp"
#include "kernels.hpp"

namespace convsel {

namespace {

constexpr size_t kZCap = (size_t)1 << 30;  // Z for a batch of images, near 1 GiB

template <typename T>
__global__ __launch_bounds__(256) void kn2row_pack_kernel(const T* __restrict__ w, T* __restrict__ wst, int Kg, int Cg,
                                                          int RS, int64_t total) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= total) return;
  // Destination order [g][tap][k][c].
  const int c = static_cast<int>(i % Cg);
  int64_t t = i / Cg;
  const int k = static_cast<int>(t % Kg);
  t /= Kg;
  const int tap = static_cast<int>(t % RS);
  const int64_t g = t / RS;
  wst[i] = w[((g * Kg + k) * Cg + c) * RS + tap];
}

struct ShiftArgs {
  const float* z;    // [nb][G][RS*Kg][H*W]
  const void* b;
  void* y;           // first output image of the batch
  int nb, K, Kg, G, H, W, P, Q, R, S, sh, sw, ph, pw, dh, dw, relu;
};

template <typename T>
__global__ __launch_bounds__(256) void kn2row_shift_add_kernel(ShiftArgs a) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int64_t PQ = static_cast<int64_t>(a.P) * a.Q;
  const int64_t total = a.nb * a.K * PQ;
  if (i >= total) return;
  const int q = static_cast<int>(i % a.Q);
  const int p = static_cast<int>((i / a.Q) % a.P);
  const int k = static_cast<int>((i / PQ) % a.K);
  const int64_t n = i / (PQ * a.K);
  const int g = k / a.Kg, kk = k - g * a.Kg;
  const int64_t HW = static_cast<int64_t>(a.H) * a.W;
  const int RS = a.R * a.S;
  const float* zg = a.z + (n * a.G + g) * (static_cast<int64_t>(RS) * a.Kg) * HW;
  float acc = a.b ? elem<T>::load(reinterpret_cast<const T*>(a.b) + k) : 0.f;
  for (int r = 0; r < a.R; ++r) {
    const int ih = p * a.sh - a.ph + r * a.dh;
    if (ih < 0 || ih >= a.H) continue;
    for (int s = 0; s < a.S; ++s) {
      const int iw = q * a.sw - a.pw + s * a.dw;
      if (iw < 0 || iw >= a.W) continue;
      acc += zg[(static_cast<int64_t>(r * a.S + s) * a.Kg + kk) * HW + static_cast<int64_t>(ih) * a.W + iw];
    }
  }
  if (a.relu) acc = fmaxf(acc, 0.f);
  elem<T>::store(reinterpret_cast<T*>(a.y) + i, acc);
}

int64_t z_batch(const Shape& s, size_t* bytes) {
  const size_t per_img = (size_t)s.G * s.R * s.S * s.Kg * s.H * s.W * sizeof(float);
  int64_t nb = (int64_t)(kZCap / per_img);
  if (nb < 1) nb = 1;
  if (nb > s.N) nb = s.N;
  if (bytes) *bytes = (size_t)nb * per_img;
  return nb;
}

}  // namespace

bool kn2row_applies(const Shape& s) {
  // One image's partial planes must be indexable in 32 bits per group GEMM.
  const int64_t rows = s.R * s.S * s.Kg;
  return rows < ((int64_t)1 << 31) / (s.H * s.W) && (rows + 63) / 64 <= 65535;  // GEMM grid rows
}

size_t kn2row_packed_bytes(const Shape& s) { return (size_t)s.K * s.Cg * s.R * s.S * s.esize(); }

size_t kn2row_z_bytes(const Shape& s) {
  size_t b = 0;
  if (s.N > 0) z_batch(s, &b);
  return b;
}

hipError_t kn2row_pack(const Shape& s, const void* w, void* wst, hipStream_t stream) {
  const int64_t total = s.K * s.Cg * s.R * s.S;
  const dim3 grid((unsigned)((total + 255) / 256));
  if (s.dtype == DT_F32)
    hipLaunchKernelGGL(kn2row_pack_kernel<float>, grid, dim3(256), 0, stream, reinterpret_cast<const float*>(w),
                       reinterpret_cast<float*>(wst), (int)s.Kg, (int)s.Cg, (int)(s.R * s.S), total);
  else
    hipLaunchKernelGGL(kn2row_pack_kernel<bf16_t>, grid, dim3(256), 0, stream, reinterpret_cast<const bf16_t*>(w),
                       reinterpret_cast<bf16_t*>(wst), (int)s.Kg, (int)s.Cg, (int)(s.R * s.S), total);
  return hipGetLastError();
}

hipError_t kn2row_main(const Shape& s, const void* x, const void* wst, const void* b, void* y, void* z,
                       hipStream_t stream) {
  const int64_t nb = z_batch(s, nullptr);
  const int64_t RS = s.R * s.S, HW = s.H * s.W, PQ = s.P * s.Q;
  for (int64_t n0 = 0; n0 < s.N; n0 += nb) {
    const int64_t cnt = s.N - n0 < nb ? s.N - n0 : nb;
    GemmArgs g;
    g.A = wst;
    g.B = reinterpret_cast<const char*>(x) + (size_t)n0 * s.C * HW * s.esize();
    g.C = z;
    g.bias = nullptr;
    g.M = (int)(RS * s.Kg); g.N = (int)HW; g.Kred = (int)s.Cg;
    g.lda = s.Cg; g.ldb = HW; g.ldc = HW;
    g.batch = (int)(cnt * s.G); g.bdiv = s.G;
    g.sA0 = 0; g.sA1 = RS * s.Kg * s.Cg;             // group g's stacked filters
    g.sB0 = s.C * HW; g.sB1 = s.Cg * HW;             // image, group's channels
    g.sC0 = s.G * RS * s.Kg * HW; g.sC1 = RS * s.Kg * HW;
    g.sBias1 = 0;
    g.relu = 0;
    g.out_f32 = 1;
    g.b_kmajor = 1;
    hipError_t e = launch_gemm_nt(s.dtype, g, stream);
    if (e != hipSuccess) return e;
    ShiftArgs a;
    a.z = reinterpret_cast<const float*>(z);
    a.b = b;
    a.y = reinterpret_cast<char*>(y) + (size_t)n0 * s.K * PQ * s.esize();
    a.nb = (int)cnt; a.K = (int)s.K; a.Kg = (int)s.Kg; a.G = s.G;
    a.H = (int)s.H; a.W = (int)s.W; a.P = (int)s.P; a.Q = (int)s.Q; a.R = (int)s.R; a.S = (int)s.S;
    a.sh = s.sh; a.sw = s.sw; a.ph = s.ph; a.pw = s.pw; a.dh = s.dh; a.dw = s.dw;
    a.relu = s.relu ? 1 : 0;
    const int64_t total = cnt * s.K * PQ;
    const dim3 grid((unsigned)((total + 255) / 256));
    if (s.dtype == DT_F32)
      hipLaunchKernelGGL(kn2row_shift_add_kernel<float>, grid, dim3(256), 0, stream, a);
    else
      hipLaunchKernelGGL(kn2row_shift_add_kernel<bf16_t>, grid, dim3(256), 0, stream, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

std::string kn2row_describe(const Shape& s) {
  char buf[256];
  snprintf(buf, sizeof(buf),
           "kn2row kernels=kn2row_pack_kernel;gemm_nt_kernel(b_kmajor, fp32 out);kn2row_shift_add_kernel "
           "gemm=%lldx%lldx%lld images_per_batch=%lld",
           (long long)(s.R * s.S * s.Kg), (long long)(s.H * s.W), (long long)s.Cg, (long long)z_batch(s, nullptr));
  return buf;
}

}  // namespace convsel
