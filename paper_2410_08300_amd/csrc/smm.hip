// SMM, scalar matrix multiplication with zero packing (paper, Sec. II-B
// item (c)): no matrix product at all.  Output plane k of an image is the sum,
// over input channels c and taps (r, s), of the input plane c shifted by the
// tap and scaled by the single number w[k][c][r][s]:
//   y[n][k] = b[k] + sum_{c,r,s} w[k][c][r][s] * shift_{r,s}(xz[n][g*Cg + c])
// where xz is the input "zero packed": copied once into planes that already
// hold the padding,
//   xz[n][c][v][u] = x[n][c][v - ph][u - pw]  (zero outside the image),
//   v < Hz = (P-1)*sh + (R-1)*dh + 1,  u < Wz = (Q-1)*sw + (S-1)*dw + 1,
// so that shift_{r,s} reads xz[.][p*sh + r*dh][q*sw + s*dw] for every output
// pixel without a bounds check.
//
// Kernel: a workgroup owns KB consecutive output channels of one group and
// 256 output pixels of one image, one pixel per thread.  Each step reads one
// element of the shifted plane per thread and scales it by KB filter values;
// the filters are repacked so that the KB values of one (c, r, s) are
// contiguous and the same for the whole workgroup, so they arrive as a
// single scalar load per step.  fp32 arithmetic on the vector ALUs (bf16
// data is widened on load and the result rounded once).
#include <stdio.h>
#include <string>

#include "common.hpp"
#include "kernels.hpp"

namespace convsel {

namespace {

constexpr size_t kZpCap = (size_t)1 << 30;  // zero-packed input of a batch of images, near 1 GiB
constexpr int kSmmPix = 256;

int smm_kb(const Shape& s) { return s.Kg >= 16 ? 16 : 8; }

// Zero packing of images n0 .. n0+nb-1 (`xz` holds nb images).
template <typename T>
__global__ __launch_bounds__(256) void smm_zero_pack_kernel(const T* __restrict__ x, T* __restrict__ xz, int64_t total,
                                                            int H, int W, int Hz, int Wz, int ph, int pw) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= total) return;
  const int u = static_cast<int>(i % Wz);
  const int v = static_cast<int>((i / Wz) % Hz);
  const int64_t plane = i / (static_cast<int64_t>(Wz) * Hz);  // n*C + c
  const int ih = v - ph, iw = u - pw;
  T val = elem<T>::from_f32(0.f);
  if (ih >= 0 && ih < H && iw >= 0 && iw < W) val = x[plane * H * W + static_cast<int64_t>(ih) * W + iw];
  xz[i] = val;
}

// Filters as [g][k block][c][r][s][KB] (zero rows past Kg).
template <typename T>
__global__ __launch_bounds__(256) void smm_pack_filters_kernel(const T* __restrict__ w, T* __restrict__ wp, int Kg,
                                                               int Cg, int RS, int KB, int kblocks, int64_t total) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= total) return;
  const int kb = static_cast<int>(i % KB);
  int64_t t = i / KB;
  const int crs = static_cast<int>(t % (static_cast<int64_t>(Cg) * RS));
  t /= static_cast<int64_t>(Cg) * RS;
  const int blk = static_cast<int>(t % kblocks);
  const int64_t g = t / kblocks;
  const int k = blk * KB + kb;
  T v = elem<T>::from_f32(0.f);
  if (k < Kg) v = w[(g * Kg + k) * Cg * RS + crs];
  wp[i] = v;
}

struct SmmArgs {
  const void* xz;   // zero-packed images of this batch
  const void* wp;
  const void* b;
  void* y;          // first output image of the batch
  int C, Cg, K, Kg, G, kblocks;
  int Hz, Wz, P, Q, R, S, sh, sw, dh, dw, relu;
  int ptiles;       // pixel tiles per image
};

template <typename T, int KB>
__global__ __launch_bounds__(kSmmPix) void smm_kernel(SmmArgs a) {
  const int pt = blockIdx.x % a.ptiles;
  const int n = blockIdx.x / a.ptiles;
  const int blk = blockIdx.y % a.kblocks;
  const int g = blockIdx.y / a.kblocks;
  const int PQ = a.P * a.Q;
  const int pix = pt * kSmmPix + threadIdx.x;
  const bool live = pix < PQ;
  const int pp = live ? pix : PQ - 1;
  const int p = pp / a.Q, q = pp - (pp / a.Q) * a.Q;
  const int RS = a.R * a.S;
  const int64_t plane = static_cast<int64_t>(a.Hz) * a.Wz;
  const T* xz = reinterpret_cast<const T*>(a.xz) + (static_cast<int64_t>(n) * a.C + g * a.Cg) * plane +
                static_cast<int64_t>(p * a.sh) * a.Wz + q * a.sw;
  const T* wp = reinterpret_cast<const T*>(a.wp) + (static_cast<int64_t>(g) * a.kblocks + blk) * a.Cg * RS * KB;

  float acc[KB];
#pragma unroll
  for (int i = 0; i < KB; ++i) acc[i] = 0.f;
  for (int c = 0; c < a.Cg; ++c) {
    for (int r = 0; r < a.R; ++r) {
      const T* row = xz + static_cast<int64_t>(c) * plane + r * a.dh * a.Wz;
      for (int s = 0; s < a.S; ++s) {
        const float xv = elem<T>::load(row + s * a.dw);
        const T* wv = wp + ((c * a.R + r) * a.S + s) * KB;  // uniform over the workgroup
#pragma unroll
        for (int i = 0; i < KB; ++i) acc[i] += elem<T>::load(wv + i) * xv;
      }
    }
  }
  if (!live) return;
  const int k0 = g * a.Kg + blk * KB;
  T* y = reinterpret_cast<T*>(a.y) + (static_cast<int64_t>(n) * a.K + k0) * PQ + pix;
  const T* bias = reinterpret_cast<const T*>(a.b);
#pragma unroll
  for (int i = 0; i < KB; ++i) {
    if (blk * KB + i >= a.Kg) continue;
    float v = acc[i] + (bias ? elem<T>::load(bias + k0 + i) : 0.f);
    if (a.relu) v = fmaxf(v, 0.f);
    elem<T>::store(y + static_cast<int64_t>(i) * PQ, v);
  }
}

struct SmmLayout {
  int Hz, Wz;
  int64_t nb;
  size_t zp_bytes;
};

SmmLayout smm_layout(const Shape& s) {
  SmmLayout L;
  L.Hz = (int)((s.P - 1) * s.sh + (s.R - 1) * s.dh + 1);
  L.Wz = (int)((s.Q - 1) * s.sw + (s.S - 1) * s.dw + 1);
  const size_t per_img = (size_t)s.C * L.Hz * L.Wz * s.esize();
  int64_t nb = (int64_t)(kZpCap / per_img);
  if (nb < 1) nb = 1;
  if (nb > s.N) nb = s.N;
  L.nb = nb;
  L.zp_bytes = s.N > 0 ? (size_t)nb * per_img : 0;
  return L;
}

template <typename T, int KB>
hipError_t smm_launch(const SmmArgs& a, int64_t cnt, hipStream_t stream) {
  const dim3 grid((unsigned)(cnt * a.ptiles), (unsigned)(a.G * a.kblocks));
  hipLaunchKernelGGL((smm_kernel<T, KB>), grid, dim3(kSmmPix), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

bool smm_applies(const Shape& s) {
  // The zero-packed planes of one image, and the reach of one filter row,
  // must stay within 32-bit element counts.
  const int64_t Hz = (s.P - 1) * s.sh + (s.R - 1) * s.dh + 1;
  const int64_t Wz = (s.Q - 1) * s.sw + (s.S - 1) * s.dw + 1;
  const int64_t kblocks = (s.Kg + smm_kb(s) - 1) / smm_kb(s);
  return Hz * Wz < ((int64_t)1 << 31) / s.C && (int64_t)s.Cg * s.R * s.S * 16 < ((int64_t)1 << 31) &&
         s.G * kblocks <= 65535;
}

size_t smm_packed_bytes(const Shape& s) {
  const int KB = smm_kb(s);
  const int64_t kblocks = (s.Kg + KB - 1) / KB;
  return (size_t)s.G * kblocks * KB * s.Cg * s.R * s.S * s.esize();
}

size_t smm_zero_pack_bytes(const Shape& s) { return smm_layout(s).zp_bytes; }

hipError_t smm_pack(const Shape& s, const void* w, void* wp, hipStream_t stream) {
  const int KB = smm_kb(s);
  const int kblocks = (int)((s.Kg + KB - 1) / KB);
  const int64_t total = (int64_t)s.G * kblocks * KB * s.Cg * s.R * s.S;
  const dim3 grid((unsigned)((total + 255) / 256));
  if (s.dtype == DT_F32)
    hipLaunchKernelGGL(smm_pack_filters_kernel<float>, grid, dim3(256), 0, stream, reinterpret_cast<const float*>(w),
                       reinterpret_cast<float*>(wp), (int)s.Kg, (int)s.Cg, (int)(s.R * s.S), KB, kblocks, total);
  else
    hipLaunchKernelGGL(smm_pack_filters_kernel<bf16_t>, grid, dim3(256), 0, stream,
                       reinterpret_cast<const bf16_t*>(w), reinterpret_cast<bf16_t*>(wp), (int)s.Kg, (int)s.Cg,
                       (int)(s.R * s.S), KB, kblocks, total);
  return hipGetLastError();
}

hipError_t smm_main(const Shape& s, const void* x, const void* wp, const void* b, void* y, void* zp,
                    hipStream_t stream) {
  const SmmLayout L = smm_layout(s);
  const int KB = smm_kb(s);
  const int64_t HW = s.H * s.W, PQ = s.P * s.Q;
  for (int64_t n0 = 0; n0 < s.N; n0 += L.nb) {
    const int64_t cnt = s.N - n0 < L.nb ? s.N - n0 : L.nb;
    const int64_t total = cnt * s.C * L.Hz * L.Wz;
    const dim3 grid((unsigned)((total + 255) / 256));
    const char* xb = reinterpret_cast<const char*>(x) + (size_t)n0 * s.C * HW * s.esize();
    if (s.dtype == DT_F32)
      hipLaunchKernelGGL(smm_zero_pack_kernel<float>, grid, dim3(256), 0, stream, reinterpret_cast<const float*>(xb),
                         reinterpret_cast<float*>(zp), total, (int)s.H, (int)s.W, L.Hz, L.Wz, s.ph, s.pw);
    else
      hipLaunchKernelGGL(smm_zero_pack_kernel<bf16_t>, grid, dim3(256), 0, stream,
                         reinterpret_cast<const bf16_t*>(xb), reinterpret_cast<bf16_t*>(zp), total, (int)s.H,
                         (int)s.W, L.Hz, L.Wz, s.ph, s.pw);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    SmmArgs a;
    a.xz = zp;
    a.wp = wp;
    a.b = b;
    a.y = reinterpret_cast<char*>(y) + (size_t)n0 * s.K * PQ * s.esize();
    a.C = (int)s.C; a.Cg = (int)s.Cg; a.K = (int)s.K; a.Kg = (int)s.Kg; a.G = s.G;
    a.kblocks = (int)((s.Kg + KB - 1) / KB);
    a.Hz = L.Hz; a.Wz = L.Wz; a.P = (int)s.P; a.Q = (int)s.Q; a.R = (int)s.R; a.S = (int)s.S;
    a.sh = s.sh; a.sw = s.sw; a.dh = s.dh; a.dw = s.dw;
    a.relu = s.relu ? 1 : 0;
    a.ptiles = (int)((PQ + kSmmPix - 1) / kSmmPix);
    if (s.dtype == DT_F32)
      e = KB == 16 ? smm_launch<float, 16>(a, cnt, stream) : smm_launch<float, 8>(a, cnt, stream);
    else
      e = KB == 16 ? smm_launch<bf16_t, 16>(a, cnt, stream) : smm_launch<bf16_t, 8>(a, cnt, stream);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

std::string smm_describe(const Shape& s) {
  const SmmLayout L = smm_layout(s);
  char buf[256];
  snprintf(buf, sizeof(buf),
           "smm kernels=smm_pack_filters_kernel;smm_zero_pack_kernel;smm_kernel<%d> zero_packed_plane=%dx%d "
           "images_per_batch=%lld",
           smm_kb(s), L.Hz, L.Wz, (long long)L.nb);
  return buf;
}

}  // namespace convsel
