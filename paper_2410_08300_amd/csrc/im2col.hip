// IM2COL (paper, Sec. II-B item (a); the "GEMM" algorithm of Sec. V-B item
// (c)): the column matrix that turns the convolution into a matrix product.
// Layout [image][group][P*Q][Cg*R*S]: one row per output pixel holding its
// receptive field in (c, r, s) order, zero where it leaves the image, so both
// GEMM operands (filters K x Cg*R*S and this matrix) are contiguous along the
// reduction.  A pure gather: every element is a bit copy of an input element.
//
// A workgroup writes a run of whole rows; consecutive threads write
// consecutive elements (coalesced stores), and the reads of neighbouring taps
// of one row fall on neighbouring input columns.
#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace convsel {

namespace {

struct Im2colArgs {
  const void* x;
  void* col;
  int C, H, W, R, S, P, Q;
  int sh, sw, ph, pw, dh, dw;
  int G, Cg;
  int64_t n0;
  int64_t rows;       // nb * G * P * Q
  int rows_per_block;
};

template <typename T>
__global__ __launch_bounds__(256) void im2col_kernel(Im2colArgs a) {
  const int RS = a.R * a.S;
  const int crs = a.Cg * RS;
  const int PQ = a.P * a.Q;
  const int64_t row0 = static_cast<int64_t>(blockIdx.x) * a.rows_per_block;
  const int64_t rows_here = min(static_cast<int64_t>(a.rows_per_block), a.rows - row0);
  const int count = static_cast<int>(rows_here) * crs;
  const T* x = reinterpret_cast<const T*>(a.x);
  T* col = reinterpret_cast<T*>(a.col) + row0 * crs;
  for (int e = threadIdx.x; e < count; e += 256) {
    const int rl = e / crs, ci = e - rl * crs;
    const int64_t row = row0 + rl;
    const int pq = static_cast<int>(row % PQ);
    const int64_t ng = row / PQ;
    const int g = static_cast<int>(ng % a.G);
    const int64_t n = a.n0 + ng / a.G;
    const int c = ci / RS, rs = ci - c * RS;
    const int r = rs / a.S, s = rs - r * a.S;
    const int p = pq / a.Q, q = pq - p * a.Q;
    const int ih = p * a.sh - a.ph + r * a.dh, iw = q * a.sw - a.pw + s * a.dw;
    T v = elem<T>::from_f32(0.f);
    if (ih >= 0 && ih < a.H && iw >= 0 && iw < a.W)
      v = x[((n * a.C + g * a.Cg + c) * a.H + ih) * a.W + iw];
    col[e] = v;
  }
}

// The same matrix when a row's length Cg*R*S is a multiple of the 16-byte
// unit: one thread per 16-byte unit of a row (UE consecutive (c, r, s)
// elements), consecutive threads along the row, so every store is one whole
// 16-byte unit and a wave writes 1 KiB of consecutive rows.  The UE input
// elements are gathered with the tap indices stepped incrementally.
template <typename T>
__global__ __launch_bounds__(256) void im2col_vec_kernel(Im2colArgs a, int64_t units) {
  constexpr int UE = elem<T>::per16;
  const int RS = a.R * a.S;
  const int CU = a.Cg * RS / UE;  // units per row
  const int PQ = a.P * a.Q;
  const T* x = reinterpret_cast<const T*>(a.x);
  for (int64_t u = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; u < units;
       u += static_cast<int64_t>(gridDim.x) * 256) {
    const int64_t row = u / CU;
    const int cu = static_cast<int>(u - row * CU);
    const int pq = static_cast<int>(row % PQ);
    const int64_t ng = row / PQ;
    const int g = static_cast<int>(ng % a.G);
    const int64_t n = a.n0 + ng / a.G;
    const int p = pq / a.Q, q = pq - p * a.Q;
    const int ci0 = cu * UE;
    int c = ci0 / RS, rs = ci0 - c * RS;
    int r = rs / a.S, s = rs - r * a.S;
    const T* xn = x + (n * a.C + g * a.Cg) * static_cast<int64_t>(a.H) * a.W;
    const int h0 = p * a.sh - a.ph, w0 = q * a.sw - a.pw;
    uint32_t e[UE];
#pragma unroll
    for (int t = 0; t < UE; ++t) {
      const int ih = h0 + r * a.dh, iw = w0 + s * a.dw;
      const bool in = ih >= 0 && ih < a.H && iw >= 0 && iw < a.W;
      const uint32_t bits = load_bits(xn + (in ? (static_cast<int64_t>(c) * a.H + ih) * a.W + iw : 0));
      e[t] = in ? bits : 0u;
      if (++s == a.S) {
        s = 0;
        if (++r == a.R) {
          r = 0;
          ++c;
        }
      }
    }
    vec16 v;
    pack16<T>(v, e);
    store16(reinterpret_cast<T*>(a.col) + u * UE, v);
  }
}

}  // namespace

hipError_t launch_im2col(const Shape& s, const void* x, void* col, int64_t n0, int64_t nb,
                         hipStream_t stream) {
  Im2colArgs a;
  a.x = x; a.col = col;
  a.C = (int)s.C; a.H = (int)s.H; a.W = (int)s.W; a.R = (int)s.R; a.S = (int)s.S;
  a.P = (int)s.P; a.Q = (int)s.Q;
  a.sh = s.sh; a.sw = s.sw; a.ph = s.ph; a.pw = s.pw; a.dh = s.dh; a.dw = s.dw;
  a.G = s.G; a.Cg = (int)s.Cg;
  a.n0 = n0;
  a.rows = nb * s.G * s.P * s.Q;
  const int64_t crs = s.Cg * s.R * s.S;
  const int ue = s.dtype == DT_F32 ? 4 : 8;
  if (crs % ue == 0 && reinterpret_cast<uintptr_t>(col) % 16 == 0) {
    const int64_t units = a.rows * (crs / ue);
    const int64_t blocks = std::min<int64_t>((units + 255) / 256, 65536);
    if (s.dtype == DT_F32)
      hipLaunchKernelGGL(im2col_vec_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, stream, a, units);
    else
      hipLaunchKernelGGL(im2col_vec_kernel<bf16_t>, dim3((unsigned)blocks), dim3(256), 0, stream, a, units);
    return hipGetLastError();
  }
  a.rows_per_block = (int)(4096 / crs > 0 ? 4096 / crs : 1);
  const int64_t blocks = (a.rows + a.rows_per_block - 1) / a.rows_per_block;
  if (s.dtype == DT_F32)
    hipLaunchKernelGGL(im2col_kernel<float>, dim3((unsigned)blocks), dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(im2col_kernel<bf16_t>, dim3((unsigned)blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace convsel
