// Winograd minimal filtering F(2x2, 3x3) (paper, Sec. V-B item (d), after
// Lavin and Gray 2016).  For a 4x4 input tile d and a 3x3 filter g, the 2x2
// output tile of the correlation is
//     Y = A^T [ (G g G^T) (.) (B^T d B) ] A
// with (.) the elementwise product, summed over input channels, so the
// 16 elementwise positions become 16 independent GEMMs:
//     M[xi,nu] (K x T) = U[xi,nu] (K x C) * V[xi,nu]^T (C x T).
// Four kernels: filter transform (U), input transform (V), the batched MFMA
// GEMM (gemm.hip), output transform (y).  U and V are kept in the data type
// (bf16 data: rounded after the fp32 transform), M in fp32.
//   B^T = [1 0 -1 0; 0 1 1 0; 0 -1 1 0; 0 1 0 -1]
//   G   = [1 0 0; 1/2 1/2 1/2; 1/2 -1/2 1/2; 0 0 1]
//   A^T = [1 1 1 0; 0 1 -1 -1]
#include "common.hpp"
#include "kernels.hpp"

namespace convsel {

namespace {

// U[xi*4+nu][k][c]; one thread per (k, c), c fastest (coalesced stores).
template <typename T>
__global__ __launch_bounds__(256) void wino_filter_kernel(const T* __restrict__ w, T* __restrict__ U, int K, int C) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= static_cast<int64_t>(K) * C) return;
  const T* g = w + idx * 9;
  float f[3][3];
#pragma unroll
  for (int i = 0; i < 3; ++i)
#pragma unroll
    for (int j = 0; j < 3; ++j) f[i][j] = elem<T>::to_f32(g[i * 3 + j]);
  // t = G f (4 x 3)
  float t[4][3];
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    t[0][j] = f[0][j];
    t[1][j] = 0.5f * (f[0][j] + f[1][j] + f[2][j]);
    t[2][j] = 0.5f * (f[0][j] - f[1][j] + f[2][j]);
    t[3][j] = f[2][j];
  }
  const int64_t plane = static_cast<int64_t>(K) * C;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float u[4] = {t[i][0], 0.5f * (t[i][0] + t[i][1] + t[i][2]), 0.5f * (t[i][0] - t[i][1] + t[i][2]),
                        t[i][2]};
#pragma unroll
    for (int j = 0; j < 4; ++j) U[(i * 4 + j) * plane + idx] = elem<T>::from_f32(u[j]);
  }
}

constexpr int TB = 8;   // tiles per workgroup along a tile row
constexpr int CB = 32;  // channels per workgroup

// V[xi*4+nu][t][c] for the tiles of images n0 .. n0+nb-1 (t counted from n0).
// A workgroup stages the 4 x (2*TB+2) input window of TB tiles for CB
// channels in LDS (coalesced row reads), then each thread transforms one
// (tile, channel) pair; consecutive threads write consecutive channels.
template <typename T>
__global__ __launch_bounds__(256) void wino_input_kernel(const T* __restrict__ x, T* __restrict__ V, int C, int H,
                                                         int W, int ph, int pw, int TP, int TQ, int64_t n0,
                                                         int64_t Tc) {
  __shared__ float tile[CB][4][2 * TB + 2];
  const int tqb = (TQ + TB - 1) / TB;
  const int tp = blockIdx.x / tqb, tq0 = (blockIdx.x % tqb) * TB;
  const int c0 = blockIdx.y * CB;
  const int nl = blockIdx.z;
  const int64_t n = n0 + nl;
  const int ih0 = 2 * tp - ph, iw0 = 2 * tq0 - pw;
  for (int i = threadIdx.x; i < CB * 4 * (2 * TB + 2); i += 256) {
    const int c = i / (4 * (2 * TB + 2)), rem = i % (4 * (2 * TB + 2));
    const int r = rem / (2 * TB + 2), col = rem % (2 * TB + 2);
    const int ih = ih0 + r, iw = iw0 + col;
    float v = 0.f;
    if (c0 + c < C && ih >= 0 && ih < H && iw >= 0 && iw < W)
      v = elem<T>::to_f32(x[((n * C + c0 + c) * H + ih) * W + iw]);
    tile[c][r][col] = v;
  }
  __syncthreads();
  const int c = threadIdx.x % CB, tb = threadIdx.x / CB;
  const int tq = tq0 + tb;
  if (tq >= TQ || c0 + c >= C) return;
  float d[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) d[i][j] = tile[c][i][2 * tb + j];
  // s = B^T d
  float s[4][4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    s[0][j] = d[0][j] - d[2][j];
    s[1][j] = d[1][j] + d[2][j];
    s[2][j] = d[2][j] - d[1][j];
    s[3][j] = d[1][j] - d[3][j];
  }
  const int64_t t = (static_cast<int64_t>(nl) * TP + tp) * TQ + tq;
  const int64_t plane = Tc * C;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float v[4] = {s[i][0] - s[i][2], s[i][1] + s[i][2], s[i][2] - s[i][1], s[i][1] - s[i][3]};
#pragma unroll
    for (int j = 0; j < 4; ++j) V[(i * 4 + j) * plane + t * C + c0 + c] = elem<T>::from_f32(v[j]);
  }
}

// y tiles from M[xi*4+nu][k][t] (fp32); one thread per (k, t), t fastest.
template <typename T>
__global__ __launch_bounds__(256) void wino_output_kernel(const float* __restrict__ M, const T* __restrict__ bias,
                                                          T* __restrict__ y, int K, int P, int Q, int TP, int TQ,
                                                          int64_t n0, int64_t Tc, int relu) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= static_cast<int64_t>(K) * Tc) return;
  const int k = static_cast<int>(idx / Tc);
  const int64_t t = idx - static_cast<int64_t>(k) * Tc;
  const int tq = static_cast<int>(t % TQ);
  const int tp = static_cast<int>((t / TQ) % TP);
  const int64_t nl = t / (static_cast<int64_t>(TQ) * TP);
  const int64_t plane = static_cast<int64_t>(K) * Tc;
  float m[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) m[i][j] = M[(i * 4 + j) * plane + idx];
  // a = A^T m (2 x 4), out = a A (2 x 2)
  float a[2][4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    a[0][j] = m[0][j] + m[1][j] + m[2][j];
    a[1][j] = m[1][j] - m[2][j] - m[3][j];
  }
  const float bv = bias ? elem<T>::to_f32(bias[k]) : 0.f;
  const int64_t n = n0 + nl;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int p = 2 * tp + i;
    if (p >= P) continue;
    const float o[2] = {a[i][0] + a[i][1] + a[i][2], a[i][1] - a[i][2] - a[i][3]};
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int q = 2 * tq + j;
      if (q >= Q) continue;
      float v = o[j] + bv;
      if (relu) v = fmaxf(v, 0.f);
      y[((n * K + k) * P + p) * Q + q] = elem<T>::from_f32(v);
    }
  }
}

}  // namespace

hipError_t launch_wino_filter(const Shape& s, const void* w, void* U, hipStream_t stream) {
  const int64_t total = s.K * s.C;
  const dim3 grid((unsigned)((total + 255) / 256));
  if (s.dtype == DT_F32)
    hipLaunchKernelGGL(wino_filter_kernel<float>, grid, dim3(256), 0, stream, (const float*)w, (float*)U,
                       (int)s.K, (int)s.C);
  else
    hipLaunchKernelGGL(wino_filter_kernel<bf16_t>, grid, dim3(256), 0, stream, (const bf16_t*)w, (bf16_t*)U,
                       (int)s.K, (int)s.C);
  return hipGetLastError();
}

hipError_t launch_wino_input(const Shape& s, const void* x, void* V, int64_t n0, int64_t nb,
                             hipStream_t stream) {
  const int TP = (int)((s.P + 1) / 2), TQ = (int)((s.Q + 1) / 2);
  const int64_t Tc = nb * TP * TQ;
  const dim3 grid((unsigned)(TP * ((TQ + TB - 1) / TB)), (unsigned)((s.C + CB - 1) / CB), (unsigned)nb);
  if (s.dtype == DT_F32)
    hipLaunchKernelGGL(wino_input_kernel<float>, grid, dim3(256), 0, stream, (const float*)x, (float*)V,
                       (int)s.C, (int)s.H, (int)s.W, s.ph, s.pw, TP, TQ, n0, Tc);
  else
    hipLaunchKernelGGL(wino_input_kernel<bf16_t>, grid, dim3(256), 0, stream, (const bf16_t*)x, (bf16_t*)V,
                       (int)s.C, (int)s.H, (int)s.W, s.ph, s.pw, TP, TQ, n0, Tc);
  return hipGetLastError();
}

hipError_t launch_wino_output(const Shape& s, const float* M, const void* b, void* y, int64_t n0, int64_t nb,
                              hipStream_t stream) {
  const int TP = (int)((s.P + 1) / 2), TQ = (int)((s.Q + 1) / 2);
  const int64_t Tc = nb * TP * TQ;
  const int64_t total = s.K * Tc;
  const dim3 grid((unsigned)((total + 255) / 256));
  if (s.dtype == DT_F32)
    hipLaunchKernelGGL(wino_output_kernel<float>, grid, dim3(256), 0, stream, M, (const float*)b, (float*)y,
                       (int)s.K, (int)s.P, (int)s.Q, TP, TQ, n0, Tc, s.relu ? 1 : 0);
  else
    hipLaunchKernelGGL(wino_output_kernel<bf16_t>, grid, dim3(256), 0, stream, M, (const bf16_t*)b,
                       (bf16_t*)y, (int)s.K, (int)s.P, (int)s.Q, TP, TQ, n0, Tc, s.relu ? 1 : 0);
  return hipGetLastError();
}

}  // namespace convsel
