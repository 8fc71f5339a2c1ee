// Direct convolution (paper, Sec. II-B item (d)): every output is the sum of
// filter taps times input pixels, with no transformed copy of the data.
// Arithmetic is fp32 FMA on the vector ALUs; bf16 inputs are widened when
// staged.
//
//  * direct_tile_kernel: a workgroup owns 32 output channels of one group and
//    an 8 x 32 block of output pixels of one image.  Per chunk of input
//    channels it stages the input halo (rows and columns the block reads,
//    zero-filled outside the image) and the chunk's filter taps in LDS, then
//    each thread accumulates 8 channels x 4 pixels in registers.  Pixels of a
//    thread are 8 columns apart so that a wave's LDS reads of one tap touch 8
//    consecutive columns (no bank conflicts) and its stores are coalesced.
//  * direct_depthwise_kernel: one input channel per group (Cg == 1, e.g.
//    depthwise layers).  A workgroup owns one image's rows of several output
//    planes, stages the input rows once, and sums the R*S taps per output.
//    These layers are bound by HBM traffic, not arithmetic.
//  * direct_dw3_kernel<T, S>: depthwise 3x3 (one input channel per output
//    channel), stride S = 1 or 2, dilation 1, padding 0 or 1, the shape of
//    MobileNet-style networks.  Bound by HBM traffic: a workgroup stages a
//    band of input rows of one or several whole planes in LDS with 16-byte
//    loads (the rows a band reads are contiguous in NCHW), then each thread
//    computes strips of 4 consecutive outputs of a row from LDS and stores
//    them as one vector.  Planes are independent, so the grid is
//    (row bands) x (groups of planes) with no halo exchange.
//  * direct_naive_kernel: one thread per output reading global memory, used
//    only when a halo tile would not fit in LDS (very large dilated filters).
#include <string>

#include "common.hpp"
#include "igemm_common.hpp"
#include "kernels.hpp"

namespace convsel {

namespace {

struct DirectArgs {
  const void* x;
  const void* w;
  const void* b;
  void* y;
  int N, C, H, W, K, R, S, P, Q;
  int sh, sw, ph, pw, dh, dw;
  int Cg, Kg, relu;
  int CC, HT, WT, XS; // tile kernel: channel chunk, halo extent, halo floats (x4)
  int TPo, PB;        // depthwise kernel: rows per tile, planes per block
};

constexpr int KT = 32, TP = 8, TQ = 32;

template <typename T>
__global__ __launch_bounds__(256) void direct_tile_kernel(DirectArgs a) {
  extern __shared__ __align__(16) float smem[];
  const int RS = a.R * a.S;
  float* xs = smem;                              // [CC][HT][WT]
  float* ws = smem + a.XS;                       // [CC][RS][KT], 16-byte aligned

  const int tid = threadIdx.x;
  const int tilesQ = (a.Q + TQ - 1) / TQ;
  const int p0 = (blockIdx.x / tilesQ) * TP, q0 = (blockIdx.x % tilesQ) * TQ;
  const int ktiles = (a.Kg + KT - 1) / KT;
  const int g = blockIdx.y / ktiles, kbase = (blockIdx.y % ktiles) * KT;
  const int n = blockIdx.z;
  const int kb = tid >> 6, lane = tid & 63;
  const int pl = lane >> 3, qb = lane & 7;

  const T* x = reinterpret_cast<const T*>(a.x) + (static_cast<int64_t>(n) * a.C + g * a.Cg) * a.H * a.W;
  const T* w = reinterpret_cast<const T*>(a.w) + static_cast<int64_t>(g * a.Kg + kbase) * a.Cg * RS;

  float acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[i][t] = 0.f;

  const int ih0 = p0 * a.sh - a.ph, iw0 = q0 * a.sw - a.pw;
  for (int c0 = 0; c0 < a.Cg; c0 += a.CC) {
    const int cc = min(a.CC, a.Cg - c0);
    const int nx = cc * a.HT * a.WT;
    for (int i = tid; i < nx; i += 256) {
      const int c = i / (a.HT * a.WT), rem = i - c * a.HT * a.WT;
      const int hh = rem / a.WT, ww = rem - hh * a.WT;
      const int ih = ih0 + hh, iw = iw0 + ww;
      float v = 0.f;
      if (ih >= 0 && ih < a.H && iw >= 0 && iw < a.W)
        v = elem<T>::load(x + (static_cast<int64_t>(c0 + c) * a.H + ih) * a.W + iw);
      xs[i] = v;
    }
    const int nw = KT * cc * RS;
    for (int i = tid; i < nw; i += 256) {
      const int kk = i / (cc * RS), rem = i - kk * cc * RS;  // rem = c*RS + rs
      float v = 0.f;
      if (kbase + kk < a.Kg) v = elem<T>::load(w + static_cast<int64_t>(kk) * a.Cg * RS + c0 * RS + rem);
      ws[rem * KT + kk] = v;
    }
    __syncthreads();
    for (int c = 0; c < cc; ++c) {
      for (int r = 0; r < a.R; ++r) {
        const float* xrow = xs + (c * a.HT + pl * a.sh + r * a.dh) * a.WT;
        for (int s = 0; s < a.S; ++s) {
          const float4* wp = reinterpret_cast<const float4*>(ws + ((c * a.R + r) * a.S + s) * KT + kb * 8);
          const float4 w0 = wp[0], w1 = wp[1];
          const float wv[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
          float xv[4];
#pragma unroll
          for (int t = 0; t < 4; ++t) xv[t] = xrow[(qb + 8 * t) * a.sw + s * a.dw];
#pragma unroll
          for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int t = 0; t < 4; ++t) acc[i][t] = fmaf(xv[t], wv[i], acc[i][t]);
        }
      }
    }
    __syncthreads();
  }

  const int p = p0 + pl;
  if (p >= a.P) return;
  T* y = reinterpret_cast<T*>(a.y);
  const T* bias = reinterpret_cast<const T*>(a.b);
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int kg = kbase + kb * 8 + i;
    if (kg >= a.Kg) continue;
    const int k = g * a.Kg + kg;
    const float bv = bias ? elem<T>::load(bias + k) : 0.f;
    T* yrow = y + ((static_cast<int64_t>(n) * a.K + k) * a.P + p) * a.Q;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int q = q0 + qb + 8 * t;
      if (q >= a.Q) continue;
      float v = acc[i][t] + bv;
      if (a.relu) v = fmaxf(v, 0.f);
      elem<T>::store(yrow + q, v);
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void direct_depthwise_kernel(DirectArgs a) {
  extern __shared__ __align__(16) float smem[];
  const int RS = a.R * a.S;
  const int HT = a.HT, WT = a.WT;
  float* xs = smem;                    // [PB][HT][WT]
  float* ws = smem + a.PB * HT * WT;   // [PB][RS]
  const int p0 = blockIdx.x * a.TPo;
  const int k0 = blockIdx.y * a.PB;
  const int n = blockIdx.z;
  const int pb_n = min(a.PB, a.K - k0);
  const int rows = min(a.TPo, a.P - p0);
  const int ih0 = p0 * a.sh - a.ph, iw0 = -a.pw;
  const T* x = reinterpret_cast<const T*>(a.x);
  const T* w = reinterpret_cast<const T*>(a.w);

  const int nx = pb_n * HT * WT;
  for (int i = threadIdx.x; i < nx; i += 256) {
    const int pb = i / (HT * WT), rem = i - pb * HT * WT;
    const int hh = rem / WT, ww = rem - hh * WT;
    const int ih = ih0 + hh, iw = iw0 + ww;
    const int cin = (k0 + pb) / a.Kg;  // Cg == 1: group index = input channel
    float v = 0.f;
    if (ih >= 0 && ih < a.H && iw >= 0 && iw < a.W)
      v = elem<T>::load(x + ((static_cast<int64_t>(n) * a.C + cin) * a.H + ih) * a.W + iw);
    xs[i] = v;
  }
  for (int i = threadIdx.x; i < pb_n * RS; i += 256) ws[i] = elem<T>::load(w + static_cast<int64_t>(k0) * RS + i);
  __syncthreads();

  const T* bias = reinterpret_cast<const T*>(a.b);
  T* y = reinterpret_cast<T*>(a.y);
  const int no = pb_n * rows * a.Q;
  for (int i = threadIdx.x; i < no; i += 256) {
    const int pb = i / (rows * a.Q), rem = i - pb * rows * a.Q;
    const int pl = rem / a.Q, q = rem - pl * a.Q;
    const float* xp = xs + (pb * HT + pl * a.sh) * WT + q * a.sw;
    const float* wp = ws + pb * RS;
    float acc = 0.f;
    for (int r = 0; r < a.R; ++r)
      for (int s = 0; s < a.S; ++s) acc = fmaf(xp[r * a.dh * WT + s * a.dw], wp[r * a.S + s], acc);
    const int k = k0 + pb;
    if (bias) acc += elem<T>::load(bias + k);
    if (a.relu) acc = fmaxf(acc, 0.f);
    elem<T>::store(y + ((static_cast<int64_t>(n) * a.K + k) * a.P + p0 + pl) * a.Q + q, acc);
  }
}

constexpr int kDwLoads = 4;  // chunk loads in flight per thread (depthwise staging)

struct Dw3Args {
  const void* x;
  const void* w;
  const void* b;
  void* y;
  uint32_t x_bytes;
  int NC, C, H, W, P, Q, ph, pw, relu;
  int TB, PB;        // output rows per band, planes per workgroup
  int HB, LP;        // staged rows per plane (for a full band), LDS floats per staged row
};

// LDS: [PB planes][HB rows][LP floats] of input, input column x at x + 4
// (LP a multiple of 4, so that a row's 16-byte-aligned chunks stay aligned;
// columns 0-3 and those past W + 3 stay zero, as do rows outside the image),
// then the PB planes' 9 taps.
constexpr int kDwCol0 = 4;

template <typename T, int S>
__global__ __launch_bounds__(256) void direct_dw3_kernel(Dw3Args a) {
  extern __shared__ __align__(16) float smem[];
  constexpr int VE = elem<T>::per16;  // elements per 16-byte load
  const int p0 = blockIdx.x * a.TB;
  const int tb = min(a.TB, a.P - p0);
  const int plane0 = blockIdx.y * a.PB;
  const int pb = min(a.PB, a.NC - plane0);
  const int ih0 = p0 * S - a.ph;
  const int hb = (tb - 1) * S + 3;  // rows this band reads
  const int per_plane = a.HB * a.LP;
  float* ws = smem + a.PB * per_plane;
  const int tid = threadIdx.x;

  for (int i = tid; i < pb * per_plane / 4; i += 256)
    reinterpret_cast<float4*>(smem)[i] = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int i = tid; i < pb * 9; i += 256) {
    const int c = (plane0 + i / 9) % a.C;
    ws[i] = elem<T>::load(reinterpret_cast<const T*>(a.w) + c * 9 + i % 9);
  }
  __syncthreads();

  // The rows of the band inside the image are one contiguous span per
  // plane, read in aligned 16-byte chunks (a chunk at either end may hold
  // elements of the neighbouring rows or planes, which are not written;
  // reads past the tensor return zeros through the buffer range).  All the
  // block's planes' chunks form one loop (at most cmax per plane), and a
  // thread issues kDwLoads loads before it consumes any.  When W is a
  // multiple of the chunk, every chunk lies inside one row and lands as
  // 16-byte LDS writes.
  const int rlo = max(ih0, 0), rhi = min(ih0 + hb, a.H);
  if (rhi > rlo) {
    const __amdgpu_buffer_rsrc_t xr = igemm::make_rsrc(a.x, a.x_bytes);
    const int span = (rhi - rlo) * a.W;
    const int cmax = (span + 2 * VE - 2) / VE;
    const int total = pb * cmax;
    const bool rowwise = a.W % VE == 0;
    for (int base = 0; base < total; base += 256 * kDwLoads) {
      igemm::u32x4_t v[kDwLoads];
      int64_t c0s[kDwLoads];
#pragma unroll
      for (int k = 0; k < kDwLoads; ++k) {
        const int idx = base + k * 256 + tid;
        const int pi = idx / cmax, t = idx - pi * cmax;
        const int64_t g0 = (static_cast<int64_t>(plane0 + pi) * a.H + rlo) * a.W;
        c0s[k] = (g0 & ~static_cast<int64_t>(VE - 1)) + static_cast<int64_t>(t) * VE;
        // chunks past the block's planes read past the buffer (zeros, unused)
        const uint32_t off = idx < total ? static_cast<uint32_t>(c0s[k] * sizeof(T)) : a.x_bytes;
        v[k] = __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0);
      }
#pragma unroll
      for (int k = 0; k < kDwLoads; ++k) {
        const int idx = base + k * 256 + tid;
        if (idx >= total) continue;
        const int pi = idx / cmax;
        const int64_t g0 = (static_cast<int64_t>(plane0 + pi) * a.H + rlo) * a.W;
        const int rel = static_cast<int>(c0s[k] - g0);  // span element at the chunk's first lane element
        if (rel >= span) continue;
        float* dst = smem + pi * per_plane + (rlo - ih0) * a.LP + kDwCol0;
        float f[VE];
#pragma unroll
        for (int e = 0; e < VE; ++e) {
          if constexpr (sizeof(T) == 4) f[e] = __uint_as_float(v[k][e]);
          else f[e] = __uint_as_float((v[k][e >> 1] >> (16 * (e & 1))) << 16);
        }
        if (rowwise) {
          const int row = rel / a.W, col = rel - row * a.W;
#pragma unroll
          for (int e = 0; e < VE; e += 4)
            *reinterpret_cast<float4*>(dst + row * a.LP + col + e) = make_float4(f[e], f[e + 1], f[e + 2], f[e + 3]);
        } else {
          int row = rel >= 0 ? rel / a.W : -1;
          int col = rel - row * a.W;
#pragma unroll
          for (int e = 0; e < VE; ++e) {
            if (rel + e >= 0 && rel + e < span) dst[row * a.LP + col] = f[e];
            if (++col == a.W) {
              col = 0;
              ++row;
            }
          }
        }
      }
    }
  }
  __syncthreads();

  // Work items: 4 output rows (a vertical strip) of one column; consecutive
  // threads take consecutive columns, so that LDS reads and global stores
  // of a wave are contiguous.  A strip reads 4 S + 2 rows of 3 columns.
  constexpr int NR = 3 * S + 3;
  const int rg = (tb + 3) / 4;
  const int items = pb * rg * a.Q;
  const T* bias = reinterpret_cast<const T*>(a.b);
  T* y = reinterpret_cast<T*>(a.y);
  for (int it = tid; it < items; it += 256) {
    const int pi = it / (rg * a.Q), rem = it - pi * rg * a.Q;
    const int g = rem / a.Q, q = rem - g * a.Q;
    const int pl0 = 4 * g;
    const float* wp = ws + pi * 9;
    const float* xp = smem + pi * per_plane + (pl0 * S) * a.LP + q * S + kDwCol0 - a.pw;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < NR; ++j) {
      const float v0 = xp[j * a.LP], v1 = xp[j * a.LP + 1], v2 = xp[j * a.LP + 2];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int r = j - t * S;  // tap row of output row pl0 + t
        if (r >= 0 && r < 3) acc[t] = fmaf(v0, wp[r * 3], fmaf(v1, wp[r * 3 + 1], fmaf(v2, wp[r * 3 + 2], acc[t])));
      }
    }
    const int plane = plane0 + pi;
    const float bv = bias ? elem<T>::load(bias + plane % a.C) : 0.f;
    T* yp = y + (static_cast<int64_t>(plane) * a.P + p0 + pl0) * a.Q + q;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      if (pl0 + t < tb) {
        float o = acc[t] + bv;
        if (a.relu) o = fmaxf(o, 0.f);
        elem<T>::store(yp + t * a.Q, o);
      }
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void direct_naive_kernel(DirectArgs a, int64_t total) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= total) return;
  const int q = static_cast<int>(idx % a.Q);
  const int p = static_cast<int>((idx / a.Q) % a.P);
  const int k = static_cast<int>((idx / (static_cast<int64_t>(a.Q) * a.P)) % a.K);
  const int n = static_cast<int>(idx / (static_cast<int64_t>(a.Q) * a.P * a.K));
  const int g = k / a.Kg;
  const T* x = reinterpret_cast<const T*>(a.x);
  const T* w = reinterpret_cast<const T*>(a.w) + static_cast<int64_t>(k) * a.Cg * a.R * a.S;
  float acc = 0.f;
  for (int c = 0; c < a.Cg; ++c) {
    const T* plane = x + (static_cast<int64_t>(n) * a.C + g * a.Cg + c) * a.H * a.W;
    for (int r = 0; r < a.R; ++r) {
      const int ih = p * a.sh - a.ph + r * a.dh;
      if (ih < 0 || ih >= a.H) continue;
      for (int s = 0; s < a.S; ++s) {
        const int iw = q * a.sw - a.pw + s * a.dw;
        if (iw < 0 || iw >= a.W) continue;
        acc = fmaf(elem<T>::load(plane + ih * a.W + iw), elem<T>::load(w + (c * a.R + r) * a.S + s), acc);
      }
    }
  }
  const T* bias = reinterpret_cast<const T*>(a.b);
  if (bias) acc += elem<T>::load(bias + k);
  if (a.relu) acc = fmaxf(acc, 0.f);
  elem<T>::store(reinterpret_cast<T*>(a.y) + idx, acc);
}

constexpr int kLdsBudget = 64 * 1024;

// Plan of the depthwise 3x3 kernel: bands of TB output rows of PB planes,
// within 32 KiB of LDS (several workgroups per CU overlap one's loads with
// another's arithmetic).
bool dw3_plan(const Shape& s, Dw3Args& a) {
  if (s.Cg != 1 || s.Kg != 1 || s.R != 3 || s.S != 3 || s.dh != 1 || s.dw != 1) return false;
  if (s.sh != s.sw || (s.sh != 1 && s.sh != 2) || s.ph > 1 || s.pw > 1) return false;
  const int64_t x_bytes = s.N * s.C * s.H * s.W * s.esize();
  if (x_bytes + 16 >= ((int64_t)1 << 31) || s.N * s.C >= ((int64_t)1 << 31)) return false;
  a.NC = (int)(s.N * s.C); a.C = (int)s.C; a.H = (int)s.H; a.W = (int)s.W;
  a.P = (int)s.P; a.Q = (int)s.Q; a.ph = s.ph; a.pw = s.pw; a.relu = s.relu ? 1 : 0;
  a.x_bytes = (uint32_t)x_bytes;
  a.LP = ((int)s.W + kDwCol0 + 1 + 3) & ~3;
  // About 4096 outputs per workgroup on planes of at least 512 outputs,
  // 2048 on smaller ones (measured on the MobileNetV2 layers: larger bands
  // amortise the staging on big planes, smaller groups keep more
  // workgroups on small ones).
  const int PQ = (int)(s.P * s.Q);
  const int target = PQ >= 512 ? 4096 : 2048;
  if (PQ >= target) {
    a.PB = 1;
    a.TB = target / (int)s.Q > 1 ? target / (int)s.Q : 1;
    if (a.TB > s.P) a.TB = (int)s.P;
  } else {
    a.TB = (int)s.P;
    a.PB = target / PQ > 1 ? target / PQ : 1;
  }
  // Rows staged per plane: those of a band rounded up to whole 4-row strips
  // (the rows past the band stay zero; the last strip reads them).
  auto rows = [&](int tb) { return (((tb + 3) / 4) * 4 - 1) * s.sh + 3; };
  auto lds = [&](int tb, int pb) { return (size_t)pb * ((size_t)rows(tb) * a.LP + 9) * 4; };
  while (a.PB > 1 && lds(a.TB, a.PB) > 32 * 1024) a.PB = (a.PB + 1) / 2;
  while (a.TB > 1 && lds(a.TB, a.PB) > 32 * 1024) a.TB = (a.TB + 1) / 2;
  if (lds(a.TB, a.PB) > 32 * 1024) return false;
  a.HB = rows(a.TB);
  return true;
}

template <typename T>
hipError_t launch_direct_typed(const Shape& s, const void* x, const void* w, const void* b, void* y,
                               hipStream_t stream) {
  DirectArgs a;
  a.x = x; a.w = w; a.b = b; a.y = y;
  a.N = (int)s.N; a.C = (int)s.C; a.H = (int)s.H; a.W = (int)s.W; a.K = (int)s.K;
  a.R = (int)s.R; a.S = (int)s.S; a.P = (int)s.P; a.Q = (int)s.Q;
  a.sh = s.sh; a.sw = s.sw; a.ph = s.ph; a.pw = s.pw; a.dh = s.dh; a.dw = s.dw;
  a.Cg = (int)s.Cg; a.Kg = (int)s.Kg; a.relu = s.relu ? 1 : 0;
  a.CC = a.HT = a.WT = a.XS = a.TPo = a.PB = 0;
  const int RS = a.R * a.S;

  Dw3Args d3;
  if (dw3_plan(s, d3)) {
    d3.x = x; d3.w = w; d3.b = b; d3.y = y;
    const dim3 grid((unsigned)((d3.P + d3.TB - 1) / d3.TB), (unsigned)((d3.NC + d3.PB - 1) / d3.PB));
    const size_t lds = (size_t)d3.PB * ((size_t)d3.HB * d3.LP + 9) * 4;
    if (s.sh == 1)
      hipLaunchKernelGGL((direct_dw3_kernel<T, 1>), grid, dim3(256), lds, stream, d3);
    else
      hipLaunchKernelGGL((direct_dw3_kernel<T, 2>), grid, dim3(256), lds, stream, d3);
    return hipGetLastError();
  }
  if (a.Cg == 1) {
    // Depthwise-style: one input channel per group.
    const int WT = (a.Q - 1) * a.sw + (a.S - 1) * a.dw + 1;
    int tpo = 2048 / a.Q > 1 ? 2048 / a.Q : 1;
    if (tpo > a.P) tpo = a.P;
    int pb = 2048 / (tpo * a.Q);
    if (pb < 1) pb = 1;
    if (pb > a.K) pb = a.K;
    auto lds = [&](int t, int p) {
      return (size_t)p * (((size_t)(t - 1) * a.sh + (size_t)(a.R - 1) * a.dh + 1) * WT + RS) * 4;
    };
    while (pb > 1 && lds(tpo, pb) > kLdsBudget) pb = (pb + 1) / 2;
    while (tpo > 1 && lds(tpo, pb) > kLdsBudget) tpo = (tpo + 1) / 2;
    if (lds(tpo, pb) <= kLdsBudget) {
      a.TPo = tpo;
      a.PB = pb;
      a.HT = (tpo - 1) * a.sh + (a.R - 1) * a.dh + 1;
      a.WT = WT;
      const dim3 grid((a.P + tpo - 1) / tpo, (a.K + pb - 1) / pb, a.N);
      hipLaunchKernelGGL(direct_depthwise_kernel<T>, grid, dim3(256), lds(tpo, pb), stream, a);
      return hipGetLastError();
    }
  } else {
    const int HT = (TP - 1) * a.sh + (a.R - 1) * a.dh + 1;
    const int WT = (TQ - 1) * a.sw + (a.S - 1) * a.dw + 1;
    const size_t per_c = ((size_t)HT * WT + (size_t)RS * KT) * 4;
    if (per_c + 16 <= (size_t)kLdsBudget) {
      int cc = (int)((kLdsBudget - 16) / per_c);
      if (cc > a.Cg) cc = a.Cg;
      if (cc > 16) cc = 16;
      a.CC = cc;
      a.HT = HT;
      a.WT = WT;
      a.XS = (cc * HT * WT + 3) & ~3;
      const size_t lds = ((size_t)a.XS + (size_t)cc * RS * KT) * 4;
      const int tiles = ((a.P + TP - 1) / TP) * ((a.Q + TQ - 1) / TQ);
      const dim3 grid(tiles, s.G * ((a.Kg + KT - 1) / KT), a.N);
      hipLaunchKernelGGL(direct_tile_kernel<T>, grid, dim3(256), lds, stream, a);
      return hipGetLastError();
    }
  }
  const int64_t total = s.N * s.K * s.P * s.Q;
  const int64_t blocks = (total + 255) / 256;
  hipLaunchKernelGGL(direct_naive_kernel<T>, dim3((unsigned)blocks), dim3(256), 0, stream, a, total);
  return hipGetLastError();
}

}  // namespace

std::string direct_describe(const Shape& s) {
  Dw3Args d3;
  if (dw3_plan(s, d3)) {
    char buf[256];
    snprintf(buf, sizeof(buf), "direct kernels=direct_dw3_kernel<%s,%d> rows_per_band=%d planes_per_block=%d",
             s.dtype == DT_F32 ? "f32" : "bf16", s.sh, d3.TB, d3.PB);
    return buf;
  }
  return s.Cg == 1 ? "direct kernels=direct_depthwise_kernel" : "direct kernels=direct_tile_kernel";
}

hipError_t launch_direct(const Shape& s, const void* x, const void* w, const void* b, void* y,
                         hipStream_t stream) {
  if (s.dtype == DT_F32) return launch_direct_typed<float>(s, x, w, b, y, stream);
  return launch_direct_typed<bf16_t>(s, x, w, b, y, stream);
}

}  // namespace convsel
