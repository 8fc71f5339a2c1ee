// Implicit GEMM (paper, Sec. V-B item (b)): the convolution as the product
//   Y[k][pixel] = sum_{(c,r,s)} Wt[k][(c,r,s)] * X[(c,r,s)][pixel]
// without ever forming the column matrix X.  On MFMA: D (output channels x
// pixels) accumulates 32 x 32 blocks in fp32.
//
// Pixels are the flattened (n, p, q) output positions; a workgroup owns BN =
// 128 consecutive pixels and BM (64 or 128) output channels of one group.  The
// reduction is walked in chunks of Cc input channels; for each chunk:
//
//  * Input halo.  The input is viewed as a stack of zero-padded images in
//    "virtual rows": pixel (n, p) with filter row r reads virtual row
//    n*Hv + p*sh + r*dh, Hv = (P-1)*sh + (R-1)*dh + 1, and virtual column
//    q*sw + s*dw (real row = virtual row mod Hv - pad_h, real column =
//    virtual column - pad_w).  The workgroup's pixels read one contiguous
//    range of VR virtual rows, each Wv columns wide.  That range is staged
//    once per chunk in LDS with the channels innermost:
//        Xs[(vrow * Wv + vcol) * PS + cg]   (16-byte units of UE channels)
//    so every filter tap of every pixel is a 16-byte LDS read, and each input
//    element is fetched from global memory once per chunk instead of R*S
//    times.  Global reads of the halo are coalesced along the image row.
//  * Filters.  The chunk's taps of the BM filters are staged as
//        As[i * UR + (tap * NG + cg)]       (16-byte units)
//    i.e. transposed from (c, r, s) to (tap, c) order so that a 16-byte unit
//    holds UE consecutive channels of one tap, matching the input units.
//  * MFMA.  One reduction step consumes two 16-byte units per lane (the two
//    halves of the wave take units 2*step and 2*step+1), i.e. 16 bf16 or 8
//    fp32 reduction terms; a unit table in LDS maps each unit to its LDS
//    offset in Xs.  A padding unit (odd unit count) has zero filter values.
//
// Row strides in LDS (UR and PS units of 16 bytes) are odd, so the 16-byte
// reads of 32 consecutive rows / pixels map to distinct bank groups.
#include "common.hpp"
#include "kernels.hpp"

namespace convsel {

namespace {

constexpr int kThreads = 256;
constexpr int BN = 128;

struct IgArgs {
  const void* x;
  const void* w;
  const void* b;
  void* y;
  int N, C, H, W, K, R, S, P, Q;
  int sh, sw, ph, pw, dh, dw;
  int Cg, Kg, relu;
  int Hv, Wv, VR;     // virtual rows per image, halo width, halo rows
  int NPQ;
  int units;          // R*S*NG
  int steps;          // ceil(units / 2)
  int UR;             // filter row stride in 16-byte units (odd)
  int PS;             // halo pixel stride in 16-byte units (odd)
  int ktiles;         // ceil(Kg / BM)
  int xs_units;       // VR * Wv * PS
};

// Virtual row of the first filter row for pixel j.
__device__ __forceinline__ int vrow_of(int j, const IgArgs& a) {
  const int PQ = a.P * a.Q;
  const int n = j / PQ, pq = j - n * PQ;
  return n * a.Hv + (pq / a.Q) * a.sh;
}

template <typename T, int BM, int NG, int RST>
__global__ __launch_bounds__(kThreads) void implicit_gemm_kernel(IgArgs a) {
  constexpr int UE = elem<T>::per16;
  constexpr int Cc = UE * NG;
  constexpr int MI = BM / 64, NJ = BN / 64;
  extern __shared__ __align__(16) vec16 smem[];
  vec16* As = smem;                         // [BM][UR]
  vec16* Xs = smem + BM * a.UR;             // [VR*Wv][PS]
  int* utab = reinterpret_cast<int*>(Xs + a.xs_units);  // [2*steps]: Xs unit offset per unit

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int half = lane >> 5, l32 = lane & 31;
  const int j0 = blockIdx.x * BN;
  const int g = blockIdx.y / a.ktiles;
  const int k0 = (blockIdx.y - g * a.ktiles) * BM;
  const int RS = a.R * a.S;
  const int jl = min(j0 + BN, a.NPQ) - 1;
  const int vr_lo = vrow_of(j0, a);

  // Unit table: unit u = tap*NG + cg -> Xs offset (tap offset * PS + cg).
  for (int u = tid; u < 2 * a.steps; u += kThreads) {
    int off = 0;
    if (u < a.units) {
      const int tap = u / NG, cg = u - tap * NG;
      const int r = tap / a.S, s = tap - r * a.S;
      off = (r * a.dh * a.Wv + s * a.dw) * a.PS + cg;
    }
    utab[u] = off;
  }

  // Per-lane pixel offsets into the halo and output base offsets.
  int pofs[NJ];
  int64_t ybase[NJ];
  bool jvalid[NJ];
  {
    const int PQ = a.P * a.Q;
#pragma unroll
    for (int nj = 0; nj < NJ; ++nj) {
      const int j = j0 + wn * (BN / 2) + nj * 32 + l32;
      jvalid[nj] = j < a.NPQ;
      const int jj = jvalid[nj] ? j : jl;
      const int n = jj / PQ, pq = jj - n * PQ;
      const int q = pq - (pq / a.Q) * a.Q;
      pofs[nj] = ((vrow_of(jj, a) - vr_lo) * a.Wv + q * a.sw) * a.PS;
      ybase[nj] = static_cast<int64_t>(n) * a.K * PQ + pq;
    }
  }

  const T* x = reinterpret_cast<const T*>(a.x);
  const T* w = reinterpret_cast<const T*>(a.w) + static_cast<int64_t>(g * a.Kg + k0) * a.Cg * RS;
  const int64_t HW = static_cast<int64_t>(a.H) * a.W;

  f32x16_t acc[MI][NJ];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int nj = 0; nj < NJ; ++nj) acc[mi][nj] = zero16();

  const int halo_items = a.VR * a.Wv * NG;
  for (int c0 = 0; c0 < a.Cg; c0 += Cc) {
    // ---- stage the input halo: item = (vrow, vcol, cg) -> UE channels ----
    for (int it = tid; it < halo_items; it += kThreads) {
      const int vc = it % a.Wv;
      const int rest = it / a.Wv;
      const int vr = rest % a.VR, cg = rest / a.VR;
      const int v = vr_lo + vr;
      const int n = v / a.Hv;
      const int ih = v - n * a.Hv - a.ph, iw = vc - a.pw;
      vec16 u = vec16_zero();
      if (n < a.N && ih >= 0 && ih < a.H && iw >= 0 && iw < a.W) {
        const int cbase = c0 + cg * UE;
        const T* src = x + (static_cast<int64_t>(n) * a.C + g * a.Cg + cbase) * HW + ih * a.W + iw;
#pragma unroll
        for (int e = 0; e < UE; ++e)
          if (cbase + e < a.Cg) vec16_set<T>(u, e, src[e * HW]);
      }
      Xs[(vr * a.Wv + vc) * a.PS + cg] = u;
    }
    // ---- stage the filters: item = (row i, cg) -> R*S units ----
    for (int it = tid; it < BM * NG; it += kThreads) {
      const int i = it / NG, cg = it - i * NG;
      const int cbase = c0 + cg * UE;
      const bool row_ok = k0 + i < a.Kg;
      const T* src = w + static_cast<int64_t>(i) * a.Cg * RS + static_cast<int64_t>(cbase) * RS;
      if constexpr (RST > 0) {
        // UE whole channels of RST taps are RST contiguous 16-byte units.
        vec16 raw[RST > 0 ? RST : 1];
#pragma unroll
        for (int m = 0; m < RST; ++m) raw[m] = (row_ok && cbase < a.Cg) ? load16(src + m * UE) : vec16_zero();
#pragma unroll
        for (int tap = 0; tap < RST; ++tap) {
          vec16 u = vec16_zero();
#pragma unroll
          for (int e = 0; e < UE; ++e) {
            const int f = e * RST + tap;  // flat (channel, tap) index in the loaded run
            vec16_set<T>(u, e, vec16_get<T>(raw[f / UE], f % UE));
          }
          As[i * a.UR + tap * NG + cg] = u;
        }
      } else {
        for (int tap = 0; tap < RS; ++tap) {
          vec16 u = vec16_zero();
          if (row_ok) {
#pragma unroll
            for (int e = 0; e < UE; ++e)
              if (cbase + e < a.Cg) vec16_set<T>(u, e, src[e * RS + tap]);
          }
          As[i * a.UR + tap * NG + cg] = u;
        }
      }
    }
    // zero the padding unit of an odd unit count
    if (a.units & 1)
      for (int i = tid; i < BM; i += kThreads) As[i * a.UR + a.units] = vec16_zero();
    __syncthreads();

    // ---- MFMA over the chunk's reduction steps ----
    for (int st = 0; st < a.steps; ++st) {
      const int u = 2 * st + half;
      const int xo = utab[u];
      vec16 af[MI], bfr[NJ];
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) af[mi] = As[(wm * (BM / 2) + mi * 32 + l32) * a.UR + u];
#pragma unroll
      for (int nj = 0; nj < NJ; ++nj) bfr[nj] = Xs[pofs[nj] + xo];
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int nj = 0; nj < NJ; ++nj) mfma_32x32<T>(acc[mi][nj], af[mi], bfr[nj]);
    }
    __syncthreads();
  }

  // ---- epilogue: bias, ReLU, NCHW store ----
  const T* bias = reinterpret_cast<const T*>(a.b);
  T* y = reinterpret_cast<T*>(a.y);
  const int64_t PQ = static_cast<int64_t>(a.P) * a.Q;
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int i = k0 + wm * (BM / 2) + mi * 32 + mfma_row(v, lane);
      if (i >= a.Kg) continue;
      const int k = g * a.Kg + i;
      const float bv = bias ? elem<T>::load(bias + k) : 0.f;
#pragma unroll
      for (int nj = 0; nj < NJ; ++nj) {
        if (!jvalid[nj]) continue;
        float val = acc[mi][nj][v] + bv;
        if (a.relu) val = fmaxf(val, 0.f);
        elem<T>::store(y + ybase[nj] + k * PQ, val);
      }
    }
  }
}

// Largest halo span (in virtual rows) over all pixel tiles.  The span of a
// tile depends only on where it starts within an image, which repeats every
// PQ / gcd(BN, PQ) tiles, so one period is scanned.
int halo_rows(const Shape& s, int Hv) {
  const int64_t PQ = s.P * s.Q, NPQ = s.N * PQ;
  const int64_t tiles = (NPQ + BN - 1) / BN;
  int64_t a = BN, b = PQ;
  while (b) {
    const int64_t t = a % b;
    a = b;
    b = t;
  }
  const int64_t period = PQ / a;
  const int64_t scan = tiles < period + 1 ? tiles : period + 1;
  auto vrow = [&](int64_t j) {
    const int64_t n = j / PQ, pq = j % PQ;
    return n * Hv + (pq / s.Q) * s.sh;
  };
  int64_t best = 0;
  for (int64_t t = 0; t < scan; ++t) {
    const int64_t j0 = t * BN;
    const int64_t j1 = (j0 + BN < NPQ ? j0 + BN : NPQ) - 1;
    const int64_t span = vrow(j1) - vrow(j0) + (s.R - 1) * s.dh + 1;
    if (span > best) best = span;
  }
  // The last, possibly partial, tile.
  {
    const int64_t j0 = (tiles - 1) * BN;
    const int64_t span = vrow(NPQ - 1) - vrow(j0) + (s.R - 1) * s.dh + 1;
    if (span > best) best = span;
  }
  return (int)best;
}

// Two workgroups per CU fit in 80 KiB each; larger halos use up to the
// 160 KiB a workgroup may hold.
constexpr size_t kLdsPreferred = 80 * 1024;
constexpr size_t kLdsLimit = 160 * 1024;

struct IgPlan {
  int BM, NG, RST;
  IgArgs a;
  size_t lds;
};

template <typename T>
bool make_plan(const Shape& s, const void* wptr, IgPlan& pl) {
  constexpr int UE = elem<T>::per16;
  IgArgs& a = pl.a;
  a.N = (int)s.N; a.C = (int)s.C; a.H = (int)s.H; a.W = (int)s.W; a.K = (int)s.K;
  a.R = (int)s.R; a.S = (int)s.S; a.P = (int)s.P; a.Q = (int)s.Q;
  a.sh = s.sh; a.sw = s.sw; a.ph = s.ph; a.pw = s.pw; a.dh = s.dh; a.dw = s.dw;
  a.Cg = (int)s.Cg; a.Kg = (int)s.Kg; a.relu = s.relu ? 1 : 0;
  a.Hv = (int)((s.P - 1) * s.sh + (s.R - 1) * s.dh + 1);
  a.Wv = (int)((s.Q - 1) * s.sw + (s.S - 1) * s.dw + 1);
  a.VR = halo_rows(s, a.Hv);
  a.NPQ = (int)(s.N * s.P * s.Q);
  const int RS = a.R * a.S;
  pl.BM = s.Kg <= 64 ? 64 : 128;
  a.ktiles = (a.Kg + pl.BM - 1) / pl.BM;
  const bool aligned = reinterpret_cast<uintptr_t>(wptr) % 16 == 0;
  const bool vec_w = aligned && s.Cg % UE == 0;
  pl.RST = 0;
  if (vec_w && RS == 1) pl.RST = 1;
  if (vec_w && RS == 9) pl.RST = 9;
  for (size_t limit : {kLdsPreferred, kLdsLimit}) {
    for (int ng = (s.Cg > UE ? 2 : 1); ng >= 1; --ng) {
      a.units = RS * ng;
      a.steps = (a.units + 1) / 2;
      a.UR = (2 * a.steps) | 1;
      a.PS = ng | 1;
      a.xs_units = a.VR * a.Wv * a.PS;
      const size_t lds = ((size_t)pl.BM * a.UR + (size_t)a.xs_units) * 16 + (size_t)2 * a.steps * 4;
      if (lds <= limit) {
        pl.NG = ng;
        pl.lds = lds;
        return true;
      }
    }
  }
  return false;
}

template <typename T, int BM, int NG, int RST>
hipError_t launch_one(const IgPlan& pl, hipStream_t stream) {
  const auto kern = implicit_gemm_kernel<T, BM, NG, RST>;
  if (pl.lds > 64 * 1024) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)pl.lds);
    if (e != hipSuccess) return e;
  }
  const dim3 grid((pl.a.NPQ + BN - 1) / BN, pl.a.ktiles * (pl.a.K / pl.a.Kg));
  hipLaunchKernelGGL(kern, grid, dim3(kThreads), pl.lds, stream, pl.a);
  return hipGetLastError();
}

template <typename T, int BM, int NG>
hipError_t launch_rst(const IgPlan& pl, hipStream_t stream) {
  switch (pl.RST) {
    case 1: return launch_one<T, BM, NG, 1>(pl, stream);
    case 9: return launch_one<T, BM, NG, 9>(pl, stream);
    default: return launch_one<T, BM, NG, 0>(pl, stream);
  }
}

template <typename T>
hipError_t launch_typed(const Shape& s, const void* x, const void* w, const void* b, void* y,
                        hipStream_t stream) {
  IgPlan pl;
  if (!make_plan<T>(s, w, pl)) return hipErrorInvalidValue;
  pl.a.x = x; pl.a.w = w; pl.a.b = b; pl.a.y = y;
  if (pl.BM == 64) return pl.NG == 2 ? launch_rst<T, 64, 2>(pl, stream) : launch_rst<T, 64, 1>(pl, stream);
  return pl.NG == 2 ? launch_rst<T, 128, 2>(pl, stream) : launch_rst<T, 128, 1>(pl, stream);
}

}  // namespace

bool implicit_gemm_fits(const Shape& s) {
  IgPlan pl;
  if (s.dtype == DT_F32) return make_plan<float>(s, nullptr, pl);
  return make_plan<bf16_t>(s, nullptr, pl);
}

hipError_t launch_implicit_gemm(const Shape& s, const void* x, const void* w, const void* b, void* y,
                                hipStream_t stream) {
  if (s.dtype == DT_F32) return launch_typed<float>(s, x, w, b, y, stream);
  return launch_typed<bf16_t>(s, x, w, b, y, stream);
}

}  // namespace convsel
