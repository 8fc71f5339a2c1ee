// Implicit precomputed-index GEMM (paper, Sec. V-B item (a)): the product
//   Y[k][pixel] = sum_{kk = (c, r, s)} W[k][kk] * X[kk][pixel]
// without a column matrix, like implicit GEMM, but every element of the
// X operand is gathered through two index tables built in a precomputation
// step and kept with the filters:
//
//  * reduction table, one entry per kk = (c*R + r)*S + s of a group:
//      delta = c*H*W + r*dh*W + s*dw  (element offset of tap (c, r, s)),
//      rs    = (r*dh) << 16 | (s*dw)  (its row and column displacement);
//    entries past C/G*R*S (the padding of the last reduction tile) carry a
//    row displacement of kOutside, which puts every pixel outside the image.
//  * pixel table, one entry per output pixel j = (n*P + p)*Q + q of a launch:
//      base = n*C*H*W + ih0*W + iw0  and  pos = ih0 << 16 | (iw0 & 0xffff),
//    with ih0 = p*sh - ph, iw0 = q*sw - pw (the top-left input of the window).
//
// Element (kk, j) of X is then x[g*C/G*H*W + base + delta] when
// 0 <= ih0 + rd < H and 0 <= iw0 + sd < W, and zero otherwise: two table
// reads, two adds and two unsigned compares, no division anywhere in the
// kernel.  Unlike the halo kernels this places no limit on the filter size,
// stride or dilation that the LDS could hold.
//
// Tiling: 4 waves in a 2 x 2 grid over a BM (64 or 128) x 128 tile of
// (output channels, pixels); reduction tiles of BK = 32 bf16 / 16 fp32 terms
// staged in LDS as rows of BK + 16 bytes (odd multiples of 16 bytes: the
// 16-byte fragment reads of 32 consecutive rows hit distinct bank groups).
// The next tile is gathered into registers while the MFMAs run on the
// current one.  The table entries of a reduction index are the same for a
// whole wave, so they are read with scalar loads.
#include <atomic>
#include <stdio.h>
#include <string>

#include "common.hpp"
#include "igemm_common.hpp"
#include "kernels.hpp"

namespace convsel {

namespace {

using namespace igemm;

constexpr int kOutside = 1 << 14;   // displacement that no in-image coordinate reaches
constexpr int kPcThreads = 256;

struct PcArgs {
  const void* x;        // first image of this launch
  const void* wp;       // packed filters [G][Kpad][KRp]
  const int2* ktab;     // [KRp]
  const int2* ptab;     // [NPQ]
  uint32_t x_bytes;     // extent of this launch's input
  uint32_t wp_bytes;
  int H, W, Cg, G;
  int KRp;              // reduction length padded to BK
  int Kpad, ktiles;
  int NPQ;
  int64_t group_stride; // elements between the input channels of two groups (Cg*H*W)
  EpiArgs e;
};

template <typename T, int BM>
__global__ __launch_bounds__(kPcThreads) void implicit_precomp_kernel(PcArgs a) {
  constexpr int UE = elem<T>::per16;
  constexpr int ES = elem<T>::bytes;
  constexpr int BK = 4 * UE;       // two MFMA steps
  constexpr int KP = BK + UE;      // padded LDS row, elements
  constexpr int UA = BM * 4 / kPcThreads;  // filter units per thread and tile
  constexpr int MI = BM / 64, NJ = BN / 64;
  constexpr size_t kTileBytes = (size_t)(BM + BN) * KP * ES;
  constexpr size_t kStageBytes = (size_t)4 * 32 * 64 * sizeof(float);  // epilogue staging, 8 KiB per wave
  constexpr size_t kSmem = kTileBytes > kStageBytes ? kTileBytes : kStageBytes;
  __shared__ __align__(16) char smem[kSmem];
  T* As = reinterpret_cast<T*>(smem);
  T* Bs = As + BM * KP;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int half = lane >> 5, l32 = lane & 31;
  const int j0 = blockIdx.x * BN;
  const int g = blockIdx.y / a.ktiles;
  const int k0 = (blockIdx.y - g * a.ktiles) * BM;

  const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, a.x_bytes);
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(a.wp, a.wp_bytes);
  const uint32_t xg = static_cast<uint32_t>(g * a.group_stride * ES);  // scalar offset of the group

  // This thread's pixel (column jl of the tile) and its two reduction units
  // (hv and hv + 2 of the four per tile; hv is the same for a whole wave).
  const int jl = tid & (BN - 1);
  const int hv = __builtin_amdgcn_readfirstlane(tid >> 7);
  const int j = j0 + jl;
  int base = 0, ih0 = kOutside, iw0 = 0;
  if (j < a.NPQ) {
    const int2 pt = a.ptab[j];
    base = pt.x;
    ih0 = pt.y >> 16;
    iw0 = static_cast<int16_t>(pt.y & 0xffff);
  }
  const unsigned H = a.H, W = a.W;

  // Filter units: unit id = tid + t*256 -> row id/4, reduction unit id%4.
  uint32_t wofs[UA];
#pragma unroll
  for (int t = 0; t < UA; ++t) {
    const int id = tid + t * kPcThreads;
    wofs[t] = static_cast<uint32_t>((static_cast<int64_t>(g * a.Kpad + k0 + id / 4) * a.KRp + (id % 4) * UE) * ES);
  }

  vec16 ra[UA], rb[2];
  auto fetch = [&](int kt) {
    const int kb = kt * BK;
#pragma unroll
    for (int t = 0; t < UA; ++t) ra[t] = buf_load16(wr, wofs[t], static_cast<uint32_t>(kb * ES));
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int kk0 = kb + (hv + 2 * u) * UE;  // wave-uniform
      uint32_t e[UE];
#pragma unroll
      for (int i = 0; i < UE; ++i) {
        const int2 kt2 = a.ktab[kk0 + i];
        const int rd = kt2.y >> 16, sd = kt2.y & 0xffff;
        const bool ok = static_cast<unsigned>(ih0 + rd) < H && static_cast<unsigned>(iw0 + sd) < W;
        const uint32_t vo = ok ? static_cast<uint32_t>((base + kt2.x) * ES) : a.x_bytes;
        e[i] = buf_load_elem(xr, vo, xg, (T*)nullptr);
      }
      pack16<T>(rb[u], e);
    }
  };
  auto stash = [&]() {
#pragma unroll
    for (int t = 0; t < UA; ++t) {
      const int id = tid + t * kPcThreads;
      store16(&As[(id / 4) * KP + (id % 4) * UE], ra[t]);
    }
#pragma unroll
    for (int u = 0; u < 2; ++u) store16(&Bs[jl * KP + (hv + 2 * u) * UE], rb[u]);
  };

  f32x16_t acc[MI][NJ];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int nj = 0; nj < NJ; ++nj) acc[mi][nj] = zero16();

  const int nk = a.KRp / BK;
  fetch(0);
  stash();
  lds_sync();
  for (int kt = 0; kt < nk; ++kt) {
    const bool more = kt + 1 < nk;
    if (more) fetch(kt + 1);
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const int kofs = st * 2 * UE + half * UE;
      vec16 af[MI], bfr[NJ];
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) af[mi] = load16(&As[(wm * (BM / 2) + mi * 32 + l32) * KP + kofs]);
#pragma unroll
      for (int nj = 0; nj < NJ; ++nj) bfr[nj] = load16(&Bs[(wn * (BN / 2) + nj * 32 + l32) * KP + kofs]);
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int nj = 0; nj < NJ; ++nj) mfma_32x32<T>(acc[mi][nj], af[mi], bfr[nj]);
    }
    lds_sync();
    if (more) {
      stash();
      lds_sync();
    }
  }
  store_tile<T, BM>(acc, reinterpret_cast<vec16*>(smem), a.e, j0, k0, g, 0);
}

// Filters, zero-padded: wp[g][k][kk] = w[g*Kg + k][kk] for k < Kg, kk < Kred.
template <typename T>
__global__ __launch_bounds__(256) void precomp_pack_filters_kernel(const T* __restrict__ w, T* __restrict__ wp, int Kg,
                                                                    int Kred, int Kpad, int KRp) {
  const int row = blockIdx.x;  // g*Kpad + k
  const int g = row / Kpad, k = row - g * Kpad;
  for (int kk = threadIdx.x; kk < KRp; kk += 256) {
    T v = elem<T>::from_f32(0.f);
    if (k < Kg && kk < Kred) v = w[(static_cast<int64_t>(g) * Kg + k) * Kred + kk];
    wp[static_cast<int64_t>(row) * KRp + kk] = v;
  }
}

// The two index tables (see the top of this file).
__global__ __launch_bounds__(256) void precomp_tables_kernel(int2* __restrict__ ktab, int2* __restrict__ ptab, int Kred,
                                                             int KRp, int NPQ, int C, int H, int W, int R, int S,
                                                             int P, int Q, int sh, int sw, int ph, int pw, int dh,
                                                             int dw) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < KRp) {
    int2 t;
    if (i < Kred) {
      const int c = i / (R * S), rs = i - c * (R * S);
      const int r = rs / S, s = rs - r * S;
      t.x = c * H * W + r * dh * W + s * dw;
      t.y = ((r * dh) << 16) | (s * dw);
    } else {
      t.x = 0;
      t.y = kOutside << 16;
    }
    ktab[i] = t;
  }
  if (i < NPQ) {
    const int PQ = P * Q;
    const int n = i / PQ, pq = i - n * PQ;
    const int p = pq / Q, q = pq - p * Q;
    const int ih0 = p * sh - ph, iw0 = q * sw - pw;
    int2 t;
    t.x = n * C * H * W + ih0 * W + iw0;
    t.y = static_cast<int>((static_cast<uint32_t>(ih0) << 16) | (static_cast<uint32_t>(iw0) & 0xffffu));
    ptab[i] = t;
  }
}

struct PcPlan {
  int BM;
  int64_t images_per_launch;
  int Kred, KRp, Kpad, ktiles;
  size_t wp_bytes, ktab_off, ptab_off, total;
};

bool make_pc_plan(const Shape& s, PcPlan& pl) {
  const int UE = s.dtype == DT_F32 ? 4 : 8;
  const int BK = 4 * UE;
  // Coordinates and displacements are packed as 16-bit halves.
  if (s.H + 2 * s.ph >= kOutside || s.W + 2 * s.pw >= kOutside) return false;
  const int64_t img_bytes = s.C * s.H * s.W * s.esize();
  if (img_bytes > kMaxLaunchBytes) return false;
  int64_t N1 = kMaxLaunchBytes / img_bytes;
  if (N1 > s.N) N1 = s.N;
  if (N1 < 1) N1 = 1;
  pl.images_per_launch = N1;
  pl.Kred = (int)(s.Cg * s.R * s.S);
  pl.KRp = (pl.Kred + BK - 1) / BK * BK;
  pl.BM = s.Kg <= 64 ? 64 : 128;
  pl.ktiles = (int)((s.Kg + pl.BM - 1) / pl.BM);
  pl.Kpad = pl.ktiles * pl.BM;
  if ((int64_t)pl.ktiles * s.G > 65535) return false;  // grid rows
  pl.wp_bytes = (size_t)s.G * pl.Kpad * pl.KRp * s.esize();
  if (pl.wp_bytes > (size_t)kMaxLaunchBytes) return false;
  pl.ktab_off = align256(pl.wp_bytes);
  pl.ptab_off = align256(pl.ktab_off + (size_t)pl.KRp * sizeof(int2));
  pl.total = pl.ptab_off + (size_t)(N1 * s.P * s.Q) * sizeof(int2);
  return true;
}

template <typename T, int BM>
hipError_t pc_launch(const PcArgs& a, hipStream_t stream) {
  const dim3 grid((unsigned)((a.NPQ + BN - 1) / BN), (unsigned)(a.ktiles * a.G));
  hipLaunchKernelGGL((implicit_precomp_kernel<T, BM>), grid, dim3(kPcThreads), 0, stream, a);
  return hipGetLastError();
}

template <typename T>
hipError_t pc_pack_typed(const Shape& s, const PcPlan& pl, const void* w, void* pkg, hipStream_t stream) {
  char* base = reinterpret_cast<char*>(pkg);
  hipLaunchKernelGGL(precomp_pack_filters_kernel<T>, dim3((unsigned)(s.G * pl.Kpad)), dim3(256), 0, stream,
                     reinterpret_cast<const T*>(w), reinterpret_cast<T*>(base), (int)s.Kg, pl.Kred, pl.Kpad, pl.KRp);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int64_t NPQ = pl.images_per_launch * s.P * s.Q;
  const int64_t n = NPQ > pl.KRp ? NPQ : pl.KRp;
  hipLaunchKernelGGL(precomp_tables_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream,
                     reinterpret_cast<int2*>(base + pl.ktab_off), reinterpret_cast<int2*>(base + pl.ptab_off),
                     pl.Kred, pl.KRp, (int)NPQ, (int)s.C, (int)s.H, (int)s.W, (int)s.R, (int)s.S, (int)s.P,
                     (int)s.Q, s.sh, s.sw, s.ph, s.pw, s.dh, s.dw);
  return hipGetLastError();
}

template <typename T>
hipError_t pc_main_typed(const Shape& s, const PcPlan& pl, const void* x, const void* pkg, const void* b, void* y,
                         hipStream_t stream) {
  const char* base = reinterpret_cast<const char*>(pkg);
  const int64_t img_elems = s.C * s.H * s.W, out_elems = s.K * s.P * s.Q;
  for (int64_t n0 = 0; n0 < s.N; n0 += pl.images_per_launch) {
    const int64_t cnt = s.N - n0 < pl.images_per_launch ? s.N - n0 : pl.images_per_launch;
    PcArgs a;
    a.x = reinterpret_cast<const T*>(x) + n0 * img_elems;
    a.wp = base;
    a.ktab = reinterpret_cast<const int2*>(base + pl.ktab_off);
    a.ptab = reinterpret_cast<const int2*>(base + pl.ptab_off);
    a.x_bytes = (uint32_t)(cnt * img_elems * s.esize());
    a.wp_bytes = (uint32_t)pl.wp_bytes;
    a.H = (int)s.H; a.W = (int)s.W; a.Cg = (int)s.Cg; a.G = s.G;
    a.KRp = pl.KRp; a.Kpad = pl.Kpad; a.ktiles = pl.ktiles;
    a.NPQ = (int)(cnt * s.P * s.Q);
    a.group_stride = s.Cg * s.H * s.W;
    EpiArgs& e = a.e;
    e.b = b;
    e.y = reinterpret_cast<T*>(y) + n0 * out_elems;
    e.partial = nullptr;
    e.K = (int)s.K; e.Kg = (int)s.Kg; e.NPQ = a.NPQ; e.PQ = (int)(s.P * s.Q);
    e.relu = s.relu ? 1 : 0;
    e.span = e.PQ;
    e.splits = 1;
    e.slab = 0;
    e.vec = store_piece(s, e.y);
    const hipError_t err = pl.BM == 64 ? pc_launch<T, 64>(a, stream) : pc_launch<T, 128>(a, stream);
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

}  // namespace

bool precomp_applies(const Shape& s) {
  PcPlan pl;
  return make_pc_plan(s, pl);
}

size_t precomp_packed_bytes(const Shape& s) {
  PcPlan pl;
  return make_pc_plan(s, pl) ? pl.total : 0;
}

hipError_t precomp_pack(const Shape& s, const void* w, void* pkg, hipStream_t stream) {
  PcPlan pl;
  if (!make_pc_plan(s, pl)) return hipErrorInvalidValue;
  return s.dtype == DT_F32 ? pc_pack_typed<float>(s, pl, w, pkg, stream)
                           : pc_pack_typed<bf16_t>(s, pl, w, pkg, stream);
}

hipError_t precomp_main(const Shape& s, const void* x, const void* pkg, const void* b, void* y, hipStream_t stream) {
  PcPlan pl;
  if (!make_pc_plan(s, pl)) return hipErrorInvalidValue;
  return s.dtype == DT_F32 ? pc_main_typed<float>(s, pl, x, pkg, b, y, stream)
                           : pc_main_typed<bf16_t>(s, pl, x, pkg, b, y, stream);
}

std::string precomp_describe(const Shape& s) {
  PcPlan pl;
  if (!make_pc_plan(s, pl)) return "implicit_precomp_gemm: not supported";
  const char* tn = s.dtype == DT_F32 ? "f32" : "bf16";
  char buf[384];
  snprintf(buf, sizeof(buf),
           "implicit_precomp_gemm kernels=precomp_pack_filters_kernel<%s>;precomp_tables_kernel;"
           "implicit_precomp_kernel<%s,%d> tile=%dx%d grid=%lldx%d reduction=%d(padded %d) images_per_launch=%lld",
           tn, tn, pl.BM, pl.BM, BN, (long long)((pl.images_per_launch * s.P * s.Q + BN - 1) / BN),
           pl.ktiles * s.G, pl.Kred, pl.KRp, (long long)pl.images_per_launch);
  return buf;
}

}  // namespace convsel
