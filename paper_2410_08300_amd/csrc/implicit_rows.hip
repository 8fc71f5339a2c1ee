// Implicit GEMM (paper, Sec. V-B item (b)) for layers with few input
// channels and wide filters, such as the 7x7 stride-2 stem of ResNet-50
// (C = 3): bf16, one group, 5 <= S <= 8, no column dilation, even column
// stride.
//
// The reduction over (c, r, s) is regrouped into filter rows: with the filter
// width padded to 8 (zero weights), reduction slice u = (c, r) of an MFMA
// lane is 8 consecutive input pixels of one input row.  When the left
// padding is odd one zero tap is put in front of the filter, so that every
// run starts at an even column: a B operand is then four aligned 32-bit LDS
// reads from the input halo, staged as it lies in memory (channels x virtual
// rows x columns, zero borders included).  No column matrix is formed and no
// channel vector is gathered.  The filters are packed once into the exact LDS
// image of a 64-channel tile ([k][(c, r)][8 taps], odd row stride in 16-byte
// units), which each workgroup copies with 16-byte loads.
#include <stdio.h>

#include <atomic>
#include <string>

#include "common.hpp"
#include "igemm_common.hpp"
#include "kernels.hpp"

namespace convsel {

namespace {

using namespace igemm;

constexpr int kRowBM = 64;
constexpr int kRowMaxUnits = 64;  // C*R filter rows per output channel
// 16-byte loads per thread issued before any is written: twelve take all of
// the stem's halo and filter tile (2,282 chunks for 256 threads) in one round
// trip (eight took two; 36.0 -> 34.4 us per prepacked call).
constexpr int kRowLoadBatch = 12;
constexpr uint32_t kOut = 0x80000000u;  // a buffer offset past every buffer: loads read zero

struct RowArgs {
  const void* x;        // input of this launch
  const void* wp;       // filter package: [K tile][64][UR][8] bf16
  uint32_t x_bytes, wp_bytes;
  int N, C, H, W, K, R, P, Q;
  int sh, sw, ph, dh;
  int S, lead;          // filter width; zero taps put in front of it (0 or 1)
  int off;              // halo column of input column 0 (a multiple of 8)
  int cshift;           // halo column read by tap 0 of output column 0 (even)
  int Hv, VR, NPQ;      // virtual rows per image, halo rows of a tile, output pixels
  int BRS;              // halo row length in elements (a multiple of 8)
  int CR;               // filter rows per output channel (C*R)
  int UR;               // filter units per output channel in the package and in LDS (odd)
  int lds_b;            // byte offset of the halo in LDS
  int lds_t;            // byte offset of the per-unit halo offsets
  EpiArgs e;
};

// VEC: the input rows are whole 16-byte chunks (W % 8 == 0, 16-byte aligned
// input), staged with 16-byte loads; otherwise element by element.
template <bool VEC>
__global__ __launch_bounds__(kThreads) void implicit_rows_kernel(RowArgs a) {
  constexpr int BM = kRowBM, NJ = 2;
  extern __shared__ __align__(16) vec16 smem[];
  char* lds = reinterpret_cast<char*>(smem);
  u32x4_t* As = reinterpret_cast<u32x4_t*>(lds);                   // [BM][UR]
  uint16_t* Bs = reinterpret_cast<uint16_t*>(lds + a.lds_b);       // [C][VR][BRS]
  int* uoff = reinterpret_cast<int*>(lds + a.lds_t);               // halo offset of unit (c, r)

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int half = lane >> 5, l32 = lane & 31;
  const int j0 = blockIdx.x * BN, k0 = blockIdx.y * BM;
  const int PQ = a.P * a.Q;
  auto vrow_of = [&](int j) {
    const int n = j / PQ, pq = j - n * PQ;
    return n * a.Hv + (pq / a.Q) * a.sh;
  };
  const int vr_lo = vrow_of(j0);
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, a.x_bytes), wr = make_rsrc(a.wp, a.wp_bytes);

  // Halo: Bs[c][vr][col] = x[n][c][ih][col - off] for virtual row vr_lo + vr
  // (image n, row ih), zero outside the image.  A load whose element lies
  // outside passes an offset past the buffer's end and reads zero.
  const int rows = a.C * a.VR;
  // Filters: the package tile is the LDS image itself.
  const int units = BM * a.UR;
  const uint32_t wbase = static_cast<uint32_t>(blockIdx.y) * units * 16;
  auto halo_off = [&](int row, int iw) -> uint32_t {  // byte offset of (row, iw), or kOut outside the image
    const int c = row / a.VR, vv = vr_lo + row - c * a.VR;
    const int n = vv / a.Hv, ih = vv - n * a.Hv - a.ph;
    const bool ok = n < a.N && ih >= 0 && ih < a.H && iw >= 0 && iw < a.W;
    return ok ? (((static_cast<uint32_t>(n) * a.C + c) * a.H + ih) * a.W + iw) * 2 : kOut;
  };
  if constexpr (VEC) {
    // Halo chunks (16 bytes: 8 columns of one row) and filter units go out
    // in one stream of loads, kRowLoadBatch per thread before any is
    // written, so a workgroup waits for memory once before its first MFMA.
    const int cpr = a.BRS / 8;  // 16-byte chunks per halo row
    const int total = rows * cpr;
    const int all = total + units;
    for (int i0 = tid; i0 < all; i0 += kRowLoadBatch * kThreads) {
      u32x4_t v[kRowLoadBatch];
#pragma unroll
      for (int t = 0; t < kRowLoadBatch; ++t) {
        const int i = i0 + t * kThreads;
        if (i < total) {
          const int row = i / cpr, ch = i - row * cpr;
          v[t] = __builtin_amdgcn_raw_buffer_load_b128(xr, halo_off(row, ch * 8 - a.off), 0, 0);
        } else {
          const int u = i - total;
          v[t] = __builtin_amdgcn_raw_buffer_load_b128(wr, u < units ? wbase + u * 16 : kOut, 0, 0);
        }
      }
#pragma unroll
      for (int t = 0; t < kRowLoadBatch; ++t) {
        const int i = i0 + t * kThreads;
        if (i < total)
          reinterpret_cast<u32x4_t*>(Bs)[i] = v[t];
        else if (i < all)
          As[i - total] = v[t];
      }
    }
  } else {
    for (int col = tid; col < a.BRS; col += kThreads) {
      const int iw = col - a.off;
      for (int r0 = 0; r0 < rows; r0 += 8) {
        uint32_t v[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const int row = r0 + t;
          v[t] = buf_load_elem(xr, row < rows ? halo_off(row, iw) : kOut, 0, (bf16_t*)nullptr);
        }
#pragma unroll
        for (int t = 0; t < 8; ++t)
          if (r0 + t < rows) Bs[(r0 + t) * a.BRS + col] = static_cast<uint16_t>(v[t]);
      }
    }
    for (int i0 = tid; i0 < units; i0 += 4 * kThreads) {
      u32x4_t v[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int i = i0 + t * kThreads;
        v[t] = __builtin_amdgcn_raw_buffer_load_b128(wr, i < units ? wbase + i * 16 : kOut, 0, 0);
      }
#pragma unroll
      for (int t = 0; t < 4; ++t)
        if (i0 + t * kThreads < units) As[i0 + t * kThreads] = v[t];
    }
  }
  for (int u = tid; u < a.CR; u += kThreads) {
    const int c = u / a.R, r = u - c * a.R;
    uoff[u] = (c * a.VR + r * a.dh) * a.BRS;
  }
  __syncthreads();

  // Each lane's output pixels: halo element of filter row 0, tap 0.
  int poff[NJ];
#pragma unroll
  for (int nj = 0; nj < NJ; ++nj) {
    const int j = j0 + wn * (BN / 2) + nj * 32 + l32;
    const int jj = j < a.NPQ ? j : a.NPQ - 1;
    const int pq = jj - (jj / PQ) * PQ;
    const int q = pq - (pq / a.Q) * a.Q;
    poff[nj] = (vrow_of(jj) - vr_lo) * a.BRS + q * a.sw + a.cshift;
  }
  // Input elements under the zero taps (before `lead`, at or after
  // lead + S, and the padding unit of an odd C*R) are masked to zero too, so
  // a non-finite input that no real tap reads cannot reach the sum.
  uint32_t smask[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e0 = 2 * q - a.lead, e1 = e0 + 1;
    smask[q] = (e0 >= 0 && e0 < a.S ? 0xFFFFu : 0u) | (e1 >= 0 && e1 < a.S ? 0xFFFF0000u : 0u);
  }
  f32x16_t acc[1][NJ];
#pragma unroll
  for (int nj = 0; nj < NJ; ++nj) acc[0][nj] = zero16();
  const int arow = (wm * 32 + l32) * a.UR;
  const int steps = (a.CR + 1) / 2;
  for (int st = 0; st < steps; ++st) {
    const int u = 2 * st + half;
    const bool real = u < a.CR;
    const int uo = uoff[real ? u : a.CR - 1];
    const bf16x8_t af = __builtin_bit_cast(bf16x8_t, As[arow + u]);
#pragma unroll
    for (int nj = 0; nj < NJ; ++nj) {
      // 8 consecutive elements starting at an even element: four aligned words.
      const uint32_t* p = reinterpret_cast<const uint32_t*>(Bs + uo + poff[nj]);
      u32x4_t b;
#pragma unroll
      for (int q = 0; q < 4; ++q) b[q] = p[q] & (real ? smask[q] : 0u);
      acc[0][nj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, __builtin_bit_cast(bf16x8_t, b), acc[0][nj], 0, 0, 0);
    }
  }
  __syncthreads();  // the epilogue stages through the same LDS
  store_tile<bf16_t, BM>(acc, smem, a.e, j0, k0, 0, 0);
}

// Package: unit (k, u) of tile kt holds taps lead .. lead+S-1 of filter row
// u = c*R + r of output channel kt*64 + k, zeros elsewhere.
__global__ __launch_bounds__(256) void rows_pack_kernel(const uint16_t* __restrict__ w, u32x4_t* __restrict__ wp, int K,
                                                       int CR, int S, int lead, int UR, int units) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= units) return;
  const int k = i / UR, u = i - k * UR;
  // All eight loads go out before any is used; a zero tap reads w[0] and is
  // then replaced by zero.
  uint32_t v[8];
  bool ok[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int s = e - lead;
    ok[e] = k < K && u < CR && s >= 0 && s < S;
    v[e] = w[ok[e] ? (static_cast<int64_t>(k) * CR + u) * S + s : 0];
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = ok[e] ? v[e] : 0u;
  u32x4_t o;
#pragma unroll
  for (int q = 0; q < 4; ++q) o[q] = v[2 * q] | (v[2 * q + 1] << 16);
  wp[i] = o;
}

struct RowPlan {
  int64_t images_per_launch;
  int ktiles;
  size_t lds;
  RowArgs a;
};

bool make_row_plan(const Shape& s, RowPlan& pl, int64_t N1 = -1) {
  if (s.dtype != DT_BF16 || s.G != 1 || s.S > 8 || s.S < 5 || s.dw != 1 || s.sw % 2 != 0) return false;
  const int lead = s.pw % 2;
  if (s.S + lead > 8) return false;
  if (s.C * s.R > kRowMaxUnits || s.P * s.Q == 0 || s.N == 0) return false;
  const int64_t img_bytes = s.C * s.H * s.W * 2;
  const int64_t Hv = (s.P - 1) * s.sh + (s.R - 1) * s.dh + 1;
  // Per image: its input, its output and its virtual rows; a launch keeps
  // each total below 2^31 (32-bit indices) and its input within 1 GiB.
  int64_t per_img = s.C * s.H * s.W;
  if (s.K * s.P * s.Q > per_img) per_img = s.K * s.P * s.Q;
  if (Hv > per_img) per_img = Hv;
  int64_t cap = ((int64_t)1 << 31) / (per_img + 1);
  if (kMaxLaunchBytes / img_bytes < cap) cap = kMaxLaunchBytes / img_bytes;
  if (cap < 1) return false;
  if (N1 < 0) N1 = s.N < cap ? s.N : cap;
  pl.images_per_launch = N1;
  RowArgs& a = pl.a;
  a.N = (int)N1; a.C = (int)s.C; a.H = (int)s.H; a.W = (int)s.W; a.K = (int)s.K;
  a.R = (int)s.R; a.S = (int)s.S; a.P = (int)s.P; a.Q = (int)s.Q;
  a.sh = s.sh; a.sw = s.sw; a.ph = s.ph; a.dh = s.dh;
  a.lead = lead;
  a.off = (s.pw + lead + 7) / 8 * 8;
  a.cshift = a.off - s.pw - lead;
  a.Hv = (int)Hv;
  a.VR = halo_rows(s, N1, a.Hv);
  a.NPQ = (int)(N1 * s.P * s.Q);
  // Columns read: cshift + q*sw + 0..7 for q < Q; input columns sit at off .. off+W-1.
  int64_t brs = a.cshift + (s.Q - 1) * s.sw + 8;
  if (a.off + s.W > brs) brs = a.off + s.W;
  a.BRS = (int)((brs + 7) / 8 * 8);
  a.CR = (int)(s.C * s.R);
  a.UR = ((a.CR + 1) / 2 * 2) | 1;
  pl.ktiles = (int)((s.K + kRowBM - 1) / kRowBM);
  const size_t a_bytes = (size_t)kRowBM * a.UR * 16;
  const size_t b_bytes = (size_t)s.C * a.VR * a.BRS * 2;
  if ((size_t)pl.ktiles * a_bytes >= ((size_t)1 << 31)) return false;
  a.wp_bytes = (uint32_t)(pl.ktiles * a_bytes);
  a.lds_b = (int)a_bytes;
  a.lds_t = (int)((a_bytes + b_bytes + 15) / 16 * 16);
  const size_t lds = a.lds_t + (size_t)kRowMaxUnits * sizeof(int);
  const size_t stage = (size_t)4 * 32 * (BN / 2) * sizeof(float);  // epilogue staging
  pl.lds = lds > stage ? lds : stage;
  if (pl.lds > kLdsLimit) return false;
  a.e.K = (int)s.K; a.e.Kg = (int)s.K; a.e.PQ = (int)(s.P * s.Q); a.e.span = a.e.PQ; a.e.relu = s.relu ? 1 : 0;
  a.e.NPQ = a.NPQ;
  a.e.splits = 1;
  a.e.slab = 0;
  a.e.partial = nullptr;
  return true;
}

}  // namespace

bool rows_applies(const Shape& s) {
  RowPlan pl;
  return make_row_plan(s, pl);
}

size_t rows_packed_bytes(const Shape& s) {
  RowPlan pl;
  return make_row_plan(s, pl) ? pl.a.wp_bytes : 0;
}

hipError_t rows_pack(const Shape& s, const void* w, void* wp, hipStream_t stream) {
  RowPlan pl;
  if (!make_row_plan(s, pl)) return hipErrorInvalidValue;
  const int units = pl.ktiles * kRowBM * pl.a.UR;
  hipLaunchKernelGGL(rows_pack_kernel, dim3((units + 255) / 256), dim3(256), 0, stream,
                     reinterpret_cast<const uint16_t*>(w), reinterpret_cast<u32x4_t*>(wp), (int)s.K, pl.a.CR,
                     (int)s.S, pl.a.lead, pl.a.UR, units);
  return hipGetLastError();
}

hipError_t rows_main(const Shape& s, const void* x, const void* wp, const void* b, void* y, hipStream_t stream,
                     const void* res) {
  RowPlan pl;
  if (!make_row_plan(s, pl)) return hipErrorInvalidValue;
  const int64_t img_elems = s.C * s.H * s.W, out_elems = s.K * s.P * s.Q;
  const bool vec = s.W % 8 == 0 && reinterpret_cast<uintptr_t>(x) % 16 == 0;
  for (int64_t n0 = 0; n0 < s.N; n0 += pl.images_per_launch) {
    const int64_t cnt = s.N - n0 < pl.images_per_launch ? s.N - n0 : pl.images_per_launch;
    RowPlan cur = pl;
    if (cnt != pl.images_per_launch && !make_row_plan(s, cur, cnt)) return hipErrorInvalidValue;
    RowArgs a = cur.a;
    a.x = reinterpret_cast<const uint16_t*>(x) + n0 * img_elems;
    a.x_bytes = (uint32_t)(cnt * img_elems * 2);
    a.wp = wp;
    a.e.y = reinterpret_cast<uint16_t*>(y) + n0 * out_elems;
    a.e.res = res ? reinterpret_cast<const uint16_t*>(res) + n0 * out_elems : nullptr;
    a.e.b = b;
    a.e.vec = store_piece(s, a.e.y);
    const dim3 grid((unsigned)((a.NPQ + BN - 1) / BN), (unsigned)cur.ktiles);
    // Raise the kernels' dynamic-LDS limit once (calls may be captured into
    // a graph after the first one).
    static std::atomic<int> lds_limit{64 * 1024};
    if ((int)cur.lds > lds_limit.load()) {
      for (const void* k : {reinterpret_cast<const void*>(implicit_rows_kernel<true>),
                            reinterpret_cast<const void*>(implicit_rows_kernel<false>)}) {
        const hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsLimit);
        if (e != hipSuccess) return e;
      }
      lds_limit.store((int)kLdsLimit);
    }
    if (vec)
      hipLaunchKernelGGL(implicit_rows_kernel<true>, grid, dim3(kThreads), cur.lds, stream, a);
    else
      hipLaunchKernelGGL(implicit_rows_kernel<false>, grid, dim3(kThreads), cur.lds, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

std::string rows_describe(const Shape& s) {
  RowPlan pl;
  if (!make_row_plan(s, pl)) return "implicit_gemm (filter rows): not applicable";
  char buf[384];
  snprintf(buf, sizeof(buf),
           "implicit_gemm kernels=rows_pack_kernel;implicit_rows_kernel tile=%dx%d grid=%dx%d filter_rows=%d "
           "lead_taps=%d halo_rows=%d halo_cols=%d lds=%zu images_per_launch=%lld (filter rows of width 8 as "
           "reduction slices; 16-byte halo loads when W %% 8 == 0)",
           kRowBM, BN, (pl.a.NPQ + BN - 1) / BN, pl.ktiles, pl.a.CR, pl.a.lead, pl.a.VR, pl.a.BRS, pl.lds,
           (long long)pl.images_per_launch);
  return buf;
}

}  // namespace convsel
