// Implicit GEMM (paper, Sec. V-B item (b)) for layers with few input
// channels and wide filters, such as the 7x7 stride-2 stem of ResNet-50
// (C = 3): bf16, one group, S <= 8, no column dilation, even column stride.
//
// The reduction over (c, r, s) is regrouped into filter rows: with the filter
// width padded to 8 (zero weights for s >= S), reduction slice u = (c, r) of
// an MFMA lane is the 8 consecutive input pixels x[n][c][ih][iw0 .. iw0+7]
// of one input row, iw0 = q*sw - pw.  With an even stride these runs start
// at an even column, so a B operand is four aligned 32-bit LDS reads from
// the input halo staged as it lies in memory (channels x virtual rows x
// columns); no column matrix is formed and no channel vector is gathered.
// The filters of a 64-channel tile ([k][(c, r)][8], 16-byte units, odd row
// stride) stay in LDS for the workgroup's whole life.
#include <stdio.h>
#include <string>

#include "common.hpp"
#include "igemm_common.hpp"
#include "kernels.hpp"

namespace convsel {

namespace {

using namespace igemm;

constexpr int kRowBM = 64;
constexpr int kRowMaxUnits = 64;  // C*R filter rows per output channel

struct RowArgs {
  const void* x;        // input of this launch
  const void* w;        // filters, K x C x R x S
  uint32_t x_bytes, w_bytes;
  int N, C, H, W, K, R, S, P, Q;
  int sh, sw, ph, pw, dh;
  int Hv, VR, NPQ;      // virtual rows per image, halo rows of a tile, output pixels
  int BRS;              // halo row length in elements (even)
  int CR;               // filter rows per output channel (C*R)
  int UR;               // LDS row stride of the filter tile, 16-byte units (odd, >= CR rounded up to even)
  int ktiles;
  int lds_b;            // byte offset of the halo in LDS
  int lds_t;            // byte offset of the per-unit halo offsets
  EpiArgs e;
};

__global__ __launch_bounds__(kThreads) void implicit_rows_kernel(RowArgs a) {
  constexpr int BM = kRowBM, MI = 1, NJ = 2;
  extern __shared__ __align__(16) vec16 smem[];
  char* lds = reinterpret_cast<char*>(smem);
  bf16x8_t* As = reinterpret_cast<bf16x8_t*>(lds);                 // [BM][UR]
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
  // Buffer loads: a lane whose element lies outside the image or the
  // filter tensor passes an offset past the buffer's end and reads zero.
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, a.x_bytes), wr = make_rsrc(a.w, a.w_bytes);
  constexpr uint32_t kOut = 0x80000000u;

  // Filters: As[k][u][s] = w[k0 + k][c][r][s] (u = c*R + r), zero for s >= S,
  // u >= CR or k0 + k >= K.  Thread i of a pass writes unit i of the tile.
  for (int i = tid; i < BM * a.UR; i += kThreads) {
    const int k = i / a.UR, u = i - k * a.UR;
    const bool ok = u < a.CR && k0 + k < a.K;
    const uint32_t base = (static_cast<uint32_t>(k0 + k) * a.CR + u) * a.S * 2;
    uint32_t v[8];
#pragma unroll
    for (int s = 0; s < 8; ++s) v[s] = buf_load_elem(wr, ok && s < a.S ? base + 2 * s : kOut, 0, (bf16_t*)nullptr);
    vec16 o;
#pragma unroll
    for (int q = 0; q < 4; ++q) o.d[q] = (v[2 * q] & 0xFFFFu) | (v[2 * q + 1] << 16);
    reinterpret_cast<vec16*>(As)[i] = o;
  }
  // Halo: Bs[c][vr][col] = x[n][c][ih][col - pw] for virtual row vr_lo + vr
  // (image n, row ih), zero outside the image.  Thread t owns columns
  // t, t + 256, ... and walks the rows, eight loads at a time.
  const int rows = a.C * a.VR;
  for (int col = tid; col < a.BRS; col += kThreads) {
    const int iw = col - a.pw;
    const bool col_ok = iw >= 0 && iw < a.W;
    for (int r0 = 0; r0 < rows; r0 += 8) {
      uint32_t v[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int row = r0 + t;
        const int c = row / a.VR, vr = row - c * a.VR;
        const int vv = vr_lo + vr;
        const int n = vv / a.Hv, ih = vv - n * a.Hv - a.ph;
        const bool ok = row < rows && col_ok && n < a.N && ih >= 0 && ih < a.H;
        const uint32_t off = (((static_cast<uint32_t>(n) * a.C + c) * a.H + ih) * a.W + iw) * 2;
        v[t] = buf_load_elem(xr, ok ? off : kOut, 0, (bf16_t*)nullptr);
      }
#pragma unroll
      for (int t = 0; t < 8; ++t)
        if (r0 + t < rows) Bs[(r0 + t) * a.BRS + col] = static_cast<uint16_t>(v[t]);
    }
  }
  for (int u = tid; u < a.CR; u += kThreads) {
    const int c = u / a.R, r = u - c * a.R;
    uoff[u] = (c * a.VR + r * a.dh) * a.BRS;
  }
  __syncthreads();

  // Each lane's output pixels: halo element of filter row 0, column 0.
  int poff[NJ];
#pragma unroll
  for (int nj = 0; nj < NJ; ++nj) {
    const int j = j0 + wn * (BN / 2) + nj * 32 + l32;
    const int jj = j < a.NPQ ? j : a.NPQ - 1;
    const int pq = jj - (jj / PQ) * PQ;
    const int q = pq - (pq / a.Q) * a.Q;
    poff[nj] = (vrow_of(jj) - vr_lo) * a.BRS + q * a.sw;
  }
  f32x16_t acc[MI][NJ];
#pragma unroll
  for (int nj = 0; nj < NJ; ++nj) acc[0][nj] = zero16();
  const int arow = (wm * 32 + l32) * a.UR;
  // Input elements under the zero weights (taps s >= S, the padding unit
  // of an odd C*R) are masked to zero as well, so a non-finite input that no
  // real tap reads cannot reach the sum.
  uint32_t smask[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) smask[q] = (2 * q < a.S ? 0xFFFFu : 0u) | (2 * q + 1 < a.S ? 0xFFFF0000u : 0u);
  const int steps = (a.CR + 1) / 2;
  for (int st = 0; st < steps; ++st) {
    const int u = 2 * st + half;
    const bool real = u < a.CR;
    const int uo = uoff[real ? u : a.CR - 1];
    const bf16x8_t af = As[arow + u];
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

struct RowPlan {
  int64_t images_per_launch;
  size_t lds;
  RowArgs a;
};

bool make_row_plan(const Shape& s, RowPlan& pl, int64_t N1 = -1) {
  if (s.dtype != DT_BF16 || s.G != 1 || s.S > 8 || s.S < 5 || s.dw != 1 || s.sw % 2 != 0) return false;
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
  if (cap < 1 || s.K * s.C * s.R * s.S * 2 > kMaxLaunchBytes) return false;
  if (N1 < 0) N1 = s.N < cap ? s.N : cap;
  pl.images_per_launch = N1;
  RowArgs& a = pl.a;
  a.N = (int)N1; a.C = (int)s.C; a.H = (int)s.H; a.W = (int)s.W; a.K = (int)s.K;
  a.R = (int)s.R; a.S = (int)s.S; a.P = (int)s.P; a.Q = (int)s.Q;
  a.sh = s.sh; a.sw = s.sw; a.ph = s.ph; a.pw = s.pw; a.dh = s.dh;
  a.Hv = (int)((s.P - 1) * s.sh + (s.R - 1) * s.dh + 1);
  a.VR = halo_rows(s, N1, a.Hv);
  a.NPQ = (int)(N1 * s.P * s.Q);
  // Columns read: q*sw + 0..7 for q < Q (the runs extend past S into zero weights).
  a.BRS = (int)(((s.Q - 1) * s.sw + 8 + 1) / 2 * 2);
  a.CR = (int)(s.C * s.R);
  a.UR = ((a.CR + 1) / 2 * 2) | 1;
  a.ktiles = (int)((s.K + kRowBM - 1) / kRowBM);
  const size_t a_bytes = (size_t)kRowBM * a.UR * 16;
  const size_t b_bytes = (size_t)s.C * a.VR * a.BRS * 2;
  a.lds_b = (int)a_bytes;
  a.lds_t = (int)((a_bytes + b_bytes + 15) / 16 * 16);
  size_t lds = a.lds_t + (size_t)kRowMaxUnits * sizeof(int);
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

hipError_t rows_main(const Shape& s, const void* x, const void* w, const void* b, void* y, hipStream_t stream) {
  RowPlan pl;
  if (!make_row_plan(s, pl)) return hipErrorInvalidValue;
  const int64_t img_elems = s.C * s.H * s.W, out_elems = s.K * s.P * s.Q;
  for (int64_t n0 = 0; n0 < s.N; n0 += pl.images_per_launch) {
    const int64_t cnt = s.N - n0 < pl.images_per_launch ? s.N - n0 : pl.images_per_launch;
    RowPlan cur = pl;
    if (cnt != pl.images_per_launch && !make_row_plan(s, cur, cnt)) return hipErrorInvalidValue;
    RowArgs a = cur.a;
    a.x = reinterpret_cast<const uint16_t*>(x) + n0 * img_elems;
    a.w = w;
    a.x_bytes = (uint32_t)(cnt * img_elems * 2);
    a.w_bytes = (uint32_t)(s.K * s.C * s.R * s.S * 2);
    a.e.y = reinterpret_cast<uint16_t*>(y) + n0 * out_elems;
    a.e.b = b;
    a.e.vec = store_piece(s, a.e.y);
    const dim3 grid((unsigned)((a.NPQ + BN - 1) / BN), (unsigned)a.ktiles);
    hipLaunchKernelGGL(implicit_rows_kernel, grid, dim3(kThreads), cur.lds, stream, a);
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
           "implicit_gemm kernels=implicit_rows_kernel tile=%dx%d grid=%dx%d filter_rows=%d halo_rows=%d lds=%zu "
           "images_per_launch=%lld (filter rows of width 8 as reduction slices; filters used as given)",
           kRowBM, BN, (pl.a.NPQ + BN - 1) / BN, pl.a.ktiles, pl.a.CR, pl.a.VR, pl.lds,
           (long long)pl.images_per_launch);
  return buf;
}

}  // namespace convsel
