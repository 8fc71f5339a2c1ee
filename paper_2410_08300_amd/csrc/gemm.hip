// Batched MFMA GEMM with both operands reduction-contiguous ("NT"):
//   C[b][i][j] = sum_k A[b][i][k] * B[b][j][k]  (+ bias[i], ReLU)
// It is the multiply step of IM2COL + GEMM (A = filters, B = the column
// matrix, C = one image's output planes) and the 16 elementwise-product
// GEMMs of Winograd (A = U, B = V, C = M).  With `b_kmajor` set, B is read
// as B[b][k][j] instead (column-contiguous: an NCHW image as channels x
// pixels), which is the multiply step of KN2ROW; its tile is transposed on
// the way into LDS.
//
// Tiling: 256 threads = 4 waves in a 2 x 2 grid; a BM x BN tile per
// workgroup, (BM/2) x (BN/2) per wave as 32 x 32 MFMA blocks.  Each k-tile of
// BK reduction elements is staged in LDS as rows of BK (+ 16 bytes padding:
// an 80-byte row stride, an odd multiple of 16 bytes, so the per-lane 16-byte
// fragment reads of 32 consecutive rows hit distinct bank groups).  The next
// k-tile is fetched into registers while the MFMAs run on the current one.
#include "common.hpp"
#include "kernels.hpp"

namespace convsel {

namespace {

constexpr int kThreads = 256;

template <typename T, int BM, int BN, bool VEC, bool OUT_F32, bool BKM>
__global__ __launch_bounds__(kThreads) void gemm_nt_kernel(GemmArgs g, int batch_base) {
  constexpr int UE = elem<T>::per16;  // elements per 16-byte unit
  constexpr int BK = 4 * UE;          // 32 bf16 or 16 fp32: two MFMA steps
  constexpr int KP = BK + UE;         // padded LDS row (elements)
  constexpr int UPR = BK / UE;        // 16-byte units per row = 4
  constexpr int UA = BM * UPR / kThreads;
  constexpr int UB = BN * UPR / kThreads;
  constexpr int MI = BM / 64, NJ = BN / 64;
  static_assert(UA >= 1 && UB >= 1, "tile too small");

  __shared__ __align__(16) T As[BM * KP];
  __shared__ __align__(16) T Bs[BN * KP];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int i0 = blockIdx.y * BM, j0 = blockIdx.x * BN;
  const int b = batch_base + blockIdx.z;
  const int b0 = b / g.bdiv, b1 = b - b0 * g.bdiv;
  const T* A = reinterpret_cast<const T*>(g.A) + b0 * g.sA0 + b1 * g.sA1;
  const T* B = reinterpret_cast<const T*>(g.B) + b0 * g.sB0 + b1 * g.sB1;

  vec16 ra[UA], rb[UB];

  // One 16-byte unit (UE consecutive reduction elements) of row `row` of a
  // row-major operand, zero outside rows < nrows and k < Kred.  Loads are
  // unconditional from a valid address and masked afterwards, so a thread's
  // loads are all in flight together.
  auto load_unit = [&](const T* base, int row, int k, int nrows, int64_t ld) -> vec16 {
    if (VEC) {
      const bool ok = row < nrows && k < g.Kred;
      const vec16 v = load16(base + (ok ? row * ld + k : 0));
      vec16 r;
#pragma unroll
      for (int i = 0; i < 4; ++i) r.d[i] = ok ? v.d[i] : 0u;
      return r;
    } else {
      uint32_t e[UE];
#pragma unroll
      for (int i = 0; i < UE; ++i) {
        const bool ok = row < nrows && k + i < g.Kred;
        const uint32_t bits = load_bits(base + (ok ? row * ld + k + i : 0));
        e[i] = ok ? bits : 0u;
      }
      vec16 r;
      pack16<T>(r, e);
      return r;
    }
  };

  auto fetch = [&](int kt) {
    const int k0 = kt * BK;
#pragma unroll
    for (int u = 0; u < UA; ++u) {
      const int id = tid + u * kThreads;
      const int row = id / UPR, kc = (id % UPR) * UE;
      const int gi = i0 + row, gk = k0 + kc;
      ra[u] = load_unit(A, gi, gk, g.M, g.lda);
    }
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int id = tid + u * kThreads;
      if constexpr (BKM) {
        // UE consecutive columns of reduction row kr.
        const int kr = id / (BN / UE), jc = id % (BN / UE);
        const int gk = k0 + kr, gj = j0 + jc * UE;
        if (VEC && gk < g.Kred && gj + UE <= g.N) {
          rb[u] = load16(B + gk * g.ldb + gj);
        } else {
          uint32_t e[UE];
#pragma unroll
          for (int i = 0; i < UE; ++i) {
            const bool ok = gk < g.Kred && gj + i < g.N;
            const uint32_t bits = load_bits(B + (ok ? gk * g.ldb + gj + i : 0));
            e[i] = ok ? bits : 0u;
          }
          pack16<T>(rb[u], e);
        }
      } else {
        const int row = id / UPR, kc = (id % UPR) * UE;
        const int gj = j0 + row, gk = k0 + kc;
        rb[u] = load_unit(B, gj, gk, g.N, g.ldb);
      }
    }
  };
  auto stash = [&]() {
#pragma unroll
    for (int u = 0; u < UA; ++u) {
      const int id = tid + u * kThreads;
      store16(&As[(id / UPR) * KP + (id % UPR) * UE], ra[u]);
    }
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int id = tid + u * kThreads;
      if constexpr (BKM) {
        const int kr = id / (BN / UE), jc = id % (BN / UE);
#pragma unroll
        for (int i = 0; i < UE; ++i) Bs[(jc * UE + i) * KP + kr] = vec16_get<T>(rb[u], i);
      } else {
        store16(&Bs[(id / UPR) * KP + (id % UPR) * UE], rb[u]);
      }
    }
  };

  f32x16_t acc[MI][NJ];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int nj = 0; nj < NJ; ++nj) acc[mi][nj] = zero16();

  const int nk = (g.Kred + BK - 1) / BK;
  fetch(0);
  stash();
  lds_sync();
  const int half = lane >> 5, l32 = lane & 31;
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) fetch(kt + 1);
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
    if (kt + 1 < nk) {
      stash();
      lds_sync();
    }
  }

  // Epilogue: bias, ReLU, store.  Lanes 0-31 write 32 consecutive j of one
  // row i, lanes 32-63 the same columns of row i+4.
  const int64_t cofs = b0 * g.sC0 + b1 * g.sC1;
  const T* bias = g.bias ? reinterpret_cast<const T*>(g.bias) + b1 * g.sBias1 : nullptr;
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
    for (int nj = 0; nj < NJ; ++nj) {
      const int j = j0 + wn * (BN / 2) + nj * 32 + l32;
      if (j >= g.N) continue;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int i = i0 + wm * (BM / 2) + mi * 32 + mfma_row(v, lane);
        if (i >= g.M) continue;
        float val = acc[mi][nj][v];
        if (bias) val += elem<T>::load(bias + i);
        if (g.relu) val = fmaxf(val, 0.f);
        const int64_t o = cofs + static_cast<int64_t>(i) * g.ldc + j;
        if (OUT_F32)
          reinterpret_cast<float*>(g.C)[o] = val;
        else
          elem<T>::store(reinterpret_cast<T*>(g.C) + o, val);
      }
    }
  }
}

template <typename T, int BM, int BN, bool OUT_F32, bool BKM>
hipError_t launch_tile(const GemmArgs& g, bool vec, hipStream_t stream) {
  const dim3 block(kThreads);
  for (int base = 0; base < g.batch; base += 65535) {
    const int nb = g.batch - base < 65535 ? g.batch - base : 65535;
    const dim3 grid((g.N + BN - 1) / BN, (g.M + BM - 1) / BM, nb);
    if (vec)
      hipLaunchKernelGGL((gemm_nt_kernel<T, BM, BN, true, OUT_F32, BKM>), grid, block, 0, stream, g, base);
    else
      hipLaunchKernelGGL((gemm_nt_kernel<T, BM, BN, false, OUT_F32, BKM>), grid, block, 0, stream, g, base);
  }
  return hipGetLastError();
}

template <typename T, bool OUT_F32>
hipError_t launch_typed(const GemmArgs& g, hipStream_t stream) {
  constexpr int UE = elem<T>::per16;
  const bool aligned = (reinterpret_cast<uintptr_t>(g.A) % 16 == 0) &&
                       (reinterpret_cast<uintptr_t>(g.B) % 16 == 0);
  const bool vec = aligned && g.lda % UE == 0 && g.ldb % UE == 0 && g.Kred % UE == 0 &&
                   g.sA0 % UE == 0 && g.sA1 % UE == 0 && g.sB0 % UE == 0 && g.sB1 % UE == 0;
  // Small M (filters per group) gets the 64-row tile so fewer MFMA rows idle.
  if (g.b_kmajor) {
    if (g.M <= 64) return launch_tile<T, 64, 128, OUT_F32, true>(g, vec, stream);
    return launch_tile<T, 128, 128, OUT_F32, true>(g, vec, stream);
  }
  if (g.M <= 64) return launch_tile<T, 64, 128, OUT_F32, false>(g, vec, stream);
  return launch_tile<T, 128, 128, OUT_F32, false>(g, vec, stream);
}

}  // namespace

hipError_t launch_gemm_nt(int dtype, const GemmArgs& g, hipStream_t stream) {
  if (dtype == DT_F32) {
    return g.out_f32 ? launch_typed<float, true>(g, stream) : launch_typed<float, false>(g, stream);
  }
  return g.out_f32 ? launch_typed<bf16_t, true>(g, stream) : launch_typed<bf16_t, false>(g, stream);
}

}  // namespace convsel
