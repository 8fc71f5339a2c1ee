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
#include "igemm_common.hpp"
#include "kernels.hpp"

namespace convsel {

namespace {

using namespace igemm;

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

// ---------------------------------------------------------------------------
// bf16 "NT" GEMM through LDS DMA (both operands reduction-contiguous, 16-byte
// aligned rows, Kred a multiple of 8).  The MFMA's A operand is a row of B
// (a pixel of IM2COL's column matrix, a Winograd tile) and its B operand a
// row of A (a filter), so each lane ends with four consecutive j of one i:
// the output row's order.
//
// A workgroup (4 waves, WJ x WI) owns TJ rows of B x TI rows of A and walks
// the reduction in k-tiles of 64.  A k-tile stage is the TJ + TI rows of 128
// bytes, two rows per 256-byte line with the 16-byte unit u of row r at
// position 8 (r & 1) + (u ^ ((r >> 1) & 7)) of line r >> 1, so 16 lanes
// reading one unit of 16 consecutive rows hit 16 distinct bank groups.  The
// stage is filled by `buffer_load ... lds` (no register round trip): DMA
// instruction J writes the stage's 16-byte units J*64 .. J*64+63, and each
// lane fetches the unit that the layout puts at its place (rows past the
// operand and reduction elements past Kred read zeros through the buffer
// range).  NST stages form a ring with NST - 1 k-tiles in flight and one
// barrier per k-tile.
template <int TJ, int TI, int WJ_>
struct GemmDmaShape {
  static constexpr int WJ = WJ_;
  static constexpr int WI = 4 / WJ;
  static constexpr int MJ = TJ / WJ / 32, NI = TI / WI / 32;  // 32 x 32 blocks per wave
  static constexpr int ROWS = TJ + TI;
  static constexpr int STAGE = ROWS * 128;
  static constexpr int NST = 3 * STAGE <= 96 * 1024 ? 4 : 3;
  static constexpr int NDMA = ROWS / 8 / 4;  // DMA instructions per wave and stage
  static_assert(WJ * WI == 4 && MJ >= 1 && NI >= 1 && TJ % 32 == 0 && TI % 32 == 0 && ROWS % 32 == 0, "tile");
  static_assert(NST * STAGE <= 160 * 1024 && NDMA * (NST - 1) <= 63, "stages");
};

template <int TJ, int TI, int WJ, bool OUT_F32>
__global__ __launch_bounds__(256) void gemm_dma_kernel(GemmArgs g, int batch_base, uint32_t a_bytes,
                                                       uint32_t b_bytes) {
  using Sh = GemmDmaShape<TJ, TI, WJ>;
  constexpr int MJ = Sh::MJ, NI = Sh::NI, NST = Sh::NST, NDMA = Sh::NDMA, STAGE = Sh::STAGE;
  extern __shared__ __align__(16) vec16 smem[];
  char* lds = reinterpret_cast<char*>(smem);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wj = wave % Sh::WJ, wi = wave / Sh::WJ;
  const int j0 = blockIdx.x * TJ, i0 = blockIdx.y * TI;
  const int b = batch_base + blockIdx.z;
  const int b0 = b / g.bdiv, b1 = b - b0 * g.bdiv;
  const bf16_t* A = reinterpret_cast<const bf16_t*>(g.A) + b0 * g.sA0 + b1 * g.sA1;
  const bf16_t* B = reinterpret_cast<const bf16_t*>(g.B) + b0 * g.sB0 + b1 * g.sB1;
  const __amdgpu_buffer_rsrc_t ar = make_rsrc(A, a_bytes);
  const __amdgpu_buffer_rsrc_t br = make_rsrc(B, b_bytes);

  // This wave's DMA instructions: J = wave * NDMA + d.  Instructions below
  // TJ / 8 fill rows of B, the rest rows of A (a row boundary never falls
  // inside one: 64 units are 8 whole rows).
  uint32_t dvo[NDMA];
  int dku[NDMA];
#pragma unroll
  for (int d = 0; d < NDMA; ++d) {
    const int U = (wave * NDMA + d) * 64 + lane;
    const int line = U >> 4, pos = U & 15;
    const int row = 2 * line + (pos >> 3), u = (pos & 7) ^ (line & 7);
    const bool isb = row < TJ;
    const int grow = isb ? j0 + row : i0 + row - TJ;
    const bool ok = grow < (isb ? g.N : g.M);
    const int64_t ld = isb ? g.ldb : g.lda;
    dvo[d] = ok ? static_cast<uint32_t>((grow * ld + u * 8) * 2) : (isb ? b_bytes : a_bytes);
    dku[d] = u * 8;
  }
  const int nk = (g.Kred + 63) / 64;
  auto issue = [&](int kt) {
    char __attribute__((address_space(3)))* st =
        (char __attribute__((address_space(3)))*)(lds + (kt % NST) * STAGE);
    const uint32_t so = static_cast<uint32_t>(kt) * 128;
    const bool tail = (kt + 1) * 64 > g.Kred;
#pragma unroll
    for (int d = 0; d < NDMA; ++d) {
      const int J = wave * NDMA + d;
      const bool isb = J < TJ / 8;
      const uint32_t vo = (!tail || kt * 64 + dku[d] < g.Kred) ? dvo[d] : (isb ? b_bytes : a_bytes);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(isb ? br : ar, (lds_void_t*)(st + J * 1024), 16, vo, so, 0, 0);
    }
  };

  // Fragment offsets within a stage: unit 2 t + half of row r.
  const int half = lane >> 5, l32 = lane & 31;
  auto frag = [&](int r, int u) { return (r >> 1) * 256 + ((8 * (r & 1) + (u ^ ((r >> 1) & 7))) << 4); };
  int aoff[MJ][4], boff[NI][4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
#pragma unroll
    for (int mj = 0; mj < MJ; ++mj) aoff[mj][t] = frag((wj * MJ + mj) * 32 + l32, 2 * t + half);
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) boff[ni][t] = frag(TJ + (wi * NI + ni) * 32 + l32, 2 * t + half);
  }

  f32x16_t acc[MJ][NI];
#pragma unroll
  for (int mj = 0; mj < MJ; ++mj)
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) acc[mj][ni] = zero16();

#pragma unroll
  for (int p = 0; p < NST - 1; ++p)
    if (p < nk) issue(p);
  for (int kt = 0; kt < nk; ++kt) {
    // k-tile kt has landed once at most the later tiles' DMAs are pending.
    const int later = min(nk - 1, kt + NST - 2) - kt;
    if (later >= 2 && NST == 4) CONVSEL_WAIT_VMCNT(2 * NDMA);
    else if (later >= 1) CONVSEL_WAIT_VMCNT(NDMA);
    else CONVSEL_WAIT_VMCNT(0);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();  // every wave's part of tile kt is in; every wave is done with tile kt - 1
    asm volatile("" ::: "memory");
    if (kt + NST - 1 < nk) issue(kt + NST - 1);  // into the stage of tile kt - 1
    const char* st = lds + (kt % NST) * STAGE;
    bf16x8_t fa[2][MJ], fb[2][NI];
    auto read = [&](auto t_c) {
      constexpr int t = decltype(t_c)::value;
#pragma unroll
      for (int mj = 0; mj < MJ; ++mj) fa[t & 1][mj] = *reinterpret_cast<const bf16x8_t*>(st + aoff[mj][t]);
#pragma unroll
      for (int ni = 0; ni < NI; ++ni) fb[t & 1][ni] = *reinterpret_cast<const bf16x8_t*>(st + boff[ni][t]);
    };
    read(std::integral_constant<int, 0>{});
    static_for<4>([&](auto t_c) {
      constexpr int t = decltype(t_c)::value;
      if constexpr (t + 1 < 4) read(std::integral_constant<int, t + 1>{});
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int mj = 0; mj < MJ; ++mj)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
          acc[mj][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[t & 1][mj], fb[t & 1][ni], acc[mj][ni], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    });
  }

  // Epilogue: bias (per i), ReLU, four consecutive j per store.
  const int64_t cofs = b0 * g.sC0 + b1 * g.sC1;
  const bf16_t* bias = g.bias ? reinterpret_cast<const bf16_t*>(g.bias) + b1 * g.sBias1 : nullptr;
  const bool vst = ((cofs | g.ldc | g.sCj) & 3) == 0 && (g.jspan == 0 || g.jspan % 4 == 0) &&
                   reinterpret_cast<uintptr_t>(g.C) % 16 == 0;
  // Offset of column j in C (a folded batch maps j to its item's columns).
  auto col = [&](int j) -> int64_t {
    if (g.jspan == 0) return j;
    const int n = j / g.jspan;
    return n * g.sCj + (j - n * g.jspan);
  };
#pragma unroll
  for (int ni = 0; ni < NI; ++ni) {
    const int i = i0 + (wi * NI + ni) * 32 + l32;
    if (i >= g.M) continue;
    const float bv = bias ? elem<bf16_t>::load(bias + i) : 0.f;
    const int64_t row = cofs + static_cast<int64_t>(i) * g.ldc;
#pragma unroll
    for (int mj = 0; mj < MJ; ++mj) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int j = j0 + (wj * MJ + mj) * 32 + 8 * q + 4 * half;
        float v[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          v[t] = acc[mj][ni][4 * q + t] + bv;
          if (g.relu) v[t] = fmaxf(v[t], 0.f);
        }
        if (OUT_F32) {
          float* c = reinterpret_cast<float*>(g.C) + row;
          if (vst && j + 4 <= g.N) {
            *reinterpret_cast<float4*>(c + col(j)) = make_float4(v[0], v[1], v[2], v[3]);
          } else {
#pragma unroll
            for (int t = 0; t < 4; ++t)
              if (j + t < g.N) c[col(j + t)] = v[t];
          }
        } else {
          uint16_t* c = reinterpret_cast<uint16_t*>(g.C) + row;
          if (vst && j + 4 <= g.N) {
            *reinterpret_cast<uint2*>(c + col(j)) =
                make_uint2(f32x2_to_bf16x2(v[0], v[1]), f32x2_to_bf16x2(v[2], v[3]));
          } else {
#pragma unroll
            for (int t = 0; t < 4; ++t)
              if (j + t < g.N) c[col(j + t)] = f32_to_bf16(v[t]);
          }
        }
      }
    }
  }
}

template <int TJ, int TI, int WJ, bool OUT_F32>
hipError_t launch_dma_tile(const GemmArgs& g, uint32_t a_bytes, uint32_t b_bytes, hipStream_t stream) {
  using Sh = GemmDmaShape<TJ, TI, WJ>;
  const auto kern = gemm_dma_kernel<TJ, TI, WJ, OUT_F32>;
  const size_t lds = (size_t)Sh::NST * Sh::STAGE;
  static bool attr = false;
  if (!attr) {
    const hipError_t e =
        hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr = true;
  }
  for (int base = 0; base < g.batch; base += 65535) {
    const int nb = g.batch - base < 65535 ? g.batch - base : 65535;
    const dim3 grid((g.N + TJ - 1) / TJ, (g.M + TI - 1) / TI, nb);
    hipLaunchKernelGGL(kern, grid, dim3(256), lds, stream, g, base, a_bytes, b_bytes);
  }
  return hipGetLastError();
}

// The DMA kernel serves bf16 operands whose rows are 16-byte aligned and
// whose per-batch extents fit a buffer range.
bool gemm_dma_ok(const GemmArgs& g, uint32_t& a_bytes, uint32_t& b_bytes) {
  if (g.b_kmajor || g.Kred % 8 != 0 || g.lda % 8 != 0 || g.ldb % 8 != 0) return false;
  if (g.sA0 % 8 != 0 || g.sA1 % 8 != 0 || g.sB0 % 8 != 0 || g.sB1 % 8 != 0) return false;
  if (reinterpret_cast<uintptr_t>(g.A) % 16 != 0 || reinterpret_cast<uintptr_t>(g.B) % 16 != 0) return false;
  if (g.M <= 0 || g.N <= 0 || g.Kred <= 0) return false;
  const int64_t ab = ((int64_t)(g.M - 1) * g.lda + g.Kred) * 2, bb = ((int64_t)(g.N - 1) * g.ldb + g.Kred) * 2;
  if (ab >= ((int64_t)1 << 31) || bb >= ((int64_t)1 << 31)) return false;
  a_bytes = (uint32_t)ab;
  b_bytes = (uint32_t)bb;
  return true;
}

// Tile (TJ x TI) choice: the largest tile whose grid fills the CUs, with TI
// no wider than M needs; small problems take the 64 x 64 tile.
template <bool OUT_F32>
hipError_t launch_dma(const GemmArgs& g, uint32_t a_bytes, uint32_t b_bytes, hipStream_t stream) {
  auto wgs = [&](int tj, int ti) { return (int64_t)((g.N + tj - 1) / tj) * ((g.M + ti - 1) / ti) * g.batch; };
  const int mr = (g.M + 63) / 64 * 64;
  if (mr >= 256 && wgs(128, 256) >= 240) return launch_dma_tile<128, 256, 1, OUT_F32>(g, a_bytes, b_bytes, stream);
  if (mr >= 128 && wgs(128, 128) >= 240) return launch_dma_tile<128, 128, 2, OUT_F32>(g, a_bytes, b_bytes, stream);
  if (wgs(256, 64) >= 240) return launch_dma_tile<256, 64, 4, OUT_F32>(g, a_bytes, b_bytes, stream);
  if (wgs(128, 64) >= 240) return launch_dma_tile<128, 64, 2, OUT_F32>(g, a_bytes, b_bytes, stream);
  return launch_dma_tile<64, 64, 2, OUT_F32>(g, a_bytes, b_bytes, stream);
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
  uint32_t ab = 0, bb = 0;
  // A batch that shares A and whose B items are consecutive rows is folded
  // into N when the items are narrow (IM2COL's small planes), so that the
  // tiles are full and the grid holds enough workgroups.
  GemmArgs f = g;
  if (g.batch > 1 && g.bdiv == 1 && g.sA0 == 0 && g.sB0 == (int64_t)g.N * g.ldb && g.N < 1024 &&
      (int64_t)g.N * g.batch < ((int64_t)1 << 31)) {
    f.jspan = g.N;
    f.sCj = g.sC0;
    f.N = g.N * g.batch;
    f.batch = 1;
    f.sB0 = f.sC0 = 0;
  }
  if (gemm_dma_ok(f, ab, bb)) return f.out_f32 ? launch_dma<true>(f, ab, bb, stream) : launch_dma<false>(f, ab, bb, stream);
  return g.out_f32 ? launch_typed<bf16_t, true>(g, stream) : launch_typed<bf16_t, false>(g, stream);
}

}  // namespace convsel
