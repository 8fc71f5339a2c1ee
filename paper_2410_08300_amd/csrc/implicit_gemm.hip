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
  int splits;         // workgroups sharing one output tile along the channels
  int chunks_per_split;
  float* partial;     // splits > 1: fp32 partial sums, [split][N][K][P][Q]
};

// Virtual row of the first filter row for pixel j.
__device__ __forceinline__ int vrow_of(int j, const IgArgs& a) {
  const int PQ = a.P * a.Q;
  const int n = j / PQ, pq = j - n * PQ;
  return n * a.Hv + (pq / a.Q) * a.sh;
}

// Halo items per thread whose global offsets are computed once per
// workgroup and whose data are prefetched into registers; items beyond
// kImax * 256 (very wide images) are staged on the fly.
constexpr int kImax = 4;

template <typename T, int BM, int NG, int RST>
__global__ __launch_bounds__(kThreads) void implicit_gemm_kernel(IgArgs a) {
  constexpr int UE = elem<T>::per16;
  constexpr int Cc = UE * NG;
  constexpr int MI = BM / 64, NJ = BN / 64;
  static_assert(BM * NG <= kThreads, "one filter item per thread");
  extern __shared__ __align__(16) vec16 smem[];
  vec16* As = smem;                         // [BM][UR]
  vec16* Xs = smem + BM * a.UR;             // [VR*Wv][PS]
  int* utab = reinterpret_cast<int*>(Xs + a.xs_units);  // runtime-tap path only

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int half = lane >> 5, l32 = lane & 31;
  const int j0 = blockIdx.x * BN;
  const int g = blockIdx.y / a.ktiles;
  const int k0 = (blockIdx.y - g * a.ktiles) * BM;
  const int RS = a.R * a.S;
  const int jl = min(j0 + BN, a.NPQ) - 1;
  const int vr_lo = vrow_of(j0, a);
  const int HW = a.H * a.W;

  if constexpr (RST == 0) {
    for (int u = tid; u < 2 * a.steps; u += kThreads) {
      int off = 0;
      if (u < a.units) {
        const int tap = u / NG, cg = u - tap * NG;
        const int r = tap / a.S, s = tap - r * a.S;
        off = (r * a.dh * a.Wv + s * a.dw) * a.PS + cg;
      }
      utab[u] = off;
    }
  }
  // The padding unit of an odd unit count holds zero filters (never rewritten).
  if (a.units & 1)
    for (int i = tid; i < BM; i += kThreads) As[i * a.UR + a.units] = vec16_zero();

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
  // Tap offsets in the halo (compile-time tap count only).
  int tapoff[RST > 0 ? RST : 1];
#pragma unroll
  for (int t = 0; t < (RST > 0 ? RST : 1); ++t) {
    const int r = t / a.S, s = t - r * a.S;
    tapoff[t] = (r * a.dh * a.Wv + s * a.dw) * a.PS;
  }

  const T* x = reinterpret_cast<const T*>(a.x);
  const T* w = reinterpret_cast<const T*>(a.w) + static_cast<int64_t>(g * a.Kg + k0) * a.Cg * RS;

  // Halo item it = pix * NG + cg, pix = vrow * Wv + vcol.  goff: element
  // offset of (image, row, column) in channel 0 of this group, or -1 where
  // the item reads padding (or does not exist).
  const int nitems = a.VR * a.Wv * NG;
  auto item_goff = [&](int it) -> int {
    if (it >= nitems) return -1;
    const int pix = it / NG;
    const int vr = pix / a.Wv, vc = pix - vr * a.Wv;
    const int v = vr_lo + vr;
    const int n = v / a.Hv;
    const int ih = v - n * a.Hv - a.ph, iw = vc - a.pw;
    if (n >= a.N || ih < 0 || ih >= a.H || iw < 0 || iw >= a.W) return -1;
    return (n * a.C + g * a.Cg) * HW + ih * a.W + iw;
  };
  // gaddr: always a valid element offset (padding items read element 0);
  // gvalid marks the items whose values are kept.
  int gaddr[kImax];
  bool gvalid[kImax];
#pragma unroll
  for (int t = 0; t < kImax; ++t) {
    const int go = item_goff(tid + t * kThreads);
    gvalid[t] = go >= 0;
    gaddr[t] = go >= 0 ? go : 0;
  }

  // Branch-free gather of UE channels at one halo position: every lane
  // loads from a valid address (element 0 stands in for padding and for
  // channels past the group) and zeroes those values afterwards, so all
  // loads are in flight together.
  auto load_item = [&](int go, int cg, int c0) -> vec16 {
    const int cb = c0 + cg * UE;
    uint32_t e[UE];
#pragma unroll
    for (int i = 0; i < UE; ++i) {
      const bool ok = go >= 0 && cb + i < a.Cg;
      const uint32_t bits = load_bits(x + (ok ? go + (cb + i) * HW : 0));
      e[i] = ok ? bits : 0u;
    }
    vec16 u;
    pack16<T>(u, e);
    return u;
  };

  // Register stage for the next chunk.  fetch() only issues loads into raw
  // registers; masking and packing wait until stash(), after the MFMAs of the
  // current chunk, so the load latency overlaps the matrix work.
  uint32_t xraw[kImax][UE];
  vec16 wr[RST > 0 ? RST : 1];
  const int wi = tid / NG, wcg = tid - (tid / NG) * NG;
  const bool w_item = tid < BM * NG;
  const bool w_row_ok = w_item && (k0 + wi < a.Kg);

  // Filter row of this thread's item, clamped into the group so that its
  // address is valid even for rows past Kg (their values are zeroed).
  const int wrow = w_item ? min(wi, a.Kg - k0 - 1) : 0;
  const T* wsrc = w + static_cast<int64_t>(wrow) * a.Cg * RS;

  // Loads only: every address is valid (channels clamped into the group), no
  // branches, so all of a thread's loads are in flight together.
  auto fetch = [&](int c0) {
#pragma unroll
    for (int t = 0; t < kImax; ++t) {
      const int cb = c0 + ((tid + t * kThreads) % NG) * UE;
#pragma unroll
      for (int i = 0; i < UE; ++i) xraw[t][i] = load_bits(x + gaddr[t] + min(cb + i, a.Cg - 1) * HW);
    }
    if constexpr (RST > 0) {
      const int cb = min(c0 + wcg * UE, a.Cg - UE);
#pragma unroll
      for (int m = 0; m < RST; ++m) wr[m] = load16(wsrc + static_cast<int64_t>(cb) * RS + m * UE);
    }
  };

  auto stash = [&](int c0) {
#pragma unroll
    for (int t = 0; t < kImax; ++t) {
      const int it = tid + t * kThreads;
      const int cb = c0 + (it % NG) * UE;
      uint32_t e[UE];
#pragma unroll
      for (int i = 0; i < UE; ++i) e[i] = (gvalid[t] && cb + i < a.Cg) ? xraw[t][i] : 0u;
      vec16 u;
      pack16<T>(u, e);
      if (it < nitems) Xs[(it / NG) * a.PS + it % NG] = u;
    }
    for (int it = tid + kImax * kThreads; it < nitems; it += kThreads)
      Xs[(it / NG) * a.PS + it % NG] = load_item(item_goff(it), it % NG, c0);
    if (w_item) {
      if constexpr (RST > 0) {
        // UE channels x RST taps arrive as RST 16-byte units in (channel,
        // tap) order; regroup them as RST units of UE channels per tap.
        const bool ok = w_row_ok && c0 + wcg * UE < a.Cg;
#pragma unroll
        for (int tap = 0; tap < RST; ++tap) {
          uint32_t e[UE];
#pragma unroll
          for (int i = 0; i < UE; ++i) {
            const int f = i * RST + tap;
            const uint32_t word = wr[f / UE].d[(f % UE) / (4 / elem<T>::bytes > 0 ? (4 / elem<T>::bytes) : 1)];
            const uint32_t bits = elem<T>::bytes == 2 ? ((f & 1) ? (word >> 16) : (word & 0xffffu)) : word;
            e[i] = ok ? bits : 0u;
          }
          vec16 u;
          pack16<T>(u, e);
          As[wi * a.UR + tap * NG + wcg] = u;
        }
      } else {
        const int cb = c0 + wcg * UE;
        const T* src = w + static_cast<int64_t>(wi) * a.Cg * RS + static_cast<int64_t>(cb) * RS;
        for (int tap = 0; tap < RS; ++tap) {
          vec16 u = vec16_zero();
          if (w_row_ok) {
#pragma unroll
            for (int e = 0; e < UE; ++e)
              if (cb + e < a.Cg) vec16_set<T>(u, e, src[e * RS + tap]);
          }
          As[wi * a.UR + tap * NG + wcg] = u;
        }
      }
    }
  };

  f32x16_t acc[MI][NJ];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int nj = 0; nj < NJ; ++nj) acc[mi][nj] = zero16();

  const int arow = (wm * (BM / 2) + l32) * a.UR;
  auto mfma_step = [&](int u, int xo) {
    vec16 af[MI], bfr[NJ];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) af[mi] = As[arow + mi * 32 * a.UR + u];
#pragma unroll
    for (int nj = 0; nj < NJ; ++nj) bfr[nj] = Xs[pofs[nj] + xo];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int nj = 0; nj < NJ; ++nj) mfma_32x32<T>(acc[mi][nj], af[mi], bfr[nj]);
  };

  // This workgroup's channel range (all channels unless split along them).
  const int split = blockIdx.z;
  const int c_begin = split * a.chunks_per_split * Cc;
  const int c_end = min(a.Cg, c_begin + a.chunks_per_split * Cc);

  fetch(c_begin);
  stash(c_begin);
  __syncthreads();
  for (int c0 = c_begin; c0 < c_end; c0 += Cc) {
    const bool more = c0 + Cc < c_end;
    fetch(more ? c0 + Cc : c0);  // the last chunk's refetch is never stashed
    // Keep the prefetch loads ahead of the MFMAs (the scheduler would
    // otherwise sink them to the end of the chunk, exposing their latency).
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (RST > 0) {
      constexpr int STEPS = (RST * NG + 1) / 2;
#pragma unroll
      for (int st = 0; st < STEPS; ++st) {
        int xo;
        if constexpr (NG == 2) {
          xo = tapoff[st] + half;                      // units 2st, 2st+1: tap st, group = half
        } else {
          const int t0 = 2 * st, t1 = 2 * st + 1 < RST ? 2 * st + 1 : RST - 1;
          xo = half ? tapoff[t1] : tapoff[t0];         // units 2st, 2st+1: taps 2st, 2st+1
        }
        mfma_step(2 * st + half, xo);
      }
    } else {
      for (int st = 0; st < a.steps; ++st) {
        const int u = 2 * st + half;
        mfma_step(u, utab[u]);
      }
    }
    __syncthreads();
    if (more) {
      stash(c0 + Cc);
      __syncthreads();
    }
  }

  // ---- epilogue: bias, ReLU, NCHW store ----
  const int64_t PQ = static_cast<int64_t>(a.P) * a.Q;
  if (a.splits > 1) {
    // Raw fp32 partial sums; the reduce kernel adds the splits, the bias and
    // the ReLU, and rounds to the output type.
    float* part = a.partial + static_cast<int64_t>(split) * a.N * a.K * PQ;
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int i = k0 + wm * (BM / 2) + mi * 32 + mfma_row(v, lane);
        if (i >= a.Kg) continue;
        const int k = g * a.Kg + i;
#pragma unroll
        for (int nj = 0; nj < NJ; ++nj)
          if (jvalid[nj]) part[ybase[nj] + k * PQ] = acc[mi][nj][v];
      }
    }
    return;
  }
  const T* bias = reinterpret_cast<const T*>(a.b);
  T* y = reinterpret_cast<T*>(a.y);
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

// Sum of the split partials, plus bias, ReLU, rounding to the output type;
// four consecutive outputs per thread.
template <typename T>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part, const T* __restrict__ bias,
                                                            T* __restrict__ y, int64_t total, int64_t PQ, int K,
                                                            int splits, int relu) {
  const int64_t i0 = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 4;
  if (i0 >= total) return;
  const int n4 = total - i0 < 4 ? static_cast<int>(total - i0) : 4;
  float sum[4] = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < splits; ++s) {
    const float* p = part + s * total + i0;
    if (n4 == 4 && (reinterpret_cast<uintptr_t>(p) & 15) == 0) {
      const float4 v = *reinterpret_cast<const float4*>(p);
      sum[0] += v.x; sum[1] += v.y; sum[2] += v.z; sum[3] += v.w;
    } else {
      for (int e = 0; e < n4; ++e) sum[e] += p[e];
    }
  }
  for (int e = 0; e < n4; ++e) {
    const int64_t i = i0 + e;
    float v = sum[e];
    if (bias) v += elem<T>::load(bias + static_cast<int>((i / PQ) % K));
    if (relu) v = fmaxf(v, 0.f);
    elem<T>::store(y + i, v);
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

// Split the channel chunks over several workgroups when the output tiles
// alone leave CUs idle: pick the split count S (1..8, at least two chunks per
// split) that minimises the number of full waves of 256 CUs per unit of work,
// ceil(tiles*S / 256) / S, plus a small charge per extra split for the
// partial-sum traffic.
constexpr int kCUs = 256;

void choose_splits(const Shape& s, IgPlan& pl, int Cc) {
  IgArgs& a = pl.a;
  const int64_t tiles = (int64_t)((a.NPQ + BN - 1) / BN) * a.ktiles * s.G;
  const int nch = (int)((s.Cg + Cc - 1) / Cc);
  int best = 1;
  double best_cost = 1e30;
  if (tiles < kCUs) {
    for (int S = 1; S <= 8 && S <= (nch + 1) / 2; ++S) {
      const double waves = (double)((tiles * S + kCUs - 1) / kCUs) / S;
      const double cost = waves + 0.05 * (S - 1);
      if (cost < best_cost - 1e-9) {
        best_cost = cost;
        best = S;
      }
    }
  }
  a.chunks_per_split = (nch + best - 1) / best;
  a.splits = (nch + a.chunks_per_split - 1) / a.chunks_per_split;
}

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
        choose_splits(s, pl, UE * ng);
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
  const dim3 grid((pl.a.NPQ + BN - 1) / BN, pl.a.ktiles * (pl.a.K / pl.a.Kg), pl.a.splits);
  hipLaunchKernelGGL(kern, grid, dim3(kThreads), pl.lds, stream, pl.a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || pl.a.splits == 1) return e;
  const int64_t total = (int64_t)pl.a.N * pl.a.K * pl.a.P * pl.a.Q;
  const int64_t blocks = (total + 1023) / 1024;
  hipLaunchKernelGGL(splitk_reduce_kernel<T>, dim3((unsigned)blocks), dim3(256), 0, stream, pl.a.partial,
                     reinterpret_cast<const T*>(pl.a.b), reinterpret_cast<T*>(pl.a.y), total,
                     (int64_t)pl.a.P * pl.a.Q, pl.a.K, pl.a.splits, pl.a.relu);
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
hipError_t launch_typed(const Shape& s, const void* x, const void* w, const void* b, void* y, void* ws,
                        hipStream_t stream) {
  IgPlan pl;
  if (!make_plan<T>(s, w, pl)) return hipErrorInvalidValue;
  pl.a.x = x; pl.a.w = w; pl.a.b = b; pl.a.y = y;
  pl.a.partial = reinterpret_cast<float*>(ws);
  if (pl.a.splits > 1 && !ws) return hipErrorInvalidValue;
  if (pl.BM == 64) return pl.NG == 2 ? launch_rst<T, 64, 2>(pl, stream) : launch_rst<T, 64, 1>(pl, stream);
  return pl.NG == 2 ? launch_rst<T, 128, 2>(pl, stream) : launch_rst<T, 128, 1>(pl, stream);
}

}  // namespace

bool implicit_gemm_fits(const Shape& s) {
  IgPlan pl;
  if (s.dtype == DT_F32) return make_plan<float>(s, nullptr, pl);
  return make_plan<bf16_t>(s, nullptr, pl);
}

size_t implicit_gemm_workspace(const Shape& s) {
  IgPlan pl;
  const bool ok = s.dtype == DT_F32 ? make_plan<float>(s, nullptr, pl) : make_plan<bf16_t>(s, nullptr, pl);
  if (!ok || pl.a.splits <= 1) return 0;
  return (size_t)pl.a.splits * s.N * s.K * s.P * s.Q * sizeof(float);
}

hipError_t launch_implicit_gemm(const Shape& s, const void* x, const void* w, const void* b, void* y, void* ws,
                                hipStream_t stream) {
  if (s.dtype == DT_F32) return launch_typed<float>(s, x, w, b, y, ws, stream);
  return launch_typed<bf16_t>(s, x, w, b, y, ws, stream);
}

}  // namespace convsel
