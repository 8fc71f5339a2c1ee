// Implicit GEMM (paper, Sec. V-B item (b)): the convolution as the product
//   Y[k][pixel] = sum_{(c,r,s)} Wt[k][(c,r,s)] * X[(c,r,s)][pixel]
// without ever forming the column matrix X.  On MFMA: D (output channels x
// pixels) accumulates 32 x 32 blocks in fp32.
//
// Pixels are the flattened (n, p, q) output positions; a workgroup owns BN =
// 128 consecutive pixels and BM (64 or 128) output channels of one group.  The
// reduction is walked in chunks of Cc input channels (Cc = 8*NG bf16 or
// 4*NG fp32, i.e. NG 16-byte units per pixel):
//
//  * Filters are first repacked (one small kernel per call) into
//        Wp[group][chunk][k (padded to BM)][tap][NG units of UE channels]
//    with zeros in the padding, so one chunk's filter tile of a workgroup is
//    a single contiguous block, staged in LDS as As[i][tap*NG + cg] by plain
//    16-byte copies.
//  * Input halo.  The input is viewed as a stack of zero-padded images in
//    "virtual rows": pixel (n, p) with filter row r reads virtual row
//    n*Hv + p*sh + r*dh, Hv = (P-1)*sh + (R-1)*dh + 1, and virtual column
//    q*sw + s*dw (real row = virtual row mod Hv - pad_h, real column =
//    virtual column - pad_w).  The workgroup's pixels read one contiguous
//    range of VR virtual rows, each Wv columns wide, staged once per chunk
//    with the channels innermost:  Xs[(vrow * Wv + vcol) * PS + cg], so
//    every filter tap of every pixel is one 16-byte LDS read and each input
//    element is fetched once per chunk instead of R*S times.
//  * Loads are AMD buffer loads: the per-lane offset of a halo element is
//    fixed for the whole kernel, the channel offset is a scalar, and reads
//    outside the buffer return zero -- padding and channels past the group
//    are mapped there, so no lane needs a select or a branch.
//  * The next chunk is fetched into registers while the MFMAs of the current
//    one run; one reduction step consumes two 16-byte units per lane (the
//    two halves of the wave take units 2*step and 2*step+1: 16 bf16 or 8 fp32
//    reduction terms); a padding unit (odd unit count) has zero filters.
//  * Layers whose output tiles leave CUs idle split the chunks over several
//    workgroups (fp32 partial sums, then a reduce kernel).
//
// Row strides in LDS (UR and PS units of 16 bytes) are odd, so the 16-byte
// reads of 32 consecutive rows / pixels map to distinct bank groups; stores
// are arranged so that consecutive lanes write consecutive or odd-strided
// units.
#include <atomic>
#include <stdio.h>
#include <string>

#include "common.hpp"
#include "kernels.hpp"

namespace convsel {

namespace {

constexpr int kThreads = 256;
constexpr int BN = 128;
constexpr uint32_t kRsrcWord3 = 0x00020000u;  // raw buffer, 32-bit data format (gfx9 family)

typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

struct IgArgs {
  const void* x;       // first image of this launch
  const void* wp;      // packed filters
  const void* b;
  void* y;             // first image of this launch
  uint32_t x_bytes;    // extent of the input buffer of this launch
  uint32_t wp_bytes;
  int N, C, H, W, K, R, S, P, Q;
  int sh, sw, ph, pw, dh, dw;
  int Cg, Kg, G, relu;
  int Hv, Wv, VR;      // virtual rows per image, halo width, halo rows
  int NPQ;
  int units;           // R*S*NG: 16-byte units per filter row and chunk
  int steps;           // ceil(units / 2)
  int UR;              // filter row stride in 16-byte units (odd)
  int PS;              // halo pixel stride in 16-byte units (odd)
  int ktiles;          // ceil(Kg / BM)
  int Kpad;            // ktiles * BM
  int nch;             // channel chunks per group
  int xs_units;        // VR * Wv * PS
  int splits;          // workgroups sharing one output tile along the channels
  int chunks_per_split;
  float* partial;      // splits > 1: fp32 partial sums, [split][N][K][P][Q]
  int slab;            // floats per split of `partial` (N*K*P*Q rounded up to 4)
  int vec_out;         // P*Q % 8 == 0 and y 16-byte aligned: staged 16-byte stores
};

// Virtual row of the first filter row for pixel j.
__device__ __forceinline__ int vrow_of(int j, const IgArgs& a) {
  const int PQ = a.P * a.Q;
  const int n = j / PQ, pq = j - n * PQ;
  return n * a.Hv + (pq / a.Q) * a.sh;
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, (int)kRsrcWord3);
}

__device__ __forceinline__ uint32_t buf_load_elem(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, float*) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0);
}
__device__ __forceinline__ uint32_t buf_load_elem(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, bf16_t*) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0);
}
__device__ __forceinline__ vec16 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
  vec16 o;
  o.d[0] = v[0];
  o.d[1] = v[1];
  o.d[2] = v[2];
  o.d[3] = v[3];
  return o;
}

// Halo items per thread kept in registers (offsets computed once, data
// prefetched one chunk ahead); items beyond kImax * 256 (very wide images)
// are loaded when stashed.
constexpr int kImax = 4;
// Filter units per thread prefetched for compile-time tap counts.
template <int RST, int BM, int NG>
struct WUnits {
  static constexpr int value = RST > 0 ? (BM * RST * NG + kThreads - 1) / kThreads : 1;
};

template <typename T, int BM, int NG, int RST>
__global__ __launch_bounds__(kThreads) void implicit_gemm_kernel(IgArgs a) {
  constexpr int UE = elem<T>::per16;
  constexpr int ES = elem<T>::bytes;
  constexpr int MI = BM / 64, NJ = BN / 64;
  constexpr int WU = WUnits<RST, BM, NG>::value;
  extern __shared__ __align__(16) vec16 smem[];
  vec16* As = smem;                         // [BM][UR]
  vec16* Xs = smem + BM * a.UR;             // [VR*Wv][PS]
  int* utab = reinterpret_cast<int*>(Xs + a.xs_units);  // runtime-tap path only

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int half = lane >> 5, l32 = lane & 31;
  const int j0 = blockIdx.x * BN;
  const int g = blockIdx.y / a.ktiles;
  const int kt = blockIdx.y - g * a.ktiles;
  const int k0 = kt * BM;
  const int jl = min(j0 + BN, a.NPQ) - 1;
  const int vr_lo = vrow_of(j0, a);
  const int HW = a.H * a.W;
  const int units = a.units;

  const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, a.x_bytes);
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(a.wp, a.wp_bytes);

  if constexpr (RST == 0) {
    for (int u = tid; u < 2 * a.steps; u += kThreads) {
      int off = 0;
      if (u < units) {
        const int tap = u / NG, cg = u - tap * NG;
        const int r = tap / a.S, s = tap - r * a.S;
        off = (r * a.dh * a.Wv + s * a.dw) * a.PS + cg;
      }
      utab[u] = off;
    }
  }
  // The padding unit of an odd unit count holds zero filters (never rewritten).
  if (units & 1)
    for (int i = tid; i < BM; i += kThreads) As[i * a.UR + units] = vec16_zero();

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

  // Halo item it = cg * (VR*Wv) + pix, pix = vrow * Wv + vcol: consecutive
  // lanes take consecutive pixels of one channel group (coalesced global
  // reads; LDS stores at the odd stride PS).  Item offset: bytes to channel 0
  // of the group at that position, or x_bytes (out of range: reads zero) for
  // padding and missing items.
  const int npix = a.VR * a.Wv;
  const int nitems = npix * NG;
  auto item_off = [&](int it) -> uint32_t {
    if (it >= nitems) return a.x_bytes;
    const int cg = it / npix, pix = it - cg * npix;
    const int vr = pix / a.Wv, vc = pix - vr * a.Wv;
    const int v = vr_lo + vr;
    const int n = v / a.Hv;
    const int ih = v - n * a.Hv - a.ph, iw = vc - a.pw;
    if (n >= a.N || ih < 0 || ih >= a.H || iw < 0 || iw >= a.W) return a.x_bytes;
    return static_cast<uint32_t>(((n * a.C + g * a.Cg + cg * UE) * HW + ih * a.W + iw) * ES);
  };
  auto item_lds = [&](int it) -> int {
    const int cg = it / npix, pix = it - cg * npix;
    return pix * a.PS + cg;
  };
  uint32_t xoff[kImax];
  int xlds[kImax];
#pragma unroll
  for (int t = 0; t < kImax; ++t) {
    const int it = tid + t * kThreads;
    xoff[t] = item_off(it);
    xlds[t] = it < nitems ? item_lds(it) : -1;
  }
  // Element e of the unit loaded for chunk offset c0: scalar (wave-uniform)
  // channel offset c0 + e; in the tail chunk, where the unit may run past the
  // group's channels, lanes past it use the out-of-range offset (zero).
  auto load_unit_elem = [&](uint32_t voff, int cgb, int c0, int e) -> uint32_t {
    const uint32_t so = static_cast<uint32_t>((c0 + e) * HW * ES);
    const bool tail = c0 + UE * NG > a.Cg;  // uniform
    const uint32_t vo = (tail && cgb + c0 + e >= a.Cg) ? a.x_bytes : voff;
    return buf_load_elem(xr, vo, so, (T*)nullptr);
  };

  // Filter units of this workgroup's tile: unit f = i*units + u.
  uint32_t wvoff[WU];
  int wlds[WU];
#pragma unroll
  for (int t = 0; t < WU; ++t) {
    const int f = tid + t * kThreads;
    const bool ok = f < BM * units;
    const int i = ok ? f / units : 0, u = ok ? f - (f / units) * units : 0;
    wvoff[t] = ok ? static_cast<uint32_t>(f * 16) : a.wp_bytes;
    wlds[t] = ok ? i * a.UR + u : -1;
  }
  // Packed-filter byte offset of chunk ch of this tile.
  auto wtile_soff = [&](int ch) -> uint32_t {
    return static_cast<uint32_t>((static_cast<int64_t>(g * a.nch + ch) * a.Kpad + k0) * units * 16);
  };

  // Register stage for the next chunk.
  uint32_t xraw[kImax][UE];
  vec16 wreg[WU];

  auto fetch = [&](int ch) {
    const int c0 = ch * UE * NG;
#pragma unroll
    for (int t = 0; t < kImax; ++t) {
      const int cgb = ((tid + t * kThreads) / npix) * UE;
#pragma unroll
      for (int e = 0; e < UE; ++e) xraw[t][e] = load_unit_elem(xoff[t], cgb, c0, e);
    }
    if constexpr (RST > 0) {
      const uint32_t so = wtile_soff(ch);
#pragma unroll
      for (int t = 0; t < WU; ++t) wreg[t] = buf_load16(wr, wvoff[t], so);
    }
  };

  auto stash = [&](int ch) {
#pragma unroll
    for (int t = 0; t < kImax; ++t) {
      vec16 u;
      pack16<T>(u, xraw[t]);
      if (xlds[t] >= 0) Xs[xlds[t]] = u;
    }
    if (nitems > kImax * kThreads) {
      const int c0 = ch * UE * NG;
      for (int it = tid + kImax * kThreads; it < nitems; it += kThreads) {
        const uint32_t off = item_off(it);
        const int cgb = (it / npix) * UE;
        uint32_t e[UE];
#pragma unroll
        for (int i = 0; i < UE; ++i) e[i] = load_unit_elem(off, cgb, c0, i);
        vec16 u;
        pack16<T>(u, e);
        Xs[item_lds(it)] = u;
      }
    }
    if constexpr (RST > 0) {
#pragma unroll
      for (int t = 0; t < WU; ++t)
        if (wlds[t] >= 0) As[wlds[t]] = wreg[t];
    } else {
      const uint32_t so = wtile_soff(ch);
      for (int f = tid; f < BM * units; f += kThreads)
        As[(f / units) * a.UR + f % units] = buf_load16(wr, static_cast<uint32_t>(f * 16), so);
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

  // This workgroup's chunk range (all chunks unless split along them).
  const int split = blockIdx.z;
  const int ch_begin = split * a.chunks_per_split;
  const int ch_end = min(a.nch, ch_begin + a.chunks_per_split);

  fetch(ch_begin);
  stash(ch_begin);
  __syncthreads();
  for (int ch = ch_begin; ch < ch_end; ++ch) {
    const bool more = ch + 1 < ch_end;
    fetch(more ? ch + 1 : ch);  // the last chunk's refetch is never stashed
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
      stash(ch + 1);
      __syncthreads();
    }
  }

  // ---- epilogue: bias, ReLU, NCHW store ----
  // With P*Q a multiple of 8, every aligned run of 8 tile pixels lies in one
  // image and starts 16-byte aligned in y, so the accumulators go through
  // LDS (the chunk buffers are free now) and leave as 16-byte stores of 8
  // consecutive pixels of one channel.  Otherwise each lane stores its own
  // values (lanes hold consecutive pixels, so stores still coalesce).
  // Split workgroups write raw fp32 partial sums instead (summed, biased and
  // rounded by the reduce kernel).
  const int64_t PQ = static_cast<int64_t>(a.P) * a.Q;
  const bool split_out = a.splits > 1;
  float* part = split_out ? a.partial + static_cast<int64_t>(split) * a.slab : nullptr;
  const T* bias = reinterpret_cast<const T*>(a.b);
  T* y = reinterpret_cast<T*>(a.y);
  if (a.vec_out) {
    constexpr int EW = BN / 2;        // pixels per wave row
    constexpr int ES_ROW = EW + 4;    // staged row stride (floats)
    float* stage = reinterpret_cast<float*>(smem) + wave * 32 * ES_ROW;
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
      for (int nj = 0; nj < NJ; ++nj)
#pragma unroll
        for (int v = 0; v < 16; ++v) stage[mfma_row(v, lane) * ES_ROW + nj * 32 + l32] = acc[mi][nj][v];
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes are done
      __builtin_amdgcn_wave_barrier();
      // 32 rows x EW pixels = 4*EW/8 runs of 8; lane takes runs lane, lane+64, ...
#pragma unroll
      for (int it = 0; it < 32 * EW / 8 / 64; ++it) {
        const int run = lane + 64 * it;
        const int row = run / (EW / 8), cb = (run % (EW / 8)) * 8;
        const int i = k0 + wm * (BM / 2) + mi * 32 + row;
        const int j = j0 + wn * (BN / 2) + cb;
        if (i >= a.Kg || j >= a.NPQ) continue;
        const int k = g * a.Kg + i;
        const int n = j / static_cast<int>(PQ), pq = j - n * static_cast<int>(PQ);
        const int64_t o = (static_cast<int64_t>(n) * a.K + k) * PQ + pq;
        const float4 lo = *reinterpret_cast<const float4*>(stage + row * ES_ROW + cb);
        const float4 hi = *reinterpret_cast<const float4*>(stage + row * ES_ROW + cb + 4);
        float vals[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        if (split_out) {
          *reinterpret_cast<float4*>(part + o) = lo;
          *reinterpret_cast<float4*>(part + o + 4) = hi;
          continue;
        }
        const float bv = bias ? elem<T>::load(bias + k) : 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          vals[e] += bv;
          if (a.relu) vals[e] = fmaxf(vals[e], 0.f);
        }
        if constexpr (sizeof(T) == 2) {
          uint4 u;
          u.x = f32x2_to_bf16x2(vals[0], vals[1]);
          u.y = f32x2_to_bf16x2(vals[2], vals[3]);
          u.z = f32x2_to_bf16x2(vals[4], vals[5]);
          u.w = f32x2_to_bf16x2(vals[6], vals[7]);
          *reinterpret_cast<uint4*>(y + o) = u;
        } else {
          *reinterpret_cast<float4*>(reinterpret_cast<float*>(y) + o) = make_float4(vals[0], vals[1], vals[2], vals[3]);
          *reinterpret_cast<float4*>(reinterpret_cast<float*>(y) + o + 4) =
              make_float4(vals[4], vals[5], vals[6], vals[7]);
        }
      }
      __builtin_amdgcn_wave_barrier();  // the next block reuses this wave's stage
    }
    return;
  }
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int i = k0 + wm * (BM / 2) + mi * 32 + mfma_row(v, lane);
      if (i >= a.Kg) continue;
      const int k = g * a.Kg + i;
      const float bv = (bias && !split_out) ? elem<T>::load(bias + k) : 0.f;
#pragma unroll
      for (int nj = 0; nj < NJ; ++nj) {
        if (!jvalid[nj]) continue;
        if (split_out) {
          part[ybase[nj] + k * PQ] = acc[mi][nj][v];
          continue;
        }
        float val = acc[mi][nj][v] + bv;
        if (a.relu) val = fmaxf(val, 0.f);
        elem<T>::store(y + ybase[nj] + k * PQ, val);
      }
    }
  }
}

// Wp[g][ch][kp][tap][cg][e] = w[g*Kg + kp][ch*Cc + cg*UE + e][tap], zero past
// Kg rows or Cg channels.  One workgroup per packed row (g, ch, kp); its
// threads write the row's RS*NG*UE elements consecutively.
template <typename T>
__global__ __launch_bounds__(256) void pack_filters_kernel(const T* __restrict__ w, T* __restrict__ wp, int Kg,
                                                           int Cg, int RS, int NG, int nch, int Kpad) {
  constexpr int UE = elem<T>::per16;
  const int row = blockIdx.x;                 // (g*nch + ch)*Kpad + kp
  const int kp = row % Kpad, gc = row / Kpad;
  const int ch = gc % nch, g = gc / nch;
  const int rowlen = RS * NG * UE;
  T* dst = wp + static_cast<int64_t>(row) * rowlen;
  const bool krow = kp < Kg;
  const T* src = w + static_cast<int64_t>(g * Kg + (krow ? kp : 0)) * Cg * RS;
  for (int i = threadIdx.x; i < rowlen; i += 256) {
    const int e = i % UE, rest = i / UE;
    const int cg = rest % NG, tap = rest / NG;
    const int c = (ch * NG + cg) * UE + e;
    T v = elem<T>::from_f32(0.f);
    if (krow && c < Cg) v = src[c * RS + tap];
    dst[i] = v;
  }
}

// Sum of the split partials, plus bias, ReLU, rounding to the output type;
// four consecutive outputs per thread (flat index: outputs stay below 2^31).
template <typename T>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part, const T* __restrict__ bias,
                                                            T* __restrict__ y, int total, int slab, int PQ, int K,
                                                            int splits, int relu) {
  const int i0 = (blockIdx.x * 256 + threadIdx.x) * 4;
  if (i0 >= total) return;
  const int n4 = total - i0 < 4 ? total - i0 : 4;
  float sum[4] = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < splits; ++s) {
    const float* p = part + static_cast<int64_t>(s) * slab + i0;
    if (n4 == 4) {
      const float4 v = *reinterpret_cast<const float4*>(p);  // slabs and i0 are multiples of 4 floats
      sum[0] += v.x; sum[1] += v.y; sum[2] += v.z; sum[3] += v.w;
    } else {
      for (int e = 0; e < n4; ++e) sum[e] += p[e];
    }
  }
  for (int e = 0; e < n4; ++e) {
    const int i = i0 + e;
    float v = sum[e];
    if (bias) v += elem<T>::load(bias + (i / PQ) % K);
    if (relu) v = fmaxf(v, 0.f);
    elem<T>::store(y + i, v);
  }
}

// Largest halo span (in virtual rows) over all pixel tiles of N images.  The
// span of a tile depends only on where it starts within an image, which
// repeats every PQ / gcd(BN, PQ) tiles, so one period is scanned.
int halo_rows(const Shape& s, int64_t N, int Hv) {
  const int64_t PQ = s.P * s.Q, NPQ = N * PQ;
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
// Each launch reads at most 1 GiB of input, so a buffer offset (at most the
// buffer size, which marks out-of-range lanes) plus a channel offset stays
// within 32 bits.
constexpr int64_t kMaxLaunchBytes = (int64_t)1 << 30;
constexpr int kCUs = 256;

struct IgPlan {
  int BM, NG, RST;
  int64_t images_per_launch;
  size_t wp_bytes;      // packed filters
  size_t part_bytes;    // split-K partial sums (per launch)
  IgArgs a;
  size_t lds;
};

// Split the channel chunks over several workgroups when the output tiles
// alone leave CUs idle: pick the split count S (1..8, at least two chunks per
// split) that minimises the number of full waves of 256 CUs per unit of work,
// ceil(tiles*S / 256) / S, plus a small charge per extra split for the
// partial-sum traffic.
void choose_splits(const Shape& s, IgPlan& pl) {
  IgArgs& a = pl.a;
  const int64_t tiles = (int64_t)((a.NPQ + BN - 1) / BN) * a.ktiles * s.G;
  int best = 1;
  double best_cost = 1e30;
  if (tiles < kCUs) {
    for (int S = 1; S <= 8 && S <= (a.nch + 1) / 2; ++S) {
      const double waves = (double)((tiles * S + kCUs - 1) / kCUs) / S;
      const double cost = waves + 0.05 * (S - 1);
      if (cost < best_cost - 1e-9) {
        best_cost = cost;
        best = S;
      }
    }
  }
  a.chunks_per_split = (a.nch + best - 1) / best;
  a.splits = (a.nch + a.chunks_per_split - 1) / a.chunks_per_split;
}

// Plan for `N1` images per launch (all of them unless the input exceeds the
// per-launch limit).
template <typename T>
bool make_plan(const Shape& s, IgPlan& pl, int64_t N1 = -1) {
  constexpr int UE = elem<T>::per16;
  const int64_t img_bytes = s.C * s.H * s.W * s.esize();
  if (img_bytes > kMaxLaunchBytes) return false;
  if (N1 < 0) {
    N1 = kMaxLaunchBytes / img_bytes;
    if (N1 > s.N) N1 = s.N;
    if (N1 < 1) N1 = 1;
  }
  pl.images_per_launch = N1;
  IgArgs& a = pl.a;
  a.N = (int)N1; a.C = (int)s.C; a.H = (int)s.H; a.W = (int)s.W; a.K = (int)s.K;
  a.R = (int)s.R; a.S = (int)s.S; a.P = (int)s.P; a.Q = (int)s.Q;
  a.sh = s.sh; a.sw = s.sw; a.ph = s.ph; a.pw = s.pw; a.dh = s.dh; a.dw = s.dw;
  a.Cg = (int)s.Cg; a.Kg = (int)s.Kg; a.G = s.G; a.relu = s.relu ? 1 : 0;
  a.Hv = (int)((s.P - 1) * s.sh + (s.R - 1) * s.dh + 1);
  a.Wv = (int)((s.Q - 1) * s.sw + (s.S - 1) * s.dw + 1);
  a.VR = halo_rows(s, N1, a.Hv);
  a.NPQ = (int)(N1 * s.P * s.Q);
  const int RS = a.R * a.S;
  pl.BM = s.Kg <= 64 ? 64 : 128;
  a.ktiles = (a.Kg + pl.BM - 1) / pl.BM;
  a.Kpad = a.ktiles * pl.BM;
  pl.RST = 0;
  if (RS == 1) pl.RST = 1;
  if (RS == 9) pl.RST = 9;
  for (size_t limit : {kLdsPreferred, kLdsLimit}) {
    for (int ng = (s.Cg > UE ? 2 : 1); ng >= 1; --ng) {
      a.units = RS * ng;
      a.steps = (a.units + 1) / 2;
      a.UR = (2 * a.steps) | 1;
      a.PS = ng | 1;
      a.xs_units = a.VR * a.Wv * a.PS;
      size_t lds = ((size_t)pl.BM * a.UR + (size_t)a.xs_units) * 16 + (size_t)2 * a.steps * 4;
      const size_t stage = (size_t)4 * 32 * (BN / 2 + 4) * sizeof(float);  // epilogue staging
      if (lds < stage) lds = stage;
      if (lds > limit) continue;
      pl.NG = ng;
      pl.lds = lds;
      a.nch = (int)((s.Cg + UE * ng - 1) / (UE * ng));
      pl.wp_bytes = (size_t)s.G * a.nch * a.Kpad * a.units * 16;
      if (pl.wp_bytes > (size_t)kMaxLaunchBytes) return false;
      choose_splits(s, pl);
      a.slab = (int)((N1 * s.K * s.P * s.Q + 3) & ~(int64_t)3);
      pl.part_bytes = a.splits > 1 ? (size_t)a.splits * a.slab * sizeof(float) : 0;
      return true;
    }
  }
  return false;
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

template <typename T, int BM, int NG, int RST>
hipError_t launch_one(const IgPlan& pl, const IgArgs& a, hipStream_t stream) {
  const auto kern = implicit_gemm_kernel<T, BM, NG, RST>;
  // Raise the kernel's dynamic-LDS limit once (not per call, so that calls
  // can be captured into a graph after the first one).
  static std::atomic<int> lds_limit{64 * 1024};
  if ((int)pl.lds > lds_limit.load()) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsLimit);
    if (e != hipSuccess) return e;
    lds_limit.store((int)kLdsLimit);
  }
  const dim3 grid((a.NPQ + BN - 1) / BN, a.ktiles * a.G, a.splits);
  hipLaunchKernelGGL(kern, grid, dim3(kThreads), pl.lds, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.splits == 1) return e;
  const int total = a.N * a.K * a.P * a.Q;
  hipLaunchKernelGGL(splitk_reduce_kernel<T>, dim3((unsigned)((total + 1023) / 1024)), dim3(256), 0, stream,
                     a.partial, reinterpret_cast<const T*>(a.b), reinterpret_cast<T*>(a.y), total, a.slab, a.P * a.Q,
                     a.K, a.splits, a.relu);
  return hipGetLastError();
}

template <typename T, int BM, int NG>
hipError_t launch_rst(const IgPlan& pl, const IgArgs& a, hipStream_t stream) {
  switch (pl.RST) {
    case 1: return launch_one<T, BM, NG, 1>(pl, a, stream);
    case 9: return launch_one<T, BM, NG, 9>(pl, a, stream);
    default: return launch_one<T, BM, NG, 0>(pl, a, stream);
  }
}

template <typename T>
hipError_t pack_typed(const Shape& s, const void* w, void* wp, hipStream_t stream) {
  IgPlan pl;
  if (!make_plan<T>(s, pl)) return hipErrorInvalidValue;
  const unsigned rows = (unsigned)(s.G * pl.a.nch * pl.a.Kpad);
  hipLaunchKernelGGL(pack_filters_kernel<T>, dim3(rows), dim3(256), 0, stream, reinterpret_cast<const T*>(w),
                     reinterpret_cast<T*>(wp), (int)s.Kg, (int)s.Cg, (int)(s.R * s.S), pl.NG, pl.a.nch, pl.a.Kpad);
  return hipGetLastError();
}

template <typename T>
hipError_t main_typed(const Shape& s, const void* x, const void* wp, const void* b, void* y, void* part_ws,
                      hipStream_t stream) {
  IgPlan pl;
  if (!make_plan<T>(s, pl)) return hipErrorInvalidValue;
  float* part = reinterpret_cast<float*>(part_ws);
  const int64_t img_elems = s.C * s.H * s.W, out_elems = s.K * s.P * s.Q;
  for (int64_t n0 = 0; n0 < s.N; n0 += pl.images_per_launch) {
    const int64_t cnt = s.N - n0 < pl.images_per_launch ? s.N - n0 : pl.images_per_launch;
    IgPlan cur = pl;
    // The last, smaller batch of images has its own tiles, halo span and
    // split count.
    if (cnt != pl.images_per_launch && !make_plan<T>(s, cur, cnt)) return hipErrorInvalidValue;
    if (cur.NG != pl.NG || cur.BM != pl.BM) return hipErrorInvalidValue;
    if (cur.a.splits > 1 && !part) return hipErrorInvalidValue;
    IgArgs a = cur.a;
    a.x = reinterpret_cast<const T*>(x) + n0 * img_elems;
    a.y = reinterpret_cast<T*>(y) + n0 * out_elems;
    a.x_bytes = (uint32_t)(cnt * img_elems * s.esize());
    a.wp = wp;
    a.wp_bytes = (uint32_t)pl.wp_bytes;
    a.b = b;
    a.partial = part;
    a.vec_out = (s.P * s.Q) % 8 == 0 && reinterpret_cast<uintptr_t>(a.y) % 16 == 0;
    hipError_t e;
    if (pl.BM == 64)
      e = pl.NG == 2 ? launch_rst<T, 64, 2>(cur, a, stream) : launch_rst<T, 64, 1>(cur, a, stream);
    else
      e = pl.NG == 2 ? launch_rst<T, 128, 2>(cur, a, stream) : launch_rst<T, 128, 1>(cur, a, stream);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <typename T>
size_t split_bytes_typed(const Shape& s) {
  IgPlan pl;
  if (!make_plan<T>(s, pl)) return 0;
  size_t part = pl.part_bytes;
  const int64_t rem = s.N % pl.images_per_launch;
  if (rem) {
    IgPlan last;
    if (make_plan<T>(s, last, rem) && last.part_bytes > part) part = last.part_bytes;
  }
  return part;
}

template <typename T>
std::string describe_typed(const Shape& s) {
  IgPlan pl;
  if (!make_plan<T>(s, pl)) return "implicit_gemm: does not fit";
  char buf[512];
  const char* tn = sizeof(T) == 2 ? "bf16" : "f32";
  snprintf(buf, sizeof(buf),
           "implicit_gemm kernels=pack_filters_kernel<%s>;implicit_gemm_kernel<%s,%d,%d,%d>%s tile=%dx%d "
           "grid=%dx%dx%d chunk=%d halo_rows=%d lds=%zu images_per_launch=%lld",
           tn, tn, pl.BM, pl.NG, pl.RST, pl.a.splits > 1 ? ";splitk_reduce_kernel" : "", pl.BM, BN,
           (pl.a.NPQ + BN - 1) / BN, pl.a.ktiles * s.G, pl.a.splits, pl.NG * elem<T>::per16, pl.a.VR, pl.lds,
           (long long)pl.images_per_launch);
  return buf;
}

}  // namespace

bool implicit_gemm_fits(const Shape& s) {
  IgPlan pl;
  if (s.dtype == DT_F32) return make_plan<float>(s, pl);
  return make_plan<bf16_t>(s, pl);
}

size_t implicit_gemm_packed_bytes(const Shape& s) {
  IgPlan pl;
  const bool ok = s.dtype == DT_F32 ? make_plan<float>(s, pl) : make_plan<bf16_t>(s, pl);
  return ok ? pl.wp_bytes : 0;
}

size_t implicit_gemm_split_bytes(const Shape& s) {
  return s.dtype == DT_F32 ? split_bytes_typed<float>(s) : split_bytes_typed<bf16_t>(s);
}

size_t implicit_gemm_workspace(const Shape& s) {
  return align256(implicit_gemm_packed_bytes(s)) + implicit_gemm_split_bytes(s);
}

hipError_t launch_implicit_pack(const Shape& s, const void* w, void* wp, hipStream_t stream) {
  return s.dtype == DT_F32 ? pack_typed<float>(s, w, wp, stream) : pack_typed<bf16_t>(s, w, wp, stream);
}

hipError_t launch_implicit_main(const Shape& s, const void* x, const void* wp, const void* b, void* y, void* part,
                                hipStream_t stream) {
  return s.dtype == DT_F32 ? main_typed<float>(s, x, wp, b, y, part, stream)
                           : main_typed<bf16_t>(s, x, wp, b, y, part, stream);
}

hipError_t launch_implicit_gemm(const Shape& s, const void* x, const void* w, const void* b, void* y, void* ws,
                                hipStream_t stream) {
  if (!ws) return hipErrorInvalidValue;
  hipError_t e = launch_implicit_pack(s, w, ws, stream);
  if (e != hipSuccess) return e;
  return launch_implicit_main(s, x, ws, b, y, reinterpret_cast<char*>(ws) + align256(implicit_gemm_packed_bytes(s)),
                              stream);
}

std::string implicit_gemm_describe(const Shape& s) {
  return s.dtype == DT_F32 ? describe_typed<float>(s) : describe_typed<bf16_t>(s);
}

}  // namespace convsel
