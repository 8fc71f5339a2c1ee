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
#include <type_traits>
#include <stdio.h>
#include <string>

#include "common.hpp"
#include "igemm_common.hpp"
#include "kernels.hpp"

namespace convsel {

namespace {

using namespace igemm;


struct IgArgs {
  const void* x;       // first image of this launch
  const void* wp;      // packed filters
  uint32_t x_bytes;    // extent of the input buffer of this launch
  uint32_t wp_bytes;
  int N, C, H, W, K, R, S, P, Q;
  int sh, sw, ph, pw, dh, dw;
  int Cg, Kg, G;
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
  int chunks_per_split;
  EpiArgs e;
};

// Virtual row of the first filter row for pixel j.
__device__ __forceinline__ int vrow_of(int j, const IgArgs& a) {
  const int PQ = a.P * a.Q;
  const int n = j / PQ, pq = j - n * PQ;
  return n * a.Hv + (pq / a.Q) * a.sh;
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
  {
    const int PQ = a.P * a.Q;
#pragma unroll
    for (int nj = 0; nj < NJ; ++nj) {
      const int j = j0 + wn * (BN / 2) + nj * 32 + l32;
      const int jj = j < a.NPQ ? j : jl;
      const int pq = jj - (jj / PQ) * PQ;
      const int q = pq - (pq / a.Q) * a.Q;
      pofs[nj] = ((vrow_of(jj, a) - vr_lo) * a.Wv + q * a.sw) * a.PS;
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
  lds_sync();
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
    lds_sync();
    if (more) {
      stash(ch + 1);
      lds_sync();
    }
  }

  store_tile<T, BM>(acc, smem, a.e, j0, k0, g, blockIdx.z);
}

// ---------------------------------------------------------------------------
// 1x1 layers (R = S = 1, one group).  The product is then a plain GEMM per
// image, Y[k][pixel] = sum_c W[k][c] * X[c][pixel]: the filters need no
// repacking (a K x C row is already reduction-contiguous) and there is no
// halo.  The input, however, is pixel-contiguous (NCHW), while an MFMA lane
// needs 8 bf16 (4 fp32) consecutive channels of one pixel; so each thread
// loads UE channels x 4 consecutive pixels with wide loads (8 bytes bf16,
// 16 bytes fp32 per channel), transposes them in registers into 4 pixel
// units of UE channels, and stores those to LDS.
//
// A chunk is 8 units (64 bf16 / 32 fp32 channels) of every pixel and filter
// row.  LDS rows of 8 units are XOR-swizzled, unit u of row r at
// r*8 + (u ^ ((r >> 1) & 7)): the MFMA reads of 16 consecutive rows and the
// stores of 16 consecutive lanes then hit distinct 16-byte bank groups.
//
// Strided or padded 1x1 layers, and plane sizes that are not a multiple of
// 4, use the same kernel with one element load per pixel (GATHER).
// ---------------------------------------------------------------------------
struct PwArgs {
  const void* x;        // first image of this launch (the DMA kernel: possibly the repacked input)
  const void* w;        // K x C filters (a 1x1 layer's KCRS layout)
  uint32_t x_bytes, w_bytes;
  int C, H, W, HW, P, Q, sh, sw, ph, pw;  // HW: input plane (the DMA kernel: its pixel span)
  int NPQ, ktiles, ptiles, nch, chunks_per_split;
  EpiArgs e;
};

constexpr int kPwUnits = 8;  // 16-byte channel units per row and chunk

__device__ __forceinline__ int pw_swz(int row, int u) { return row * kPwUnits + (u ^ ((row >> 1) & 7)); }

__device__ __forceinline__ u32x4_t buf_load_px4(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, float*) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
}
__device__ __forceinline__ u32x4_t buf_load_px4(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, bf16_t*) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0);
  u32x4_t o;
  o[0] = v[0];
  o[1] = v[1];
  o[2] = 0u;
  o[3] = 0u;
  return o;
}

// Work is handed out in units (pixel tile, filter tile, channel split), with
// the k-tiles and splits of one pixel tile adjacent.  The grid is persistent:
// workgroup w serves XCD w % 8 (workgroups are dealt to the 8 XCDs
// round-robin by id), each XCD takes one contiguous range of units -- so the
// units that read the same input or the same filters share an L2 -- and the
// workgroups of an XCD take its units in turn.  A workgroup runs through the
// (unit, chunk) items of its units with the loads of the next NS items in
// flight (NS register stages), across unit boundaries: a tile's epilogue
// overlaps the loads of the next tile.
template <typename T, int BM, bool GATHER, int NS>
__global__ __launch_bounds__(kThreads) void pointwise_gemm_kernel(PwArgs a) {
  constexpr int UE = elem<T>::per16;
  constexpr int ES = elem<T>::bytes;
  constexpr int MI = BM / 64, NJ = BN / 64;
  constexpr int CC = kPwUnits * UE;               // channels per chunk
  constexpr int AU = BM * kPwUnits / kThreads;    // filter units per thread
  extern __shared__ __align__(16) vec16 smem[];
  vec16* As = smem;                               // [BM][8], swizzled
  vec16* Bs = smem + BM * kPwUnits;               // [BN][8], swizzled

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int half = lane >> 5, l32 = lane & 31;
  const int cg = tid & 7, pg = tid >> 3;  // input: channel unit cg of pixels 4*pg .. +3

  // This workgroup's units: u_first, u_first + stride, ... below u_end.
  const int units = a.ptiles * a.ktiles * a.e.splits;
  const int per_xcd = (units + 7) >> 3;
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3, slots = gridDim.x >> 3;
  const int u_end = min(units, (xcd + 1) * per_xcd);
  const int u_first = xcd * per_xcd + slot;

  const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, a.x_bytes);
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(a.w, a.w_bytes);
  const uint32_t plane = static_cast<uint32_t>(a.H * a.W * ES);  // bytes per input channel plane

  // Register stages.
  u32x4_t braw[NS][GATHER ? 1 : UE];     // contiguous: 4 pixels of channel e (BW words used)
  uint32_t graw[NS][GATHER ? UE : 1][4]; // gather: channel e of pixel i
  vec16 areg[NS][AU];

  // Chunk range of unit u.
  auto chunk_begin = [&](int u) { return (u % a.e.splits) * a.chunks_per_split; };
  auto chunk_end = [&](int u) { return min(a.nch, (u % a.e.splits + 1) * a.chunks_per_split); };

  // Loads of item (u, ch) into stage S.  u and ch are workgroup-uniform;
  // readfirstlane keeps everything derived from them in scalar registers.
  auto fetch = [&](auto stage, int u_in, int ch_in) {
    constexpr int S = decltype(stage)::value;
    const int u = __builtin_amdgcn_readfirstlane(u_in);
    const int ch = __builtin_amdgcn_readfirstlane(ch_in);
    const int tile = u / a.e.splits;
    const int pt = tile / a.ktiles, kt = tile - pt * a.ktiles;
    const int j0 = pt * BN, k0 = kt * BM;
    const int c0 = ch * CC;
    const bool tail = c0 + CC > a.C;  // uniform
    const bool cvalid = !tail || c0 + cg * UE < a.C;
    // The channel offset (c0 + e) * plane is the scalar offset; a lane's
    // vector offset is its pixel's, or x_bytes (reads zero) past the data.
    if constexpr (!GATHER) {
      // Plane size a multiple of 4: the 4 pixels are consecutive in one image.
      const int j = j0 + 4 * pg;
      const int n = j / a.HW, pix = j - n * a.HW;
      const uint32_t vo = (cvalid && j < a.NPQ) ? static_cast<uint32_t>(((n * a.C + cg * UE) * a.HW + pix) * ES)
                                                : a.x_bytes;
#pragma unroll
      for (int e = 0; e < UE; ++e)
        braw[S][e] = buf_load_px4(xr, vo, static_cast<uint32_t>(c0 + e) * plane, (T*)nullptr);
    } else {
      const int PQ = a.P * a.Q;
      uint32_t vo[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = j0 + 4 * pg + i;
        const int n = j / PQ, pq = j - n * PQ;
        const int p = pq / a.Q, q = pq - p * a.Q;
        const int ih = p * a.sh - a.ph, iw = q * a.sw - a.pw;
        const bool ok = cvalid && j < a.NPQ && ih >= 0 && ih < a.H && iw >= 0 && iw < a.W;
        vo[i] = ok ? static_cast<uint32_t>(((n * a.C + cg * UE) * a.H * a.W + ih * a.W + iw) * ES) : a.x_bytes;
      }
#pragma unroll
      for (int e = 0; e < UE; ++e)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          graw[S][e][i] = buf_load_elem(xr, vo[i], static_cast<uint32_t>(c0 + e) * plane, (T*)nullptr);
    }
    // Filters: unit f = tid + t*256 is row f / 8, unit f % 8 of the tile;
    // rows past K fall past the buffer.
    const uint32_t wso = static_cast<uint32_t>(c0 * ES);
#pragma unroll
    for (int t = 0; t < AU; ++t) {
      const int f = tid + t * kThreads;
      const int row = f >> 3, cu = f & 7;
      const uint32_t vo = (!tail || c0 + cu * UE < a.C) ? static_cast<uint32_t>(((k0 + row) * a.C + cu * UE) * ES)
                                                        : a.w_bytes;
      areg[S][t] = buf_load16(wr, vo, wso);
    }
  };

  // Stage S into LDS.
  auto stash = [&](auto stage) {
    constexpr int S = decltype(stage)::value;
    // Pixel units: unit i holds channels cg*UE .. +UE-1 of pixel 4*pg + i.
    vec16 u[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        if constexpr (GATHER) {
          if constexpr (sizeof(T) == 2)
            u[i].d[d] = (graw[S][2 * d][i] & 0xffffu) | (graw[S][2 * d + 1][i] << 16);
          else
            u[i].d[d] = graw[S][d][i];
        } else {
          if constexpr (sizeof(T) == 2) {
            // channel 2d / 2d+1 of pixel i: half i&1 of word i>>1
            const uint32_t lo = braw[S][2 * d][i >> 1], hi = braw[S][2 * d + 1][i >> 1];
            u[i].d[d] = (i & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
          } else {
            u[i].d[d] = braw[S][d][i];
          }
        }
      }
    }
    // Odd pixel groups store their units in the order 1,0,3,2 so that the
    // 16 lanes of two neighbouring groups write both pixel parities at once.
    const uint32_t odd = static_cast<uint32_t>(pg & 1);
    const uint32_t m = 0u - odd;  // all ones for odd groups (bit select, no register indexing)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      vec16 v;
#pragma unroll
      for (int d = 0; d < 4; ++d) v.d[d] = (u[i ^ 1].d[d] & m) | (u[i].d[d] & ~m);
      Bs[pw_swz(4 * pg + (i ^ static_cast<int>(odd)), cg)] = v;
    }
#pragma unroll
    for (int t = 0; t < AU; ++t) {
      const int f = tid + t * kThreads;
      As[pw_swz(f >> 3, f & 7)] = areg[S][t];
    }
  };

  f32x16_t acc[MI][NJ];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int nj = 0; nj < NJ; ++nj) acc[mi][nj] = zero16();

  const int arow0 = wm * (BM / 2) + l32;
  const int brow0 = wn * (BN / 2) + l32;
  auto mfma_chunk = [&]() {
#pragma unroll
    for (int st = 0; st < kPwUnits / 2; ++st) {
      const int u = 2 * st + half;
      vec16 af[MI], bfr[NJ];
#pragma unroll
      for (int mi = 0; mi < MI; ++mi) af[mi] = As[pw_swz(arow0 + mi * 32, u)];
#pragma unroll
      for (int nj = 0; nj < NJ; ++nj) bfr[nj] = Bs[pw_swz(brow0 + nj * 32, u)];
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int nj = 0; nj < NJ; ++nj) mfma_32x32<T>(acc[mi][nj], af[mi], bfr[nj]);
    }
  };

  // Items in order: (u, ch) for ch in the chunk range of u, then the next
  // unit u + slots.  The fetch cursor (fu, fch) runs NS items ahead of the
  // compute cursor (cu, cch).
  int fu = u_first, fch = 0;
  if (fu < u_end) fch = chunk_begin(fu);
  static_for<NS>([&](auto s) {
    if (fu < u_end) {
      fetch(s, fu, fch);
      if (++fch >= chunk_end(fu)) {
        fu += slots;
        fch = fu < u_end ? chunk_begin(fu) : 0;
      }
    }
  });
  int cu = u_first;
  if (cu >= u_end) return;  // uniform: no work for this workgroup
  int cch = chunk_begin(cu);
  stash(std::integral_constant<int, 0>{});
  lds_sync();
  bool done = false;
  while (!done) {
    static_for<NS>([&](auto s) {
      if (done) return;
      constexpr int S = decltype(s)::value;
      // LDS holds item (cu, cch), which came from stage S; refill S.
      if (fu < u_end) {
        fetch(s, fu, fch);
        if (++fch >= chunk_end(fu)) {
          fu += slots;
          fch = fu < u_end ? chunk_begin(fu) : 0;
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      mfma_chunk();
      lds_sync();
      if (++cch >= chunk_end(cu)) {
        const int tile = cu / a.e.splits;
        const int pt = tile / a.ktiles, kt = tile - pt * a.ktiles;
        store_tile<T, BM>(acc, smem, a.e, pt * BN, kt * BM, 0, cu % a.e.splits);
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
#pragma unroll
          for (int nj = 0; nj < NJ; ++nj) acc[mi][nj] = zero16();
        lds_sync();
        cu += slots;
        if (cu >= u_end) {
          done = true;
          return;
        }
        cch = chunk_begin(cu);
      }
      stash(std::integral_constant<int, (S + 1) % NS>{});
      lds_sync();
    });
  }
}

// ---------------------------------------------------------------------------
// bf16 1x1 layers, stride 1, no padding, plane size a multiple of 2 pixels:
// the chunk of input (64 channels x 128 pixels) is copied by the buffer-to-LDS
// DMA exactly as it lies in memory, pixel-contiguous, and the MFMA B
// fragments are read with the gfx950 transposing LDS read ds_read_b64_tr_b16.
// No operand passes through registers on its way in, so a workgroup keeps NS
// chunks in LDS and the loads of NS-1 of them in flight while it multiplies
// the oldest one (and, between tiles, while it stores the finished tile).
//
// ds_read_b64_tr_b16 works on 16-lane groups: lane r of a group addresses
// 4 consecutive 16-bit elements (8 bytes); lane j receives element j % 4 of
// the rows addressed by lanes j/4, j/4 + 4, j/4 + 8, j/4 + 12.  With lane r
// addressing channel row c0 + r/4, pixels n0 + 4*(r%4) .. +3, lane j gets
// channels c0 .. c0+3 of pixel n0 + j: four consecutive reduction elements of
// one B column, half of an MFMA 32x32x16 B operand.
//
// LDS stage (32 KiB): A = 128 filter rows x 64 channels, 16-byte unit u of
// row r at r*8 + (u ^ ((r >> 1) & 7)); B = 64 channel rows x 128 pixels,
// 16-byte unit u of row c at c*16 + (u ^ 4*(c & 3)).  The DMA writes 64
// consecutive units per instruction; the swizzles are realised by choosing
// which global unit each lane fetches.  A reads of 16 consecutive rows, the
// transposing reads of 4 rows x 64 bytes per half-wave and the epilogue
// staging are free of bank conflicts.
// ---------------------------------------------------------------------------
constexpr int kDmaStageBytes = 32 * 1024;
constexpr int kDmaStages = 4;
// Loader waves of the 1x1 DMA kernel.  Eight measured slower on most ResNet-50
// 1x1 layers: at 768 threads the kernel must fit 168 VGPRs and spills.
constexpr int kDmaLoaders = 4;  // LDS stages of the 1x1 DMA kernel (plus 32 KiB of epilogue staging)


// NL loader waves (waves 4 .. 4+NL-1) share each chunk's DMA instructions.
template <int UB, int NS, int NL>
__global__ __launch_bounds__((4 + NL) * 64) void pointwise_dma_kernel(PwArgs a) {
  // Compute waves in a 4 x 1 layout: wave w holds rows 32 w .. 32 w + 31 of
  // the 128 x 128 tile and all 128 pixels, as pixels x channels (the MFMA's
  // A operand is the pixel fragment), so that its epilogue stores whole
  // 256-byte channel rows.
  constexpr int BM = 128, MI = 1, NJ = 4;
  constexpr int CC = 64;                                // channels per chunk
  constexpr int A_INS = 16 / NL;                         // A DMA instructions per loader wave per chunk
  constexpr int B_INS = (CC * BN * 2) / (64 * UB) / NL;  // B DMA instructions per loader wave per chunk
  static_assert(A_INS * NL == 16 && B_INS * NL * 64 * UB == CC * BN * 2 && (UB == 16 || B_INS % 4 == 0),
                "loader waves must split the chunk evenly");
  constexpr int INS = A_INS + B_INS;
  static_assert(UB == 16 || UB == 4, "DMA unit");
  static_assert((NS - 1) * INS <= 63, "vmcnt range");
  extern __shared__ __align__(16) vec16 smem[];
  char* lds = reinterpret_cast<char*>(smem);
  vec16* staging = reinterpret_cast<vec16*>(lds + NS * kDmaStageBytes);  // 8 KiB per compute wave

  // The wave index is uniform: reading it into a scalar register keeps the
  // DMA destinations (and so M0) in scalar arithmetic.
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool loader = wave >= 4;                        // waves 4.. issue the DMA, 0..3 multiply
  const int lw = loader ? wave - 4 : wave;
  const int half = lane >> 5, l32 = lane & 31;

  const int units = a.ptiles * a.ktiles * a.e.splits;
  const int per_xcd = (units + 7) >> 3;
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3, slots = gridDim.x >> 3;
  const int u_end = min(units, (xcd + 1) * per_xcd);
  const int u_first = xcd * per_xcd + slot;
  if (u_first >= u_end) return;  // uniform: no work for this workgroup

  auto chunk_begin = [&](int u) { return (u % a.e.splits) * a.chunks_per_split; };
  auto chunk_end = [&](int u) { return min(a.nch, (u % a.e.splits + 1) * a.chunks_per_split); };

  if (loader) {
    // ---- loader waves: DMA of item (u, ch) into stage st ----
    const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, a.x_bytes);
    const __amdgpu_buffer_rsrc_t wr = make_rsrc(a.w, a.w_bytes);
    const uint32_t plane = static_cast<uint32_t>(a.HW * 2);
    // A instruction i fills units (lw*4 + i)*64 + lane: row (lw*4+i)*8 +
    // lane/8, stored unit lane%8, global unit (lane%8) ^ ((row >> 1) & 7).
    int a_row[A_INS], a_unit[A_INS];
#pragma unroll
    for (int i = 0; i < A_INS; ++i) {
      const int row = (lw * A_INS + i) * 8 + (lane >> 3);
      a_row[i] = row;
      a_unit[i] = (lane & 7) ^ ((row >> 1) & 7);
    }
    // B instruction i: UB = 16 fills 4 channel rows (lw*4+i)*4 + lane/16,
    // stored unit lane%16; UB = 4 fills channel row lw*16 + i, 4-byte slot
    // lane (stored unit lane/4, pixel pair lane%4 within it).
    auto b_chan = [&](int i) { return UB == 16 ? (lw * B_INS + i) * 4 + (lane >> 4) : lw * B_INS + i; };
    auto b_pix = [&](int i) {  // first pixel (within the tile) of the lane's unit
      const int c = b_chan(i);
      if constexpr (UB == 16) return ((lane & 15) ^ (4 * (c & 3))) * 8;
      else return (((lane >> 2) ^ (4 * (c & 3))) * 8) + 2 * (lane & 3);
    };
    // Pixel offsets per unit: UB = 16 has one pixel unit per lane for all
    // instructions; UB = 4 one per value of c & 3 = i & 3.
    constexpr int NPX = UB == 16 ? 1 : 4;
    uint32_t pixoff[NPX];
    int pix_unit = -1;
    // Per-lane offsets of the current unit, recomputed only when the unit
    // changes (the chunk's channel offset goes into the scalar offset): A
    // row k0 + a_row[i], unit a_unit[i] (rows past K fall past the buffer);
    // B the lane's pixel in channel row b_chan(i), or x_bytes past the last
    // pixel.  Channels past C are masked only in a layer's last, partial
    // chunk.
    uint32_t a_vo[A_INS], b_vo[B_INS];
    auto issue = [&](int u_in, int ch_in, int st) {
      const int u = __builtin_amdgcn_readfirstlane(u_in);
      const int ch = __builtin_amdgcn_readfirstlane(ch_in);
      const int c0 = ch * CC;
      if (u != pix_unit) {
        pix_unit = u;
        const int tile = u / a.e.splits;
        const int pt = tile / a.ktiles, kt = tile - pt * a.ktiles;
        const int j0 = pt * BN, k0 = kt * BM;
#pragma unroll
        for (int q = 0; q < NPX; ++q) {
          const int j = j0 + b_pix(q);
          const int n = j / a.HW, pix = j - n * a.HW;
          pixoff[q] = j < a.NPQ ? static_cast<uint32_t>((n * a.C * a.HW + pix) * 2) : a.x_bytes;
        }
#pragma unroll
        for (int i = 0; i < A_INS; ++i)
          a_vo[i] = static_cast<uint32_t>(((k0 + a_row[i]) * a.C + a_unit[i] * 8) * 2);
#pragma unroll
        for (int i = 0; i < B_INS; ++i) {
          const uint32_t po = pixoff[UB == 16 ? 0 : (i & 3)];
          b_vo[i] = po != a.x_bytes ? po + static_cast<uint32_t>(b_chan(i)) * plane : a.x_bytes;
        }
      }
      const bool tail = c0 + CC > a.C;  // uniform
      char __attribute__((address_space(3)))* base =
          (char __attribute__((address_space(3)))*)(lds + st * kDmaStageBytes);
      const uint32_t wso = static_cast<uint32_t>(c0 * 2);
#pragma unroll
      for (int i = 0; i < A_INS; ++i) {
        const uint32_t vo = (!tail || c0 + a_unit[i] * 8 < a.C) ? a_vo[i] : a.w_bytes;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (lds_void_t*)(base + (lw * A_INS + i) * 1024), 16, vo, wso, 0,
                                                 0);
      }
      const uint32_t xso = static_cast<uint32_t>(c0) * plane;
#pragma unroll
      for (int i = 0; i < B_INS; ++i) {
        const uint32_t vo = (!tail || c0 + b_chan(i) < a.C) ? b_vo[i] : a.x_bytes;
        lds_void_t* dst = (lds_void_t*)(base + 16384 + (lw * B_INS + i) * 64 * UB);
        if constexpr (UB == 16)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, dst, 16, vo, xso, 0, 0);
        else
          __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, dst, 4, vo, xso, 0, 0);
      }
    };
    // Fetch cursor (fu, fch).  NS - 1 stages are filled up front and the
    // last right after barrier A of the first item (the first item's data
    // arrives a little sooner than behind a full queue); after that the
    // stage freed at barrier B of item k-1 is refilled right after barrier A
    // of item k, while the compute waves multiply item k, so the issue never
    // delays the barrier.  `later` counts the items issued after
    // the one being waited for (this wave issues nothing else, so that is
    // the vmcnt to wait for).
    int fu = u_first, fch = chunk_begin(u_first), fstage = 0;
    auto fetch_next = [&]() -> bool {
      if (fu >= u_end) return false;
      issue(fu, fch, fstage);
      fstage = fstage + 1 == NS ? 0 : fstage + 1;
      if (++fch >= chunk_end(fu)) {
        fu += slots;
        if (fu < u_end) fch = chunk_begin(fu);
      }
      return true;
    };
    int later = -1;
    for (int s = 0; s < NS - 1; ++s)
      if (fetch_next()) ++later;
    int cu = u_first, cch = chunk_begin(u_first);
    for (;;) {
      static_for<NS>([&](auto m) {
        if (later == decltype(m)::value) CONVSEL_WAIT_VMCNT(decltype(m)::value * INS);
      });
      // Plain barriers: the wait above already covers the item's DMA, and an
      // LDS fence here would also wait for the later items still in flight.
      __builtin_amdgcn_s_barrier();  // A: item visible to the compute waves
      if (fetch_next()) ++later;  // the last stage, then the one freed at the previous B
      __builtin_amdgcn_s_barrier();  // B: compute waves are done with this item's stage
      --later;                       // the next item to wait for is one further on
      if (++cch >= chunk_end(cu)) {
        cu += slots;
        if (cu >= u_end) break;
        cch = chunk_begin(cu);
      }
    }
    return;
  }

  // ---- compute waves ----
  // B fragment addresses (transposing reads): group g = lane/16 covers
  // pixels n0 = 16*(g&1) of the 32-column block and channels kk0 = 8*(g>>1)
  // of the 16-channel step; lane r = lane%16 reads channel row kk0 + r/4 (+4
  // for the second read), pixels n0 + 4*(r%4).
  int b_off[NJ];
  {
    const int g = lane >> 4, r = lane & 15;
    const int c_rel = 8 * (g >> 1) + (r >> 2);
#pragma unroll
    for (int nj = 0; nj < NJ; ++nj) {
      const int px = nj * 32 + 16 * (g & 1) + 4 * (r & 3);
      b_off[nj] = c_rel * 256 + ((((px >> 3) ^ (4 * (c_rel & 3)))) << 4) + ((px >> 2) & 1) * 8;
    }
  }
  int a_off[MI], a_swz[MI];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) {
    const int row = lw * 32 + mi * 32 + l32;
    a_off[mi] = row * 8;
    a_swz[mi] = (row >> 1) & 7;
  }

  // Without a split the accumulators start from the bias of the lane's
  // output channel (row kt * BM + 32 lw + l32 of the unit), so the epilogue
  // does not add it; the next unit's bias is loaded while this one's
  // epilogue runs.
  const uint16_t* bias = a.e.splits == 1 ? reinterpret_cast<const uint16_t*>(a.e.b) : nullptr;
  auto bias_of = [&](int u) -> float {
    const int kt = (u / a.e.splits) % a.ktiles;
    const int row = kt * BM + lw * 32 + l32;
    return (bias && row < a.e.Kg) ? bf16_to_f32(bias[row]) : 0.f;
  };
  f32x16_t acc[MI][NJ];
  {
    const float b0 = bias_of(u_first);
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int nj = 0; nj < NJ; ++nj)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[mi][nj][v] = b0;
  }

  int cu = u_first, cch = chunk_begin(u_first), cstage = 0;
  for (;;) {
    lds_sync();  // A
    const char* As = lds + cstage * kDmaStageBytes;
    const char* Bs = As + 16384;
#pragma unroll
    for (int kst = 0; kst < CC / 16; ++kst) {
      const int u = 2 * kst + half;
      bf16x8_t af[MI], bfr[NJ];
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
        af[mi] = *reinterpret_cast<const bf16x8_t*>(As + (a_off[mi] + (u ^ a_swz[mi])) * 16);
#pragma unroll
      for (int nj = 0; nj < NJ; ++nj) {
        const char* p = Bs + kst * 16 * 256 + b_off[nj];
        const v4s_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t*)(p));
        const v4s_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t*)(p + 4 * 256));
        bfr[nj] = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      }
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int nj = 0; nj < NJ; ++nj)
          acc[mi][nj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[nj], af[mi], acc[mi][nj], 0, 0, 0);
    }
    lds_sync();  // B: the stage may be refilled
    cstage = cstage + 1 == NS ? 0 : cstage + 1;
    if (++cch >= chunk_end(cu)) {
      // Tile done: each compute wave stages its part in its own region.
      const int tile = cu / a.e.splits;
      const int pt = tile / a.ktiles, kt = tile - pt * a.ktiles;
      const float bn = cu + slots < u_end ? bias_of(cu + slots) : 0.f;
      store_block128t<bf16_t>(acc, reinterpret_cast<float*>(staging) + lw * 32 * 64, a.e, kt * BM + lw * 32, pt * BN,
                              0, cu % a.e.splits, true);
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int nj = 0; nj < NJ; ++nj)
#pragma unroll
          for (int v = 0; v < 16; ++v) acc[mi][nj][v] = bn;
      cu += slots;
      if (cu >= u_end) break;
      cch = chunk_begin(cu);
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 1x1 layers, stride 1, no padding, on planes of P*Q = 4 (mod 8) pixels
// (14 x 14): a tile is 128 output channels of one whole image.  Channel rows
// of such a plane are 8-byte aligned, so 16-byte units of one row do not
// exist in memory, but two consecutive rows (c even, c+1) are 4*P*Q bytes,
// 16-byte aligned and contiguous: the chunk's input, 64 channels of the
// image, is copied as 32 row pairs with 16-byte LDS DMA exactly as it lies,
// each pair PU = P*Q/4 units, PU+1 units apart in LDS (the extra unit reads
// zero).  Row c of the chunk starts at pair(c)*(PU+1)*16 + (c&1)*2*P*Q bytes,
// 8-byte aligned, which is all the transposing read ds_read_b64_tr_b16
// needs: the compute waves read pixel fragments as in the kernel above, from
// these row addresses.  Tile pixels past P*Q read the next row (or the zero
// unit) and land in output columns that are not stored.
//
// The tile spans NJ*32 >= P*Q pixels (7 blocks for 196): each compute wave
// holds 32 channels x NJ*32 pixels.  Its epilogue stages 16 channel rows at
// a time as bf16 (after the bias and, without a residual, the ReLU) and
// stores them as one contiguous run of 16*P*Q*2 bytes (the rows of one image
// are contiguous, 16-byte aligned when K is even), adding the residual, if
// any, to the rounded values as the other epilogues do.  K must be a multiple
// of 32, so a wave's rows are all real or all past K.
//
// Units (image, channel tile), channel tiles innermost, walked as in the
// kernel above; three 41 KiB stages.
// ---------------------------------------------------------------------------
constexpr int kImgStages = 3;
constexpr int kImgMaxPU = 49;                                   // P*Q <= 196
constexpr int kImgStageBytes = 16384 + 32 * (kImgMaxPU + 1) * 16;  // 41,984

template <int NJ>
__global__ __launch_bounds__(8 * 64) void pointwise_img_kernel(PwArgs a) {
  constexpr int BM = 128, CC = 64, NS = kImgStages;
  constexpr int A_INS = 4;  // filter DMA instructions per loader wave per chunk
  extern __shared__ __align__(16) vec16 smem[];
  char* lds = reinterpret_cast<char*>(smem);
  const int HW = a.H * a.W, PU = HW / 4, pitch = (PU + 1) * 16;
  const int NBI = (32 * (PU + 1) + 63) / 64;  // input DMA instructions per chunk (all loader waves)

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool loader = wave >= 4;
  const int lw = loader ? wave - 4 : wave;
  const int half = lane >> 5, l32 = lane & 31;

  const int units = a.ptiles * a.ktiles;  // ptiles = images of this launch
  const int per_xcd = (units + 7) >> 3;
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3, slots = gridDim.x >> 3;
  const int u_end = min(units, (xcd + 1) * per_xcd);
  const int u_first = xcd * per_xcd + slot;
  if (u_first >= u_end) return;  // uniform

  if (loader) {
    const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, a.x_bytes);
    const __amdgpu_buffer_rsrc_t wr = make_rsrc(a.w, a.w_bytes);
    // Filters as in the kernel above: instruction i fills rows
    // (lw*4 + i)*8 + lane/8, stored unit lane%8, global unit
    // (lane%8) ^ ((row >> 1) & 7).
    int a_unit[A_INS];
    uint32_t a_vo[A_INS];
#pragma unroll
    for (int i = 0; i < A_INS; ++i) a_unit[i] = (lane & 7) ^ ((((lw * A_INS + i) * 8 + (lane >> 3)) >> 1) & 7);
    // Input instruction j (this wave: j = lw, lw+4, ...) fills LDS units
    // j*64 + lane: pair i = unit / (PU+1), unit k of the pair (k == PU: the
    // zero unit).  Byte offset within the chunk: i*4*HW + 16k.
    const int nb = (NBI - lw + 3) / 4;  // this wave's input instructions
    const int ins = A_INS + nb;
    auto b_pair = [&](int q) { return ((lw + 4 * q) * 64 + lane) / (PU + 1); };
    auto b_off = [&](int q) -> uint32_t {
      const int U = (lw + 4 * q) * 64 + lane, i = U / (PU + 1), k = U - i * (PU + 1);
      return (i < 32 && k < PU) ? static_cast<uint32_t>(i * 4 * HW + 16 * k) : a.x_bytes;
    };
    int tile_u = -1;
    uint32_t xbase = 0;
    int fu = u_first, fch = 0, fstage = 0;
    auto fetch_next = [&]() -> bool {
      if (fu >= u_end) return false;
      const int u = __builtin_amdgcn_readfirstlane(fu);
      const int c0 = __builtin_amdgcn_readfirstlane(fch) * CC;
      if (u != tile_u) {
        tile_u = u;
        const int n = u / a.ktiles, k0 = (u - n * a.ktiles) * BM;
#pragma unroll
        for (int i = 0; i < A_INS; ++i)
          a_vo[i] = static_cast<uint32_t>(((k0 + (lw * A_INS + i) * 8 + (lane >> 3)) * a.C + a_unit[i] * 8) * 2);
        xbase = static_cast<uint32_t>(n) * a.C * HW * 2;
      }
      const bool tail = c0 + CC > a.C;  // uniform
      char __attribute__((address_space(3)))* base =
          (char __attribute__((address_space(3)))*)(lds + fstage * kImgStageBytes);
      const uint32_t wso = static_cast<uint32_t>(c0 * 2);
#pragma unroll
      for (int i = 0; i < A_INS; ++i) {
        const uint32_t vo = (!tail || c0 + a_unit[i] * 8 < a.C) ? a_vo[i] : a.w_bytes;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (lds_void_t*)(base + (lw * A_INS + i) * 1024), 16, vo, wso, 0,
                                                 0);
      }
      const uint32_t xso = xbase + static_cast<uint32_t>(c0) * HW * 2;
      for (int q = 0; q < nb; ++q) {
        const uint32_t vo = (!tail || c0 + 2 * b_pair(q) < a.C) ? b_off(q) : a.x_bytes;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void_t*)(base + 16384 + (lw + 4 * q) * 1024), 16, vo, xso,
                                                 0, 0);
      }
      fstage = fstage + 1 == NS ? 0 : fstage + 1;
      if (++fch >= a.nch) {
        fu += slots;
        fch = 0;
      }
      return true;
    };
    // As in the kernel above: NS-1 items ahead, the wave's DMA counted in
    // order (`later` items issued after the one waited for).
    int later = -1;
    for (int s = 0; s < NS - 1; ++s)
      if (fetch_next()) ++later;
    int cu = u_first, cch = 0;
    for (;;) {
      wait_vmcnt(later * ins);
      __builtin_amdgcn_s_barrier();  // A: item visible to the compute waves
      if (fetch_next()) ++later;
      __builtin_amdgcn_s_barrier();  // B: compute waves are done with this item's stage
      --later;
      if (++cch >= a.nch) {
        cu += slots;
        if (cu >= u_end) break;
        cch = 0;
      }
    }
    return;
  }

  // ---- compute waves: 32 channels (rows lw*32 ..) x NJ*32 pixels ----
  // Transposing reads: group g = lane/16 covers pixels 16*(g&1) of a block
  // and channels 8*(g>>1) of the 16-channel step; lane r = lane%16 reads
  // channel row cr = 8*(g>>1) + r/4 (and cr + 4), pixels 4*(r%4) .. +3.
  int b_lane;
  {
    const int g = lane >> 4, r = lane & 15;
    const int cr = 8 * (g >> 1) + (r >> 2);
    b_lane = (cr >> 1) * pitch + (cr & 1) * HW * 2 + (16 * (g & 1) + 4 * (r & 3)) * 2;
  }
  const int a_off = (lw * 32 + l32) * 8, a_swz = ((lw * 32 + l32) >> 1) & 7;
  const uint16_t* bias = reinterpret_cast<const uint16_t*>(a.e.b);
  uint16_t* y = reinterpret_cast<uint16_t*>(a.e.y);
  const uint16_t* res = reinterpret_cast<const uint16_t*>(a.e.res);
  char* staging = lds + NS * kImgStageBytes + lw * (16 * HW * 2);  // 16 rows of this wave
  const int run_units = 16 * HW * 2 / 16;                          // 16-byte units of 16 rows

  // The bias of a unit's channel is read when the unit starts, long before
  // its epilogue needs it.
  auto bias_of = [&](int u) -> float {
    const int kb = (u % a.ktiles) * BM + lw * 32 + l32;
    return (bias && kb < a.e.K) ? bf16_to_f32(bias[kb]) : 0.f;
  };
  float bv = bias_of(u_first);
  f32x16_t acc[NJ];
#pragma unroll
  for (int nj = 0; nj < NJ; ++nj) acc[nj] = zero16();
  int cu = u_first, cch = 0, cstage = 0;
  for (;;) {
    lds_sync();  // A
    const char* As = lds + cstage * kImgStageBytes;
    const char* Bs = As + 16384;
    // Step kst (16 channels: pairs 8 kst .., the second read 4 channels = 2
    // pairs on): its fragments are read while the previous step's MFMAs run.
    bf16x8_t af[2], bfr[2][NJ];
    auto load_step = [&](int kst, auto set_c) {
      constexpr int SET = decltype(set_c)::value;
      const int u = 2 * kst + half;
      af[SET] = *reinterpret_cast<const bf16x8_t*>(As + (a_off + (u ^ a_swz)) * 16);
      const char* p0 = Bs + kst * 8 * pitch + b_lane;
#pragma unroll
      for (int nj = 0; nj < NJ; ++nj) {
        const char* p = p0 + nj * 64;
        const v4s_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t*)(p));
        const v4s_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t*)(p + 2 * pitch));
        bfr[SET][nj] = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      }
    };
    // (Scheduling barriers keep each step's reads together ahead of the
    // previous step's MFMAs; left alone, the compiler interleaves one read
    // per MFMA and waits for it.)
    load_step(0, std::integral_constant<int, 0>{});
    static_for<CC / 16>([&](auto k_c) {
      constexpr int KST = decltype(k_c)::value, SET = KST & 1;
      if constexpr (KST + 1 < CC / 16) load_step(KST + 1, std::integral_constant<int, SET ^ 1>{});
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int nj = 0; nj < NJ; ++nj)
        acc[nj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[SET][nj], af[SET], acc[nj], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    });
    lds_sync();  // B: the stage may be refilled
    cstage = cstage + 1 == NS ? 0 : cstage + 1;
    if (++cch < a.nch) continue;

    // Unit done: image n, channels k0 + lw*32 ...
    const int n = cu / a.ktiles, kw = (cu - n * a.ktiles) * BM + lw * 32;
    if (kw < a.e.K) {  // uniform per wave (K is a multiple of 32)
      const bool relu_now = a.e.relu && !res;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        // Stage rows 16h .. 16h+15 (lanes whose channel is among them).
        if ((l32 >> 4) == h) {
          char* row = staging + (l32 - 16 * h) * HW * 2;
#pragma unroll
          for (int nj = 0; nj < NJ; ++nj)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              const int px = nj * 32 + 8 * g + 4 * half;
              if (px < HW) {
                float v[4];
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                  v[t] = acc[nj][4 * g + t] + bv;
                  if (relu_now) v[t] = fmaxf(v[t], 0.f);
                }
                uint2 w;
                w.x = f32x2_to_bf16x2(v[0], v[1]);
                w.y = f32x2_to_bf16x2(v[2], v[3]);
                *reinterpret_cast<uint2*>(row + px * 2) = w;
              }
            }
        }
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's staging writes
        __builtin_amdgcn_wave_barrier();
        // The 16 rows are one contiguous run of y (and of the residual).
        const int64_t o = (static_cast<int64_t>(n) * a.e.K + kw + 16 * h) * HW;  // elements
        for (int q = lane; q < run_units; q += 64) {
          uint4 d = *reinterpret_cast<const uint4*>(staging + q * 16);
          if (res) {
            uint4 rr;
            __builtin_memcpy(&rr, res + o + q * 8, 16);
            const uint32_t dw[4] = {d.x, d.y, d.z, d.w}, rw[4] = {rr.x, rr.y, rr.z, rr.w};
            uint32_t ow[4];
#pragma unroll
            for (int m = 0; m < 4; ++m) {
              float lo = __uint_as_float(dw[m] << 16) + __uint_as_float(rw[m] << 16);
              float hi = __uint_as_float(dw[m] & 0xFFFF0000u) + __uint_as_float(rw[m] & 0xFFFF0000u);
              if (a.e.relu) {
                lo = fmaxf(lo, 0.f);
                hi = fmaxf(hi, 0.f);
              }
              ow[m] = f32x2_to_bf16x2(lo, hi);
            }
            d = make_uint4(ow[0], ow[1], ow[2], ow[3]);
          }
          __builtin_memcpy(y + o + q * 8, &d, 16);
        }
        __builtin_amdgcn_wave_barrier();  // the next rows reuse the staging
      }
    }
#pragma unroll
    for (int nj = 0; nj < NJ; ++nj) acc[nj] = zero16();
    cu += slots;
    if (cu >= u_end) break;
    cch = 0;
    bv = bias_of(cu);
  }
}

// Input of the 1x1 DMA kernel for layers whose plane is not a multiple of 8
// pixels, or that are strided or padded: xr[n][c][pix] = the input pixel
// that output pixel pix = p*Q + q reads (zero outside the image), and zero
// for P*Q <= pix < span (span = P*Q rounded up to 8).  Each thread writes 8
// consecutive pixels (one 16-byte store).
__global__ __launch_bounds__(256) void repack_plane_kernel(const uint16_t* __restrict__ x, uint16_t* __restrict__ xr,
                                                           int planes, int H, int W, int P, int Q, int sh, int sw,
                                                           int ph, int pw, int span) {
  const int per_plane = span / 8;
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= planes * per_plane) return;
  const int plane = t / per_plane, pix0 = (t - plane * per_plane) * 8;
  const int HW = H * W;
  const uint16_t* src = x + static_cast<int64_t>(plane) * HW;
  const int64_t left = static_cast<int64_t>(planes - plane) * HW;  // elements from src to the end of x
  const int PQ = P * Q;
  uint32_t v[8];
  // 16-byte loads need only 2-byte alignment on gfx950 (the compiler emits
  // them for any 16-byte copy); a load must not run past the end of x.
  auto load8 = [&](int64_t off, uint32_t (&e)[8]) {
    uint4 u;
    __builtin_memcpy(&u, src + off, 16);
    e[0] = u.x & 0xFFFFu; e[1] = u.x >> 16; e[2] = u.y & 0xFFFFu; e[3] = u.y >> 16;
    e[4] = u.z & 0xFFFFu; e[5] = u.z >> 16; e[6] = u.w & 0xFFFFu; e[7] = u.w >> 16;
  };
  const int p0 = pix0 / Q, q0 = pix0 - p0 * Q;
  const int ih0 = p0 * sh - ph, iw0 = q0 * sw - pw;
  if (sh == 1 && sw == 1 && ph == 0 && pw == 0 && pix0 + 8 <= left) {
    // Unstrided, unpadded: output pixel pix is input pixel pix.
    load8(pix0, v);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = pix0 + e < PQ ? v[e] : 0u;
  } else if (sw <= 2 && pix0 + 8 <= PQ && q0 + 8 <= Q && ih0 >= 0 && ih0 < H && iw0 >= 0 &&
             iw0 + 7 * sw < W && static_cast<int64_t>(ih0) * W + iw0 + 16 <= left) {
    // Eight outputs of one row with every input inside the image: one
    // 16-byte load (column stride 1) or two (stride 2: the even elements of
    // 16), both issued before either is unpacked.
    const uint16_t* row = src + static_cast<int64_t>(ih0) * W + iw0;
    if (sw == 1) {
      load8(row - src, v);
    } else {
      uint4 ua, ub;
      __builtin_memcpy(&ua, row, 16);
      __builtin_memcpy(&ub, row + 8, 16);
      v[0] = ua.x & 0xFFFFu; v[1] = ua.y & 0xFFFFu; v[2] = ua.z & 0xFFFFu; v[3] = ua.w & 0xFFFFu;
      v[4] = ub.x & 0xFFFFu; v[5] = ub.y & 0xFFFFu; v[6] = ub.z & 0xFFFFu; v[7] = ub.w & 0xFFFFu;
    }
  } else {
    // Element by element, walking the 8 pixels along the output row.  All
    // eight loads are issued before any is used (an element outside the
    // image reads the plane's first element and is then replaced by zero):
    // one memory round trip per thread, not eight.
    int p = p0, q = q0;
    int idx[8];
    bool ok[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int ih = p * sh - ph, iw = q * sw - pw;
      ok[e] = pix0 + e < PQ && ih >= 0 && ih < H && iw >= 0 && iw < W;
      idx[e] = ok[e] ? ih * W + iw : 0;
      if (++q == Q) {
        q = 0;
        ++p;
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = src[idx[e]];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = ok[e] ? v[e] : 0u;
  }
  uint4 o;
  o.x = v[0] | (v[1] << 16);
  o.y = v[2] | (v[3] << 16);
  o.z = v[4] | (v[5] << 16);
  o.w = v[6] | (v[7] << 16);
  *reinterpret_cast<uint4*>(xr + static_cast<int64_t>(plane) * span + pix0) = o;
}

// The same repack for stride 2 on both axes without padding (the ResNet
// projections), one thread per 8-pixel group of one output row: output row p
// reads input row 2p, so a group is the even elements of 16 consecutive
// input values, two 16-byte loads issued together.  Groups never cross an
// output row (rows of 28, 14 or 7 pixels end in a shorter group, stored in
// 8-, 4- and 2-byte pieces), so no thread takes the element-by-element path
// of the kernel above except where the loads would run past the end of x.
// The thread holding a plane's last group also zeroes the span's tail.
__global__ __launch_bounds__(256) void repack_s2_rows_kernel(const uint16_t* __restrict__ x, uint16_t* __restrict__ xr,
                                                             int planes, int H, int W, int P, int Q, int span) {
  const int G = (Q + 7) / 8;  // groups per output row
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= planes * P * G) return;
  const int plane = t / (P * G), rem = t - plane * (P * G);
  const int p = rem / G, q0 = (rem - p * G) * 8;
  const int n = Q - q0 < 8 ? Q - q0 : 8;  // pixels of this group
  const int HW = H * W;
  const uint16_t* src = x + static_cast<int64_t>(plane) * HW;
  const int64_t left = static_cast<int64_t>(planes - plane) * HW;  // elements from src to the end of x
  const int64_t in0 = static_cast<int64_t>(2 * p) * W + 2 * q0;
  uint32_t v[8];
  if (in0 + 16 <= left) {
    uint4 ua, ub;
    __builtin_memcpy(&ua, src + in0, 16);
    __builtin_memcpy(&ub, src + in0 + 8, 16);
    v[0] = ua.x & 0xFFFFu; v[1] = ua.y & 0xFFFFu; v[2] = ua.z & 0xFFFFu; v[3] = ua.w & 0xFFFFu;
    v[4] = ub.x & 0xFFFFu; v[5] = ub.y & 0xFFFFu; v[6] = ub.z & 0xFFFFu; v[7] = ub.w & 0xFFFFu;
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = e < n ? src[in0 + 2 * e] : 0u;
  }
  uint16_t* dst = xr + static_cast<int64_t>(plane) * span + p * Q + q0;
  if (n == 8) {
    const uint4 o = make_uint4(v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16), v[6] | (v[7] << 16));
    __builtin_memcpy(dst, &o, 16);
  } else {
    int e = 0;
    if (n - e >= 4) {
      const uint2 o = make_uint2(v[0] | (v[1] << 16), v[2] | (v[3] << 16));
      __builtin_memcpy(dst, &o, 8);
      e = 4;
    }
    if (n - e >= 2) {
      const uint32_t o = v[e] | (v[e + 1] << 16);
      __builtin_memcpy(dst + e, &o, 4);
      e += 2;
    }
    if (n - e >= 1) dst[e] = static_cast<uint16_t>(v[e]);
  }
  if (p == P - 1 && q0 + n == Q)
    for (int e = P * Q; e < span; ++e) xr[static_cast<int64_t>(plane) * span + e] = 0;
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
  split_chunks(tiles, a.nch, &a.e.splits, &a.chunks_per_split);
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
  a.Cg = (int)s.Cg; a.Kg = (int)s.Kg; a.G = s.G;
  a.e.K = (int)s.K; a.e.Kg = (int)s.Kg; a.e.relu = s.relu ? 1 : 0; a.e.PQ = (int)(s.P * s.Q);
  a.e.span = a.e.PQ;
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
      const size_t stage = (size_t)4 * 32 * (BN / 2) * sizeof(float);  // epilogue staging
      if (lds < stage) lds = stage;
      if (lds > limit) continue;
      pl.NG = ng;
      pl.lds = lds;
      a.nch = (int)((s.Cg + UE * ng - 1) / (UE * ng));
      pl.wp_bytes = (size_t)s.G * a.nch * a.Kpad * a.units * 16;
      if (pl.wp_bytes > (size_t)kMaxLaunchBytes) return false;
      choose_splits(s, pl);
      a.e.slab = (int)((N1 * s.K * s.P * s.Q + 3) & ~(int64_t)3);
      pl.part_bytes = a.e.splits > 1 ? (size_t)a.e.splits * a.e.slab * sizeof(float) : 0;
      return true;
    }
  }
  return false;
}

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
  const dim3 grid((a.NPQ + BN - 1) / BN, a.ktiles * a.G, a.e.splits);
  hipLaunchKernelGGL(kern, grid, dim3(kThreads), pl.lds, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.e.splits == 1) return e;
  const int total = a.N * a.K * a.P * a.Q;
  hipLaunchKernelGGL(splitk_reduce_kernel<T>, dim3(reduce_blocks(total)), dim3(256), 0, stream,
                     a.e.partial, reinterpret_cast<const T*>(a.e.b), reinterpret_cast<T*>(a.e.y), total, a.e.slab,
                     a.P * a.Q, a.K, a.e.splits, a.e.relu, reinterpret_cast<const T*>(a.e.res));
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
                      hipStream_t stream, const void* res) {
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
    if (cur.a.e.splits > 1 && !part) return hipErrorInvalidValue;
    IgArgs a = cur.a;
    a.x = reinterpret_cast<const T*>(x) + n0 * img_elems;
    a.e.y = reinterpret_cast<T*>(y) + n0 * out_elems;
    a.e.res = res ? reinterpret_cast<const T*>(res) + n0 * out_elems : nullptr;
    a.x_bytes = (uint32_t)(cnt * img_elems * s.esize());
    a.wp = wp;
    a.wp_bytes = (uint32_t)pl.wp_bytes;
    a.e.b = b;
    a.e.partial = part;
    a.e.NPQ = a.NPQ;
    a.e.vec = store_piece(s, a.e.y);
    hipError_t e;
    if (pl.BM == 64)
      e = pl.NG == 2 ? launch_rst<T, 64, 2>(cur, a, stream) : launch_rst<T, 64, 1>(cur, a, stream);
    else
      e = pl.NG == 2 ? launch_rst<T, 128, 2>(cur, a, stream) : launch_rst<T, 128, 1>(cur, a, stream);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// ---- 1x1 layers ----

struct PwPlan {
  int BM;
  bool gather;
  bool dma;              // bf16: the LDS-DMA kernel
  bool repack;           // ... on a repacked input (see repack_plane_kernel)
  bool ub4;              // ... reading pixel pairs in place (4-byte DMA units)
  bool img;              // ... or, 14 x 14 planes with enough images, whole-image tiles (pointwise_img_kernel)
  int span;              // pixels per image of the tile index space
  size_t repack_bytes;   // repacked input of one launch
  int64_t images_per_launch;
  size_t part_bytes;
  size_t lds;
  PwArgs a;
};

template <typename T>
bool make_pw_plan(const Shape& s, PwPlan& pl, int64_t N1 = -1, bool allow_dma = true, bool allow_img = true) {
  constexpr int UE = elem<T>::per16;
  if (s.R != 1 || s.S != 1 || s.G != 1 || s.C % UE != 0) return false;
  // bf16: the DMA kernel, on the input as it is when the layer is
  // unstrided and unpadded and its plane a multiple of 8 pixels (16-byte
  // units) or of 2 (4-byte units: pixel pairs, as on 14 x 14 planes), else
  // on a repacked copy (plane = P*Q rounded up to 8).
  pl.dma = sizeof(T) == 2 && allow_dma;
  const bool plain = s.sh == 1 && s.sw == 1 && s.ph == 0 && s.pw == 0;
  // (In place as pixel pairs only for planes of at least 8 pixels: the
  // epilogue's runs of 8 may cross one image boundary, not several.)
  pl.ub4 = pl.dma && plain && (s.H * s.W) % 8 != 0 && (s.H * s.W) % 2 == 0 && s.H * s.W > 8;
  pl.repack = pl.dma && !(plain && (s.H * s.W) % 8 == 0) && !pl.ub4;
  pl.span = pl.repack ? (int)((s.P * s.Q + 7) / 8 * 8) : pl.dma ? (int)(s.H * s.W) : (int)(s.P * s.Q);
  int64_t img_bytes = s.C * s.H * s.W * s.esize();
  if (pl.repack && s.C * pl.span * s.esize() > img_bytes) img_bytes = s.C * pl.span * s.esize();
  if (img_bytes > kMaxLaunchBytes || s.K * s.C * s.esize() > kMaxLaunchBytes) return false;
  if (N1 < 0) {
    N1 = kMaxLaunchBytes / img_bytes;
    if (N1 > s.N) N1 = s.N;
    if (N1 < 1) N1 = 1;
  }
  pl.images_per_launch = N1;
  PwArgs& a = pl.a;
  a.C = (int)s.C; a.H = (int)s.H; a.W = (int)s.W;
  a.HW = pl.dma ? pl.span : (int)(s.H * s.W);
  a.P = (int)s.P; a.Q = (int)s.Q; a.sh = s.sh; a.sw = s.sw; a.ph = s.ph; a.pw = s.pw;
  a.NPQ = (int)(N1 * (pl.dma ? pl.span : s.P * s.Q));
  // fp32 takes the 64-row tile at every K: its matrix cores run at a
  // sixteenth of the bf16 rate, so rows past K in a 128-row tile (K = 144,
  // 160, 192, 320 in MobileNetV2) cost more than the 64-row tile's extra
  // input reads, and two of its workgroups share a CU (MobileNetV2's 1x1
  // layers at N = 64: 1246 -> 1084 us over the unique layers).
  pl.BM = pl.dma || (sizeof(T) == 2 && s.K > 64) ? 128 : 64;
  a.ktiles = (int)((s.K + pl.BM - 1) / pl.BM);
  a.ptiles = (a.NPQ + BN - 1) / BN;
  a.nch = (int)((s.C + kPwUnits * UE - 1) / (kPwUnits * UE));
  pl.gather = !(s.sh == 1 && s.sw == 1 && s.ph == 0 && s.pw == 0 && (s.H * s.W) % 4 == 0);
  pl.repack_bytes = pl.repack ? (size_t)N1 * s.C * pl.span * s.esize() : 0;
  if (pl.dma) {
    // Split the channel chunks S ways only where the shorter walk saves
    // more than the split costs: estimated rounds x chunks x 0.5 us per
    // 64-channel chunk, plus, when split, the reduction's launch (3 us)
    // and the fp32 partial sums written and read back at about 5 TB/s.
    // (ResNet-50 at N = 32: the 7^2 2048 -> 512 layer splits four ways,
    // 21.5 us against 28.2 unsplit; the 14^2 1024 -> 256 layer does not,
    // 19.2 us against 21.5 split two ways.)
    const int64_t tiles = (int64_t)a.ptiles * a.ktiles;
    double best = 0;
    for (int S = 1; S <= 8 && S <= a.nch; S *= 2) {
      const int cps = (a.nch + S - 1) / S;
      if ((a.nch + cps - 1) / cps != S) continue;
      double t = (double)((tiles * S + kCUs - 1) / kCUs) * cps * 0.5;
      if (S > 1) t += 3.0 + (double)S * N1 * s.P * s.Q * s.K * 8.0 / 5e6;
      if (S == 1 || t < best) {
        best = t;
        a.e.splits = S;
        a.chunks_per_split = cps;
      }
    }
  } else {
    split_chunks((int64_t)a.ptiles * a.ktiles, a.nch, &a.e.splits, &a.chunks_per_split);
  }
  // 14 x 14 planes: whole-image tiles when the images and channel tiles
  // fill most of the CUs in one unsplit round (ResNet-50's 256 -> 1024
  // layers at batch 32: 256 units of 4 chunks, against 392 units of the
  // pixel-pair kernel); the rows of one image's 128 channels are then one
  // contiguous run of the output.
  pl.img = allow_img && pl.ub4 && s.H * s.W == 196 && s.K % 32 == 0 && N1 * a.ktiles >= 192 && N1 * a.ktiles <= 2 * kCUs;
  if (pl.img) {
    a.ptiles = (int)N1;
    a.e.splits = 1;
    a.chunks_per_split = a.nch;
  }
  a.e.K = (int)s.K; a.e.Kg = (int)s.K; a.e.PQ = (int)(s.P * s.Q); a.e.relu = s.relu ? 1 : 0;
  a.e.NPQ = a.NPQ;
  a.e.span = pl.dma ? pl.span : (int)(s.P * s.Q);
  a.e.slab = (int)((N1 * s.K * s.P * s.Q + 3) & ~(int64_t)3);
  pl.part_bytes = a.e.splits > 1 ? (size_t)a.e.splits * a.e.slab * sizeof(float) : 0;
  const size_t tiles = (size_t)(pl.BM + BN) * kPwUnits * 16;
  const size_t stage = (size_t)4 * 32 * (BN / 2) * sizeof(float);  // epilogue staging
  pl.lds = tiles > stage ? tiles : stage;
  if (pl.dma) pl.lds = (size_t)(kDmaStages + 1) * kDmaStageBytes;
  if (pl.img) pl.lds = (size_t)kImgStages * kImgStageBytes + (size_t)4 * 16 * 196 * 2;
  return true;
}

// Persistent grid of the 1x1 kernel: a multiple of 8 workgroups (one per
// XCD slot), as many as fit on the CUs at once (the 128-row tile holds one
// workgroup per CU, the 64-row tile two).
constexpr int kPwStages = 2;

// The DMA kernel keeps kDmaStages chunks of 32 KiB in LDS: workgroups per
// CU = 160 KiB / (kDmaStages * 32 KiB).
int pw_dma_grid(const PwArgs& a) {
  const int units = a.ptiles * a.ktiles * a.e.splits;
  const int g = (units + 7) / 8 * 8;
  const int resident = kCUs * (int)(kLdsLimit / ((size_t)(kDmaStages + 1) * kDmaStageBytes));
  return g < resident ? g : resident;
}

int pw_grid(const PwArgs& a, int BM) {
  const int units = a.ptiles * a.ktiles * a.e.splits;
  const int g = (units + 7) / 8 * 8;
  const int resident = kCUs * (BM == 64 ? 2 : 1);
  return g < resident ? g : resident;
}

template <int UB>
hipError_t pw_dma_launch(const PwPlan& pl, const PwArgs& a, hipStream_t stream) {
  const auto kern = pointwise_dma_kernel<UB, kDmaStages, kDmaLoaders>;
  static std::atomic<int> lds_raised{0};
  if (!lds_raised.load()) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsLimit);
    if (e != hipSuccess) return e;
    lds_raised.store(1);
  }
  const dim3 grid((unsigned)pw_dma_grid(a));
  hipLaunchKernelGGL(kern, grid, dim3((4 + kDmaLoaders) * 64), pl.lds, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.e.splits == 1) return e;
  // Outputs: images x K x P*Q (a.NPQ counts the padded pixel span).
  const int total = (int)((int64_t)(a.NPQ / a.e.span) * a.e.PQ * a.e.K);
  hipLaunchKernelGGL(splitk_reduce_kernel<bf16_t>, dim3(reduce_blocks(total)), dim3(256), 0, stream,
                     a.e.partial, reinterpret_cast<const bf16_t*>(a.e.b), reinterpret_cast<bf16_t*>(a.e.y), total,
                     a.e.slab, a.e.PQ, a.e.K, a.e.splits, a.e.relu, reinterpret_cast<const bf16_t*>(a.e.res));
  return hipGetLastError();
}

hipError_t pw_img_launch(const PwPlan& pl, const PwArgs& a, hipStream_t stream) {
  const auto kern = pointwise_img_kernel<7>;
  static std::atomic<int> lds_raised{0};
  if (!lds_raised.load()) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsLimit);
    if (e != hipSuccess) return e;
    lds_raised.store(1);
  }
  const int g = (a.ptiles * a.ktiles + 7) / 8 * 8;
  hipLaunchKernelGGL(kern, dim3((unsigned)(g < kCUs ? g : kCUs)), dim3(8 * 64), pl.lds, stream, a);
  return hipGetLastError();
}

template <typename T, int BM, bool GATHER>
hipError_t pw_launch(const PwPlan& pl, const PwArgs& a, hipStream_t stream) {
  const dim3 grid((unsigned)pw_grid(a, BM));
  hipLaunchKernelGGL((pointwise_gemm_kernel<T, BM, GATHER, kPwStages>), grid, dim3(kThreads), pl.lds, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.e.splits == 1) return e;
  const int total = (int)((int64_t)a.NPQ * a.e.K);
  hipLaunchKernelGGL(splitk_reduce_kernel<T>, dim3(reduce_blocks(total)), dim3(256), 0, stream,
                     a.e.partial, reinterpret_cast<const T*>(a.e.b), reinterpret_cast<T*>(a.e.y), total, a.e.slab,
                     a.e.PQ, a.e.K, a.e.splits, a.e.relu, reinterpret_cast<const T*>(a.e.res));
  return hipGetLastError();
}

template <typename T>
hipError_t pw_main_typed(const Shape& s, const void* x, const void* w, const void* b, void* y, void* part_ws,
                         const void* res, hipStream_t stream) {
  PwPlan pl;
  if (!make_pw_plan<T>(s, pl)) return hipErrorInvalidValue;
  if (reinterpret_cast<uintptr_t>(w) % 16 != 0) return hipErrorInvalidValue;
  // An unaligned input that would be read in place cannot go through the
  // DMA: those calls take the register-transposing kernel.
  if (pl.dma && !pl.repack && reinterpret_cast<uintptr_t>(x) % (pl.ub4 ? 4 : 16) != 0 &&
      !make_pw_plan<T>(s, pl, -1, false))
    return hipErrorInvalidValue;
  // Whole-image tiles store 16-byte runs and read the input by 16-byte DMA:
  // other alignments take the pixel-pair kernel.
  const bool img_ok = reinterpret_cast<uintptr_t>(x) % 16 == 0 && reinterpret_cast<uintptr_t>(y) % 16 == 0 &&
                      reinterpret_cast<uintptr_t>(res) % 16 == 0;
  if (pl.img && !img_ok && !make_pw_plan<T>(s, pl, -1, true, false)) return hipErrorInvalidValue;
  char* ws = reinterpret_cast<char*>(part_ws);
  const int64_t img_elems = s.C * s.H * s.W, out_elems = s.K * s.P * s.Q;
  for (int64_t n0 = 0; n0 < s.N; n0 += pl.images_per_launch) {
    const int64_t cnt = s.N - n0 < pl.images_per_launch ? s.N - n0 : pl.images_per_launch;
    PwPlan cur = pl;
    if (cnt != pl.images_per_launch && !make_pw_plan<T>(s, cur, cnt, pl.dma, img_ok)) return hipErrorInvalidValue;
    if ((cur.repack || cur.a.e.splits > 1) && !ws) return hipErrorInvalidValue;
    PwArgs a = cur.a;
    a.x = reinterpret_cast<const T*>(x) + n0 * img_elems;
    a.w = w;
    a.x_bytes = (uint32_t)(cnt * img_elems * s.esize());
    a.w_bytes = (uint32_t)(s.K * s.C * s.esize());
    a.e.y = reinterpret_cast<T*>(y) + n0 * out_elems;
    a.e.res = res ? reinterpret_cast<const T*>(res) + n0 * out_elems : nullptr;
    a.e.b = b;
    a.e.partial = reinterpret_cast<float*>(ws + align256(cur.repack_bytes));
    a.e.vec = store_piece(s, a.e.y);
    const int64_t y_bytes = cnt * out_elems * s.esize();
    a.e.y_bytes = y_bytes < ((int64_t)1 << 31) ? (uint32_t)y_bytes : 0u;
    hipError_t e;
    if (cur.dma) {
      if (cur.repack) {
        const int planes = (int)(cnt * s.C);
        if (s.sh == 2 && s.sw == 2 && s.ph == 0 && s.pw == 0) {
          const int threads = planes * (int)s.P * (int)((s.Q + 7) / 8);
          hipLaunchKernelGGL(repack_s2_rows_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, stream,
                             reinterpret_cast<const uint16_t*>(a.x), reinterpret_cast<uint16_t*>(ws), planes,
                             (int)s.H, (int)s.W, (int)s.P, (int)s.Q, cur.span);
        } else {
          const int threads = planes * (cur.span / 8);
          hipLaunchKernelGGL(repack_plane_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, stream,
                             reinterpret_cast<const uint16_t*>(a.x), reinterpret_cast<uint16_t*>(ws), planes,
                             (int)s.H, (int)s.W, (int)s.P, (int)s.Q, s.sh, s.sw, s.ph, s.pw, cur.span);
        }
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        a.x = ws;
        a.x_bytes = (uint32_t)(cnt * s.C * cur.span * s.esize());
      }
      e = cur.img ? pw_img_launch(cur, a, stream)
                  : cur.ub4 ? pw_dma_launch<4>(cur, a, stream) : pw_dma_launch<16>(cur, a, stream);
    } else {
      // Pixel-quad loads need the input aligned to 4 elements.
      const bool gather = cur.gather || reinterpret_cast<uintptr_t>(a.x) % (4 * s.esize()) != 0;
      if (cur.BM == 64)
        e = gather ? pw_launch<T, 64, true>(cur, a, stream) : pw_launch<T, 64, false>(cur, a, stream);
      else
        e = gather ? pw_launch<T, 128, true>(cur, a, stream) : pw_launch<T, 128, false>(cur, a, stream);
    }
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// Input-dependent workspace of a 1x1 layer: the repacked input (DMA kernel,
// 256-byte aligned) followed by the split partial sums, the largest over
// the launches.
template <typename T>
size_t pw_split_bytes(const Shape& s) {
  PwPlan pl;
  if (!make_pw_plan<T>(s, pl)) return 0;
  size_t need = (pl.repack_bytes ? align256(pl.repack_bytes) : 0) + pl.part_bytes;
  const int64_t rem = s.N % pl.images_per_launch;
  if (rem) {
    PwPlan last;
    if (make_pw_plan<T>(s, last, rem)) {
      const size_t n2 = (last.repack_bytes ? align256(last.repack_bytes) : 0) + last.part_bytes;
      if (n2 > need) need = n2;
    }
  }
  // Calls that fall back to the register-transposing kernel (unaligned
  // input) use their own split count.
  PwPlan alt;
  if (make_pw_plan<T>(s, alt, -1, false) && alt.part_bytes > need) need = alt.part_bytes;
  // ... and calls whose operands do not allow whole-image tiles.
  if (pl.img && make_pw_plan<T>(s, alt, -1, true, false)) {
    size_t n2 = (alt.repack_bytes ? align256(alt.repack_bytes) : 0) + alt.part_bytes;
    if (rem) {
      PwPlan last;
      if (make_pw_plan<T>(s, last, rem, true, false)) {
        const size_t n3 = (last.repack_bytes ? align256(last.repack_bytes) : 0) + last.part_bytes;
        if (n3 > n2) n2 = n3;
      }
    }
    if (n2 > need) need = n2;
  }
  return need;
}

template <typename T>
std::string pw_describe(const Shape& s) {
  PwPlan pl;
  make_pw_plan<T>(s, pl);
  char buf[512];
  const char* tn = sizeof(T) == 2 ? "bf16" : "f32";
  if (pl.img) {
    snprintf(buf, sizeof(buf),
             "implicit_gemm kernels=pointwise_img_kernel<7> tile=128x196 units=%dx%d grid=%d chunk=64 lds=%zu "
             "images_per_launch=%lld (1x1: filters used as given; whole-image tiles, channel-row pairs by 16-byte "
             "DMA)",
             pl.a.ptiles, pl.a.ktiles, std::min(kCUs, (pl.a.ptiles * pl.a.ktiles + 7) / 8 * 8), pl.lds,
             (long long)pl.images_per_launch);
    return buf;
  }
  if (pl.dma) {
    snprintf(buf, sizeof(buf),
             "implicit_gemm kernels=%spointwise_dma_kernel<%d,%d,%d>%s tile=128x%d units=%dx%dx%d grid=%d chunk=64 "
             "span=%d lds=%zu images_per_launch=%lld (1x1: filters used as given)",
             !pl.repack ? ""
             : s.sh == 2 && s.sw == 2 && s.ph == 0 && s.pw == 0 ? "repack_s2_rows_kernel;"
                                                                 : "repack_plane_kernel;",
             pl.ub4 ? 4 : 16, kDmaStages, kDmaLoaders,
             pl.a.e.splits > 1 ? ";splitk_reduce_kernel" : "",
             BN, pl.a.ptiles, pl.a.ktiles, pl.a.e.splits, pw_dma_grid(pl.a), pl.span, pl.lds,
             (long long)pl.images_per_launch);
    return buf;
  }
  snprintf(buf, sizeof(buf),
           "implicit_gemm kernels=pointwise_gemm_kernel<%s,%d,%d,%d>%s tile=%dx%d units=%dx%dx%d grid=%d "
           "chunk=%d lds=%zu images_per_launch=%lld (1x1: filters used as given)",
           tn, pl.BM, pl.gather ? 1 : 0, kPwStages, pl.a.e.splits > 1 ? ";splitk_reduce_kernel" : "", pl.BM, BN,
           pl.a.ptiles, pl.a.ktiles, pl.a.e.splits, pw_grid(pl.a, pl.BM), kPwUnits * elem<T>::per16, pl.lds,
           (long long)pl.images_per_launch);
  return buf;
}

bool use_pointwise(const Shape& s) {
  PwPlan pl;
  return s.dtype == DT_F32 ? make_pw_plan<float>(s, pl) : make_pw_plan<bf16_t>(s, pl);
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
           tn, tn, pl.BM, pl.NG, pl.RST, pl.a.e.splits > 1 ? ";splitk_reduce_kernel" : "", pl.BM, BN,
           (pl.a.NPQ + BN - 1) / BN, pl.a.ktiles * s.G, pl.a.e.splits, pl.NG * elem<T>::per16, pl.a.VR, pl.lds,
           (long long)pl.images_per_launch);
  return buf;
}

}  // namespace

bool implicit_gemm_fits(const Shape& s) {
  if (use_pointwise(s) || rows_applies(s) || k3_applies(s) || ws_applies(s)) return true;
  IgPlan pl;
  if (s.dtype == DT_F32) return make_plan<float>(s, pl);
  return make_plan<bf16_t>(s, pl);
}

size_t implicit_gemm_packed_bytes(const Shape& s) {
  if (use_pointwise(s)) return (size_t)(s.K * s.C * s.esize());  // a plain copy of the filters
  if (rows_applies(s)) return rows_packed_bytes(s);
  if (k3_applies(s)) return k3_uses_package(s) ? k3_package_bytes(s) : (size_t)(s.K * s.C * 9 * 2);
  if (ws_applies(s)) return ws_packed_bytes(s);
  IgPlan pl;
  const bool ok = s.dtype == DT_F32 ? make_plan<float>(s, pl) : make_plan<bf16_t>(s, pl);
  return ok ? pl.wp_bytes : 0;
}

size_t implicit_gemm_split_bytes(const Shape& s) {
  if (rows_applies(s)) return 0;
  if (k3_applies(s)) return k3_split_bytes(s);
  if (ws_applies(s)) return ws_split_bytes(s);
  if (use_pointwise(s)) return s.dtype == DT_F32 ? pw_split_bytes<float>(s) : pw_split_bytes<bf16_t>(s);
  return s.dtype == DT_F32 ? split_bytes_typed<float>(s) : split_bytes_typed<bf16_t>(s);
}

size_t implicit_gemm_workspace(const Shape& s) {
  return align256(implicit_gemm_packed_bytes(s)) + implicit_gemm_split_bytes(s);
}

hipError_t launch_implicit_pack(const Shape& s, const void* w, void* wp, hipStream_t stream) {
  if (rows_applies(s)) return rows_pack(s, w, wp, stream);
  if (k3_applies(s) && k3_uses_package(s)) return k3_pack(s, w, wp, stream);
  if (k3_applies(s) || use_pointwise(s)) return launch_copy(w, wp, implicit_gemm_packed_bytes(s), stream);
  if (ws_applies(s)) return ws_pack(s, w, wp, stream);
  return s.dtype == DT_F32 ? pack_typed<float>(s, w, wp, stream) : pack_typed<bf16_t>(s, w, wp, stream);
}

hipError_t launch_implicit_main(const Shape& s, const void* x, const void* wp, const void* b, void* y, void* part,
                                hipStream_t stream, const void* res) {
  if (rows_applies(s)) return rows_main(s, x, wp, b, y, stream, res);
  if (k3_applies(s)) return k3_main(s, x, wp, b, y, part, stream, res, true);
  if (ws_applies(s)) return ws_main(s, x, wp, b, y, part, stream, res);
  if (use_pointwise(s))
    return s.dtype == DT_F32 ? pw_main_typed<float>(s, x, wp, b, y, part, res, stream)
                             : pw_main_typed<bf16_t>(s, x, wp, b, y, part, res, stream);
  return s.dtype == DT_F32 ? main_typed<float>(s, x, wp, b, y, part, stream, res)
                           : main_typed<bf16_t>(s, x, wp, b, y, part, stream, res);
}

hipError_t launch_implicit_gemm(const Shape& s, const void* x, const void* w, const void* b, void* y, void* ws,
                                hipStream_t stream) {
  char* part = ws ? reinterpret_cast<char*>(ws) + align256(implicit_gemm_packed_bytes(s)) : nullptr;
  // A 1x1 layer reads its filters as given when they are 16-byte aligned;
  // otherwise (and for every other layer) the package is built in the
  // workspace first.
  if (use_pointwise(s) && reinterpret_cast<uintptr_t>(w) % 16 == 0) return launch_implicit_main(s, x, w, b, y, part, stream);
  if (k3_applies(s)) {
    // The filters as given (a copy in the workspace when they are not
    // 16-byte aligned), regrouped inside the kernel.
    const void* wk = w;
    if (reinterpret_cast<uintptr_t>(w) % 16 != 0) {
      if (!ws) return hipErrorInvalidValue;
      hipError_t e = launch_copy(w, ws, (size_t)(s.K * s.C * 9 * 2), stream);
      if (e != hipSuccess) return e;
      wk = ws;
    }
    return k3_main(s, x, wk, b, y, part, stream, nullptr, false);
  }
  if (!ws) return hipErrorInvalidValue;
  hipError_t e = launch_implicit_pack(s, w, ws, stream);
  if (e != hipSuccess) return e;
  return launch_implicit_main(s, x, ws, b, y, part, stream);
}

std::string implicit_gemm_describe(const Shape& s) {
  if (rows_applies(s)) return rows_describe(s);
  if (k3_applies(s)) {
    std::string d = k3_describe(s);
    if (k3_uses_package(s)) {
      const std::string p = k3_describe(s, true);
      const size_t a = p.find("conv3x3_kernel"), b = p.find(' ', a);
      d += " prepacked_kernel=" + p.substr(a, b - a);
    }
    return d;
  }
  if (ws_applies(s)) return ws_describe(s);
  if (use_pointwise(s)) return s.dtype == DT_F32 ? pw_describe<float>(s) : pw_describe<bf16_t>(s);
  return s.dtype == DT_F32 ? describe_typed<float>(s) : describe_typed<bf16_t>(s);
}

}  // namespace convsel
