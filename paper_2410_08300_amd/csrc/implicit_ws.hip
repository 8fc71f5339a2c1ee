// Implicit GEMM (paper, Sec. V-B item (b)) for bf16 layers with nine filter
// taps (3x3, any stride, padding and dilation, one group), with loader and
// compute waves.
//
// The operation is that of implicit_gemm_kernel: output channels as rows,
// flattened (n, p, q) pixels as columns, a 128-pixel tile whose input rows
// (the halo) are staged channel-innermost in LDS, so that every tap of every
// pixel is one 16-byte LDS read of 8 channels.  What differs is where the
// operands travel.  A 3x3 filter tile is nine times larger per channel than
// its halo, and LDS bandwidth, not MFMA, bounded the design that staged both:
// here only the halo goes through LDS.  In a workgroup of 8 waves, waves 4..7
// load each 16-channel chunk's halo as pairs of pixels (one 32-bit load gives
// two pixels of one channel), transpose it in registers and write it to one
// of two LDS stages, one chunk ahead of the compute waves, with the next
// chunk's loads already in flight.  Waves 0..3 multiply; each owns 32 filter
// rows (BM = 128) or 32 rows x 64 pixels (BM = 64) and loads its filter
// fragments straight from the (L2-resident) package into registers, one tap
// at a time and one chunk ahead, so no filter byte is read twice per CU.
#include <stdio.h>

#include <atomic>
#include <string>

#include "common.hpp"
#include "igemm_common.hpp"
#include "kernels.hpp"

namespace convsel {

namespace {

using namespace igemm;

constexpr int kWsNG = 2;          // 8-channel groups per chunk (16 channels)
constexpr int kWsTaps = 9;
constexpr int kWsUnits = kWsTaps * kWsNG;  // 16-byte filter units per row and chunk
constexpr int kWsUR = kWsUnits | 1;        // LDS / package row stride (odd)
constexpr int kWsPS = kWsNG | 1;           // halo pixel stride in units (odd)
constexpr int kWsMaxH = 4;                 // halo items per loader lane per chunk
// One 32-row fragment per compute wave (4 x 1 layout at BM = 128): two
// fragments per wave (2 x 2) halve the LDS operand reads but duplicate the
// filter loads of each wave pair, and measured 10-20% slower.
constexpr int kWsMW128 = 1;

struct WsArgs {
  const void* x;        // first image of this launch
  const void* wp;       // package: [chunk][Kpad][kWsUR] units of 8 bf16
  uint32_t x_bytes, wp_bytes;
  int N, C, H, W, K, S, P, Q;
  int sh, sw, ph, pw, dh, dw;
  int Hv, Wv, VR, NPQ;
  int Kpad, nch, chunks_per_split;
  int npr;              // items per halo row: pixel pairs (PAIR) or pixels
  int items;            // halo items per chunk: VR * npr * kWsNG
  int nh;               // items per loader lane: ceil(items / 256) <= kWsMaxH
  int stage_bytes;      // one halo stage: VR * Wv * kWsPS units, rounded up to 256 bytes
  EpiArgs e;
};

__device__ __forceinline__ int ws_vrow(int j, const WsArgs& a) {
  const int PQ = a.P * a.Q;
  const int n = j / PQ, pq = j - n * PQ;
  return n * a.Hv + (pq / a.Q) * a.sh;
}

// PAIR: the halo is read as pixel pairs (W even: a pair at an even input
// column is one aligned 32-bit word per channel); otherwise pixel by pixel.
// MW: 32-row filter fragments per compute wave (its rows: 32 MW).
template <int BM, bool PAIR, int MW>
__global__ __launch_bounds__(2 * kThreads) void implicit_ws_kernel(WsArgs a) {
  extern __shared__ __align__(16) vec16 smem[];
  char* lds = reinterpret_cast<char*>(smem);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int j0 = blockIdx.x * BN;
  const int k0 = blockIdx.y * BM;
  const int split = blockIdx.z;
  const int ch_begin = split * a.chunks_per_split;
  const int nchunks = min(a.nch, ch_begin + a.chunks_per_split) - ch_begin;
  const int vr_lo = ws_vrow(j0, a);

  if (wave >= 4) {
    // ---------------- loader waves ----------------
    const int lt = tid - 4 * 64;
    const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, a.x_bytes);
    const uint32_t plane = static_cast<uint32_t>(a.H * a.W * 2);

    // Halo items of this lane: t-th item it = lt + 256 t.  Byte offset of
    // its channel 0 (x_bytes: outside the image, reads zero), halo position
    // of its (first) pixel, channel group, and whether the first and (PAIR)
    // second pixel lie inside the halo row.
    uint32_t hvo[kWsMaxH];
    int hpix[kWsMaxH], hcg[kWsMaxH];
    bool h1[kWsMaxH], h2[kWsMaxH];
#pragma unroll
    for (int t = 0; t < kWsMaxH; ++t) {
      const int it = lt + t * 256;
      hvo[t] = a.x_bytes;
      hpix[t] = 0;
      hcg[t] = 0;
      h1[t] = false;
      h2[t] = false;
      if (t < a.nh && it < a.items) {
        const int per_cg = a.VR * a.npr;
        const int cg = it / per_cg, rem = it - cg * per_cg;
        const int vr = rem / a.npr, pr = rem - vr * a.npr;
        const int vc = PAIR ? 2 * pr - (a.pw & 1) : pr;  // PAIR: input column of the pair is even
        const int v = vr_lo + vr;
        const int n = v / a.Hv, ih = v - n * a.Hv - a.ph, iw = vc - a.pw;
        const bool in = n < a.N && ih >= 0 && ih < a.H && iw >= 0 && iw + (PAIR ? 1 : 0) < a.W;
        if (in) hvo[t] = static_cast<uint32_t>(((n * a.C + cg * 8) * a.H + ih) * a.W + iw) * 2;
        hcg[t] = cg;
        hpix[t] = vr * a.Wv + vc;
        h1[t] = vc >= 0;  // with odd left padding the first pair starts one column left of the halo
        h2[t] = PAIR && vc + 1 < a.Wv;
      }
    }
    uint32_t hd[kWsMaxH][8];
    // Channel c0 + e of an item lies at its channel-0 offset plus
    // (c0 + e) * plane: the second part is the same for every lane, so it
    // goes into the load's scalar offset and the per-lane offset stays fixed
    // for the whole tile.  Only the last, partial chunk checks channels per
    // lane.  An item outside the image has offset x_bytes, which stays past
    // the buffer's end whatever is added.
    auto issue_halo = [&](int ch) {
      const int c0 = (ch_begin + ch) * 16;
      const bool tail = c0 + 16 > a.C;
#pragma unroll
      for (int t = 0; t < kWsMaxH; ++t) {
        if (t < a.nh) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const uint32_t so = static_cast<uint32_t>(c0 + e) * plane;
            uint32_t vo = hvo[t];
            if (tail && c0 + hcg[t] * 8 + e >= a.C) vo = a.x_bytes;
            if constexpr (PAIR)
              hd[t][e] = __builtin_amdgcn_raw_buffer_load_b32(xr, vo, so, 0);
            else
              hd[t][e] = __builtin_amdgcn_raw_buffer_load_b16(xr, vo, so, 0);
          }
        }
      }
    };
    auto write_halo = [&](int st) {
      u32x4_t* Xs = reinterpret_cast<u32x4_t*>(lds + st * a.stage_bytes);
#pragma unroll
      for (int t = 0; t < kWsMaxH; ++t) {
        if (t < a.nh) {
          u32x4_t lo, hi;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const uint32_t d0 = hd[t][2 * q], d1 = hd[t][2 * q + 1];
            lo[q] = (d0 & 0xFFFFu) | (d1 << 16);
            hi[q] = (d0 >> 16) | (d1 & 0xFFFF0000u);
          }
          const int pix = hpix[t];
          if (h1[t]) Xs[pix * kWsPS + hcg[t]] = lo;
          if (PAIR && h2[t]) Xs[(pix + 1) * kWsPS + hcg[t]] = hi;
        }
      }
    };

    // Prologue: chunk 0 in stage 0, chunk 1's halo in flight.
    issue_halo(0);
    CONVSEL_WAIT_VMCNT(0);
    write_halo(0);
    if (nchunks > 1) issue_halo(1);
    // The loaders' LDS writes are ordered before each barrier by an explicit
    // lgkmcnt(0) wait; the empty asm statements keep the compiler from
    // moving memory operations across the waits and barriers.
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): the halo writes are done
    for (int i = 0; i < nchunks; ++i) {
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_barrier();  // A(i): chunk i visible to the compute waves
      asm volatile("" ::: "memory");
      if (i + 1 < nchunks) {
        // Chunk i+1's halo into the stage freed at B(i-1), then chunk i+2's
        // loads.  The wait is for all loads issued so far (the halo of i+1),
        // which the compiler can see, so it adds none of its own.
        CONVSEL_WAIT_VMCNT(0);
        write_halo((i + 1) & 1);
        if (i + 2 < nchunks) issue_halo(i + 2);
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_waitcnt(0xc07f);
      }
      // Plain barrier: an LDS fence here would also wait for the halo loads
      // of chunk i+2, which are meant to stay in flight.
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_barrier();  // B(i): compute waves are done with stage i & 1
      asm volatile("" ::: "memory");
    }
    return;
  }

  // ---------------- compute waves ----------------
  // Layout: WM x WN waves, each 32 MW filter rows x (BN / WN) pixels.  With
  // 128 pixels per wave (NJW = 4) the MFMA computes pixels x channels for
  // the channel-row epilogue; otherwise channels x pixels.
  constexpr int WM = BM / (32 * MW), WN = 4 / WM, NJW = BN / 32 / WN;
  static_assert(WM * WN == 4 && (NJW != 4 || MW == 1), "four compute waves");
  const int wm = wave / WN, wn = wave - (wave / WN) * WN;
  const int half = lane >> 5, l32 = lane & 31;
  const int PQ = a.P * a.Q;
  const int jl = min(j0 + BN, a.NPQ) - 1;
  const int col0 = j0 + wn * (BN / WN);
  int pofs[NJW];
#pragma unroll
  for (int nj = 0; nj < NJW; ++nj) {
    const int j = col0 + nj * 32 + l32;
    const int jj = j < a.NPQ ? j : jl;
    const int pq = jj - (jj / PQ) * PQ;
    const int q = pq - (pq / a.Q) * a.Q;
    pofs[nj] = ((ws_vrow(jj, a) - vr_lo) * a.Wv + q * a.sw) * kWsPS + half;
  }
  int tapoff[kWsTaps];
#pragma unroll
  for (int t = 0; t < kWsTaps; ++t) {
    const int r = t / a.S, s = t - r * a.S;
    tapoff[t] = (r * a.dh * a.Wv + s * a.dw) * kWsPS;
  }
  // Filter fragments: lane l of tap t, fragment m reads unit 2t + l/32 of
  // row k0 + 32 (MW wm + m) + l%32 (the package is zero past K and C).
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(a.wp, a.wp_bytes);
  const uint32_t aoff = static_cast<uint32_t>(((k0 + wm * 32 * MW + l32) * kWsUR + half) * 16);
  constexpr uint32_t kFragStride = 32 * kWsUR * 16;  // bytes between 32-row fragments
  auto chunk_soff = [&](int ch) { return static_cast<uint32_t>((ch_begin + ch) * a.Kpad * kWsUR * 16); };
  // At BM = 128 two fragment sets alternate by chunk parity: chunk i+1's
  // fragments are requested into one set before chunk i multiplies with the
  // other (with one set refilled in place the compiler shuffled registers
  // and waited for every outstanding load at the top of each chunk).  At
  // BM = 64 the second set would raise the kernel past 128 VGPRs and halve
  // the workgroups per CU, which costs more: there one set is refilled tap
  // by tap right after its last use.
  constexpr bool kTwoSets = BM == 128;
  u32x4_t afA[kWsTaps][MW], afB[kTwoSets ? kWsTaps : 1][MW];
  {
    const uint32_t so = chunk_soff(0);
#pragma unroll
    for (int t = 0; t < kWsTaps; ++t)
#pragma unroll
      for (int m = 0; m < MW; ++m)
        afA[t][m] = __builtin_amdgcn_raw_buffer_load_b128(wr, aoff + m * kFragStride + 32 * t, so, 0);
  }

  f32x16_t acc[MW][NJW];
#pragma unroll
  for (int m = 0; m < MW; ++m)
#pragma unroll
    for (int nj = 0; nj < NJW; ++nj) acc[m][nj] = zero16();

  // One chunk: LDS stage `par`, fragments `cur`; `nxt` receives chunk i+1's.
  auto chunk = [&](int i, int par, u32x4_t(&cur)[kWsTaps][MW], u32x4_t(&nxt)[kWsTaps][MW]) {
    lds_sync();  // A(i)
    const u32x4_t* Xs = reinterpret_cast<const u32x4_t*>(lds + par * a.stage_bytes);
    const bool more = i + 1 < nchunks;
    const uint32_t so_next = chunk_soff(more ? i + 1 : i);
    if constexpr (kTwoSets) {
      // Requested on every chunk (the last one reloading its own, unused,
      // so that the compiler can count the loads in flight); the scheduling
      // barrier keeps them from being sunk to the end of the chunk.
#pragma unroll
      for (int st = 0; st < kWsTaps; ++st)
#pragma unroll
        for (int m = 0; m < MW; ++m)
          nxt[st][m] = __builtin_amdgcn_raw_buffer_load_b128(wr, aoff + m * kFragStride + 32 * st, so_next, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int st = 0; st < kWsTaps; ++st) {
      // Units 2st (channels 0-7) and 2st+1 (8-15) of tap st: lane half h
      // takes unit 2st+h, i.e. channel group h.
      bf16x8_t bfr[NJW], a0[MW];
#pragma unroll
      for (int nj = 0; nj < NJW; ++nj) bfr[nj] = __builtin_bit_cast(bf16x8_t, Xs[pofs[nj] + tapoff[st]]);
#pragma unroll
      for (int m = 0; m < MW; ++m) a0[m] = __builtin_bit_cast(bf16x8_t, cur[st][m]);
      if constexpr (!kTwoSets) {
        if (more)
#pragma unroll
          for (int m = 0; m < MW; ++m)
            cur[st][m] = __builtin_amdgcn_raw_buffer_load_b128(wr, aoff + m * kFragStride + 32 * st, so_next, 0);
      }
#pragma unroll
      for (int m = 0; m < MW; ++m)
#pragma unroll
        for (int nj = 0; nj < NJW; ++nj)
          acc[m][nj] = NJW == 4 ? __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[nj], a0[m], acc[m][nj], 0, 0, 0)
                                : __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0[m], bfr[nj], acc[m][nj], 0, 0, 0);
    }
    lds_sync();  // B(i)
  };
  if constexpr (kTwoSets) {
    for (int i0 = 0; i0 < nchunks; i0 += 2) {
      chunk(i0, 0, afA, afB);
      if (i0 + 1 < nchunks) chunk(i0 + 1, 1, afB, afA);
    }
  } else {
    for (int i = 0; i < nchunks; ++i) chunk(i, i & 1, afA, afA);
  }
  // The loaders are done with LDS after B of the last chunk: stage there.
  float* stage = reinterpret_cast<float*>(smem) + wave * 32 * 64;
  if constexpr (NJW == 4)
    store_block128t<bf16_t>(acc, stage, a.e, k0 + wm * 32, col0, 0, split);
  else
    store_block<bf16_t, MW, NJW>(acc, stage, a.e, k0 + wm * 32 * MW, col0, 0, split);
}

// Package: unit (ch, kp, u) with u = tap * 2 + cg holds channels
// ch*16 + cg*8 .. +7 of filter kp at that tap; unit 18 of each row and
// everything past K or C is zero.  One thread per (row (ch, kp), channel
// group cg): its source, channels ch*16 + cg*8 .. +7 x 9 taps of filter kp,
// is 72 consecutive elements of w (144 bytes), read as 9 loads of 16 bytes
// when w is 16-byte aligned and C % 16 == 0, and regrouped in registers into
// the group's 9 units.
constexpr int kPackWsThreads = 64;
__global__ __launch_bounds__(kPackWsThreads) void pack_filters_ws_kernel(const uint16_t* __restrict__ w,
                                                                        u32x4_t* __restrict__ wp, int K, int C,
                                                                        int Kpad, int items, int vec) {
  const int item = blockIdx.x * kPackWsThreads + threadIdx.x;
  if (item >= items) return;
  const int cg = item & 1, row = item >> 1;
  const int kp = row % Kpad, ch = row / Kpad;
  u32x4_t* dst = wp + static_cast<int64_t>(row) * kWsUR;
  uint32_t v[72];  // element i = (c - ch*16 - cg*8) * 9 + tap, zero-extended
  if (kp < K && vec) {
    const u32x4_t* src =
        reinterpret_cast<const u32x4_t*>(w + (static_cast<int64_t>(kp) * C + ch * 16 + cg * 8) * kWsTaps);
#pragma unroll
    for (int q = 0; q < 9; ++q) {
      const u32x4_t d = src[q];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[8 * q + 2 * e] = d[e] & 0xFFFFu;
        v[8 * q + 2 * e + 1] = d[e] >> 16;
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < 72; ++i) {
      const int c = ch * 16 + cg * 8 + i / kWsTaps;
      v[i] = kp < K && c < C ? w[(static_cast<int64_t>(kp) * C + c) * kWsTaps + i % kWsTaps] : 0u;
    }
  }
#pragma unroll
  for (int tap = 0; tap < kWsTaps; ++tap) {
    u32x4_t o;
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] = v[(2 * q) * kWsTaps + tap] | (v[(2 * q + 1) * kWsTaps + tap] << 16);
    dst[tap * kWsNG + cg] = o;
  }
  if (cg == 0) dst[kWsUnits] = u32x4_t{0u, 0u, 0u, 0u};
}

struct WsPlan {
  int BM;
  bool pair;
  int64_t images_per_launch;
  size_t wp_bytes, part_bytes, lds;
  WsArgs a;
};

bool make_ws_plan(const Shape& s, WsPlan& pl, int64_t N1 = -1) {
  if (s.dtype != DT_BF16 || s.G != 1 || s.R * s.S != kWsTaps || s.C <= 8) return false;
  if (s.P * s.Q < 8) return false;  // the channel-row epilogue's runs cross at most one image
  const int64_t img_bytes = s.C * s.H * s.W * 2;
  if (img_bytes > kMaxLaunchBytes) return false;
  if (N1 < 0) {
    N1 = kMaxLaunchBytes / img_bytes;
    if (N1 > s.N) N1 = s.N;
    if (N1 < 1) N1 = 1;
  }
  pl.images_per_launch = N1;
  pl.BM = s.K <= 64 ? 64 : 128;
  pl.pair = s.W % 2 == 0;
  WsArgs& a = pl.a;
  a.N = (int)N1; a.C = (int)s.C; a.H = (int)s.H; a.W = (int)s.W; a.K = (int)s.K; a.S = (int)s.S;
  a.P = (int)s.P; a.Q = (int)s.Q;
  a.sh = s.sh; a.sw = s.sw; a.ph = s.ph; a.pw = s.pw; a.dh = s.dh; a.dw = s.dw;
  a.Hv = (int)((s.P - 1) * s.sh + (s.R - 1) * s.dh + 1);
  a.Wv = (int)((s.Q - 1) * s.sw + (s.S - 1) * s.dw + 1);
  a.VR = halo_rows(s, N1, a.Hv);
  a.NPQ = (int)(N1 * s.P * s.Q);
  const int ktiles = (int)((s.K + pl.BM - 1) / pl.BM);
  a.Kpad = ktiles * pl.BM;
  a.nch = (int)((s.C + 15) / 16);
  a.npr = pl.pair ? (a.Wv + (s.pw & 1) + 1) / 2 : a.Wv;
  a.items = a.VR * a.npr * kWsNG;
  a.nh = (a.items + 255) / 256;
  if (a.nh > kWsMaxH) return false;
  a.stage_bytes = (int)(((size_t)a.VR * a.Wv * kWsPS * 16 + 255) / 256 * 256);
  pl.lds = (size_t)2 * a.stage_bytes;
  const size_t staging = (size_t)4 * 32 * 64 * sizeof(float);  // epilogue, after the last chunk
  if (pl.lds < staging) pl.lds = staging;
  if (pl.lds > kLdsLimit) return false;
  pl.wp_bytes = (size_t)a.nch * a.Kpad * kWsUR * 16;
  if (pl.wp_bytes > (size_t)kMaxLaunchBytes) return false;
  const int64_t tiles = (int64_t)((a.NPQ + BN - 1) / BN) * ktiles;
  split_chunks(tiles, a.nch, &a.e.splits, &a.chunks_per_split);
  a.e.K = (int)s.K; a.e.Kg = (int)s.K; a.e.relu = s.relu ? 1 : 0; a.e.PQ = (int)(s.P * s.Q);
  a.e.span = a.e.PQ;
  a.e.NPQ = a.NPQ;
  a.e.slab = (int)((N1 * s.K * s.P * s.Q + 3) & ~(int64_t)3);
  pl.part_bytes = a.e.splits > 1 ? (size_t)a.e.splits * a.e.slab * sizeof(float) : 0;
  return true;
}

template <int BM, bool PAIR, int MW>
hipError_t ws_launch(const WsPlan& pl, const WsArgs& a, hipStream_t stream) {
  const auto kern = implicit_ws_kernel<BM, PAIR, MW>;
  // Raise the dynamic-LDS limit once (calls may be captured into a graph
  // after the first one).
  static std::atomic<int> lds_limit{64 * 1024};
  if ((int)pl.lds > lds_limit.load()) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsLimit);
    if (e != hipSuccess) return e;
    lds_limit.store((int)kLdsLimit);
  }
  const dim3 grid((unsigned)((a.NPQ + BN - 1) / BN), (unsigned)(a.Kpad / BM), (unsigned)a.e.splits);
  hipLaunchKernelGGL(kern, grid, dim3(2 * kThreads), pl.lds, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.e.splits == 1) return e;
  const int total = a.N * a.K * a.P * a.Q;
  hipLaunchKernelGGL(splitk_reduce_kernel<bf16_t>, dim3(reduce_blocks(total)), dim3(256), 0, stream,
                     a.e.partial, reinterpret_cast<const bf16_t*>(a.e.b), reinterpret_cast<bf16_t*>(a.e.y), total,
                     a.e.slab, a.P * a.Q, a.K, a.e.splits, a.e.relu, reinterpret_cast<const bf16_t*>(a.e.res));
  return hipGetLastError();
}

}  // namespace

bool ws_applies(const Shape& s) {
  WsPlan pl;
  return make_ws_plan(s, pl);
}

size_t ws_packed_bytes(const Shape& s) {
  WsPlan pl;
  return make_ws_plan(s, pl) ? pl.wp_bytes : 0;
}

size_t ws_split_bytes(const Shape& s) {
  WsPlan pl;
  if (!make_ws_plan(s, pl)) return 0;
  size_t m = pl.part_bytes;
  const int64_t rest = s.N % pl.images_per_launch;
  if (rest) {
    WsPlan last;
    if (make_ws_plan(s, last, rest) && last.part_bytes > m) m = last.part_bytes;
  }
  return m;
}

hipError_t ws_pack(const Shape& s, const void* w, void* wp, hipStream_t stream) {
  WsPlan pl;
  if (!make_ws_plan(s, pl)) return hipErrorInvalidValue;
  const int items = pl.a.nch * pl.a.Kpad * kWsNG;
  const int vec = s.C % 16 == 0 && reinterpret_cast<uintptr_t>(w) % 16 == 0;
  hipLaunchKernelGGL(pack_filters_ws_kernel, dim3((unsigned)((items + kPackWsThreads - 1) / kPackWsThreads)),
                     dim3(kPackWsThreads), 0, stream, reinterpret_cast<const uint16_t*>(w), reinterpret_cast<u32x4_t*>(wp),
                     (int)s.K, (int)s.C, pl.a.Kpad, items, vec);
  return hipGetLastError();
}

hipError_t ws_main(const Shape& s, const void* x, const void* wp, const void* b, void* y, void* part_ws,
                   hipStream_t stream, const void* res) {
  WsPlan pl;
  if (!make_ws_plan(s, pl)) return hipErrorInvalidValue;
  const int64_t img_elems = s.C * s.H * s.W, out_elems = s.K * s.P * s.Q;
  for (int64_t n0 = 0; n0 < s.N; n0 += pl.images_per_launch) {
    const int64_t cnt = s.N - n0 < pl.images_per_launch ? s.N - n0 : pl.images_per_launch;
    WsPlan cur = pl;
    if (cnt != pl.images_per_launch && !make_ws_plan(s, cur, cnt)) return hipErrorInvalidValue;
    if (cur.a.e.splits > 1 && !part_ws) return hipErrorInvalidValue;
    WsArgs a = cur.a;
    a.x = reinterpret_cast<const uint16_t*>(x) + n0 * img_elems;
    a.x_bytes = (uint32_t)(cnt * img_elems * 2);
    a.wp = wp;
    a.wp_bytes = (uint32_t)cur.wp_bytes;
    a.e.y = reinterpret_cast<uint16_t*>(y) + n0 * out_elems;
    a.e.res = res ? reinterpret_cast<const uint16_t*>(res) + n0 * out_elems : nullptr;
    a.e.b = b;
    a.e.partial = reinterpret_cast<float*>(part_ws);
    a.e.vec = store_piece(s, a.e.y);
    // Pairs of pixels are read as aligned 32-bit words.
    const bool pair = cur.pair && reinterpret_cast<uintptr_t>(a.x) % 4 == 0;
    hipError_t e;
    if (cur.BM == 64)
      e = pair ? ws_launch<64, true, 1>(cur, a, stream) : ws_launch<64, false, 1>(cur, a, stream);
    else
      e = pair ? ws_launch<128, true, kWsMW128>(cur, a, stream) : ws_launch<128, false, kWsMW128>(cur, a, stream);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

std::string ws_describe(const Shape& s) {
  WsPlan pl;
  if (!make_ws_plan(s, pl)) return "implicit_gemm (loader/compute waves): not applicable";
  char buf[448];
  snprintf(buf, sizeof(buf),
           "implicit_gemm kernels=pack_filters_ws_kernel;implicit_ws_kernel<%d,%d,%d>%s tile=%dx%d grid=%dx%dx%d "
           "chunk=16 halo_rows=%d halo_items=%d lds=%zu images_per_launch=%lld (loader waves: halo %s loads "
           "into LDS; compute waves: filters from L2 into registers, MFMA)",
           pl.BM, pl.pair ? 1 : 0, pl.BM == 128 ? kWsMW128 : 1, pl.a.e.splits > 1 ? ";splitk_reduce_kernel" : "", pl.BM, BN,
           (pl.a.NPQ + BN - 1) / BN, pl.a.Kpad / pl.BM, pl.a.e.splits, pl.a.VR, pl.a.items, pl.lds,
           (long long)pl.images_per_launch, pl.pair ? "pixel-pair" : "pixel");
  return buf;
}

}  // namespace convsel
