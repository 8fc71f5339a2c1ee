// Implicit GEMM (paper, Sec. V-B item (b)) for bf16 3x3 layers with stride 1
// or 2, dilation 1, one group and C a multiple of the channel chunk.
//
// The contraction is Y[pixel][k] = sum over (tap, c) of X~[pixel + tap][c] *
// W[k][c][tap]: output pixels (flattened n, p, q) as the MFMA's A rows,
// output channels as its B columns, reduced 16 channels of one tap per
// v_mfma_f32_32x32x16_bf16.  A workgroup owns a tile of TP consecutive
// pixels x TK channels and walks the input channels in chunks of CH.  Per
// chunk, LDS holds
//
//   * the halo: every input row the tile's pixels read, pixel-major (the CH
//     channels of one input pixel are contiguous, 16-byte units XOR-swizzled
//     so that 16 consecutive pixels hit distinct banks), with the zero
//     padding columns in place.  Any tap of any pixel is then one 16-byte LDS
//     read of 8 channels, which is exactly one lane's MFMA operand.  For
//     stride 2 each row is split into its even and odd columns, so that the
//     pixels of one tap are again consecutive slots;
//   * the filters of the tile: [tap][TK][CH], swizzled the same way.
//
// Loader waves (the last kLoaders waves) fill these.  The halo always comes
// from the NCHW input as given: 16-byte loads (8 pixels of one channel; 8
// channels per lane), transposed in registers into 8 pixel vectors.  The
// filters come one of two ways:
//
//   * per call (PK = false), from the KCRS tensor as given: nine 16-byte
//     loads per (filter, 8 channels) -- the 72 consecutive values of 8
//     channels x 9 taps -- regrouped in registers into nine tap vectors.  No
//     packing kernel runs before the convolution.  All four loader waves do
//     both jobs; two LDS stages alternate, and while the compute waves
//     multiply chunk i the loaders write chunk i+1 and have chunk i+2's
//     loads in flight;
//   * prepacked (PK = true), from a package that k3_pack builds once per
//     filter tensor, each (chunk, channel tile) filter tile stored in its
//     LDS order: two loader waves copy it by LDS DMA with no register
//     traffic while the other two transpose the halo, over three LDS stages
//     (the DMA of chunk i+2 goes out while chunk i is multiplied);
//   * prepacked into registers (BG = true), from the same package: each
//     compute wave loads the 16-byte fragments it multiplies straight into
//     registers, a chunk ahead, and all four loader waves stage only the
//     halo (two LDS stages).
//
// Compute waves form a WP x WK grid; each holds MB x NB blocks of 32 x 32
// accumulators (32 MB pixels x 32 NB channels), so that each operand read
// from LDS feeds NB (pixel fragments) or MB (filter fragments) MFMAs.  The
// epilogue adds bias (and the model executor's residual), applies ReLU,
// rounds and stores each lane's runs of four consecutive pixels of one
// channel as 8-byte stores, or stores fp32 partials for a split reduction.
#include <stdio.h>

#include <algorithm>
#include <atomic>
#include <string>
#include <type_traits>

#include "common.hpp"
#include "igemm_common.hpp"
#include "kernels.hpp"

namespace convsel {

namespace {

using namespace igemm;

constexpr int kLoaders = 4;   // loader waves per workgroup
constexpr int kK3Taps = 9;
constexpr int kHSMax = 2;     // halo items per loader lane and chunk (at most)

struct K3Args {
  const void* x;       // first image of this launch
  const void* w;       // filters, K x C x 3 x 3
  uint32_t x_bytes, w_bytes;
  int N, C, H, W, K, P, Q;
  int sh, ph, pw;      // stride (both axes), padding
  int Hp;              // virtual rows per image (at least (P - 1) * sh + 3)
  int E, PE;           // enumerated columns per output row (E >= Q), pixels per image (P * E)
  int NPQ;             // enumerated pixels of the launch: N * P * E
  int ptiles, ktiles;
  int nch, chunks_per_split;
  int VR;              // halo rows staged per chunk
  int RS, PS;          // LDS slots per halo row; stride 2: slots per column-parity plane
  int NG;              // column windows per input row
  int halo_items;      // VR * NG * (CH / 8)
  int halo_bytes;      // one stage's halo, rounded to 256 bytes
  int stage_bytes;     // halo + filter tile
  EpiArgs e;
};

// Bank swizzle of the 16-byte unit u of slot `pos` (a pixel or a filter row
// of UP units): 16 consecutive slots' units land in 16 distinct 16-byte bank
// groups.
template <int UP>
__device__ __forceinline__ int k3_swz(int pos) {
  return (pos / (16 / UP)) & (UP - 1);
}

// Epilogue of one compute wave: NB blocks of 32 channels (channel block nb
// starts at kb0 + 32 nb) x 32 MB pixels (tile pixels col0 ..), in the MFMA
// layout (block (mb, nb), accumulator v of lane l: channel l % 32, pixel
// 32 mb + 8 (v / 4) + 4 (l / 32) + v % 4).  Channel block by channel block,
// the values are rounded (bf16, after bias and ReLU) or kept (fp32 partials
// of a split reduction), staged in this wave's LDS region as
// [channel][pixels] rows of 16-byte units XOR-swizzled by the channel, read
// back as 8-pixel runs and stored with one 16-byte store per run (two for
// fp32) -- every store instruction then covers whole contiguous rows of
// 64 to 512 bytes instead of 32 separate 16-byte pieces.  A run that crosses
// an image boundary or passes the last pixel is stored element by element
// (runs cross at most one boundary: P*Q >= 8).
// Stores the first n (1..7) bf16 values of an 8-value run: 8, 4 and 2-byte
// pieces.
__device__ __forceinline__ void k3_store_head(uint16_t* p, uint32_t d0, uint32_t d1, uint32_t d2, uint32_t d3,
                                              int n) {
  const bool b4 = n >= 4;
  if (b4) {
    const uint2 v = make_uint2(d0, d1);
    __builtin_memcpy(p, &v, 8);
  }
  const int t2 = b4 ? 4 : 0;
  const uint32_t w2 = b4 ? d2 : d0;
  const bool b2 = n - t2 >= 2;
  if (b2) __builtin_memcpy(p + t2, &w2, 4);
  const int t1 = t2 + (b2 ? 2 : 0);
  const uint32_t w1 = t1 == 0 ? d0 : t1 == 2 ? d1 : t1 == 4 ? d2 : d3;
  if (n - t1 >= 1) p[t1] = static_cast<uint16_t>(w1);
}

// Output run of the 8 enumerated pixels col0 + px .. +7 (channel row0).
// With E == Q the enumeration is the output order itself (runs may cross
// rows and one image boundary); with E > Q (E a multiple of 8) a run lies in
// one output row, and its pixels at columns >= Q are padding, not stored.
struct K3Map {
  int E, PE, Q, NPQ;
};
__device__ __forceinline__ Run128t k3_run(const EpiArgs& e, const K3Map& m, int row0, int col0, int px) {
  if (m.E == m.Q) return run128t(e, row0, col0, 0, px);
  Run128t r;
  const int j = col0 + px;
  const int n = j / m.PE, rem = j - n * m.PE;
  const int p = rem / m.E, q = rem - p * m.E;
  r.nvalid = (j < m.NPQ && q < m.Q) ? min(8, m.Q - q) : 0;
  r.wrap = 8;
  r.full = r.nvalid == 8;
  r.o = (static_cast<int64_t>(n) * e.K + row0) * e.PQ + p * m.Q + q;
  return r;
}

template <int MB, int NB>
__device__ __forceinline__ void k3_epilogue(const f32x16_t (&acc)[MB][NB], char* stage, const EpiArgs& e,
                                            const K3Map& m, int kb0, int col0, int split) {
  const int lane = threadIdx.x & 63;
  const int l32 = lane & 31, h = lane >> 5;
  const int PQ = e.PQ;
  const int64_t next_img = static_cast<int64_t>(e.K - 1) * PQ;
  if (e.splits <= 1) {
    constexpr int U = MB * 4;          // 16-byte units per staged channel row (8 pixels each)
    constexpr int RPI = 64 / U;        // rows covered by one pass of the wave
    constexpr int PASSES = 32 / RPI;
    const uint16_t* bias = reinterpret_cast<const uint16_t*>(e.b);
    uint16_t* y = reinterpret_cast<uint16_t*>(e.y);
    const int rrow = lane / U, u = lane % U;
    const Run128t r = k3_run(e, m, kb0, col0, u * 8);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int kb = kb0 + 32 * nb;
      const float bv = (bias && kb + l32 < e.K) ? bf16_to_f32(bias[kb + l32]) : 0.f;
      const bool relu_now = e.relu && !e.res;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float v4[4];
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            v4[t] = acc[mb][nb][4 * g + t] + bv;
            if (relu_now) v4[t] = fmaxf(v4[t], 0.f);
          }
          uint2 w;
          w.x = f32x2_to_bf16x2(v4[0], v4[1]);
          w.y = f32x2_to_bf16x2(v4[2], v4[3]);
          const int px0 = mb * 32 + 8 * g + 4 * h;
          *reinterpret_cast<uint2*>(stage + l32 * (U * 16) + (((px0 >> 3) ^ (l32 & (U - 1))) << 4) +
                                    ((px0 >> 2) & 1) * 8) = w;
        }
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's staging writes are done
      __builtin_amdgcn_wave_barrier();
      uint4 d[PASSES];
#pragma unroll
      for (int it = 0; it < PASSES; ++it) {
        const int row = rrow + RPI * it;
        d[it] = *reinterpret_cast<const uint4*>(stage + row * (U * 16) + ((u ^ (row & (U - 1))) << 4));
      }
      const int64_t ob = r.o + static_cast<int64_t>(kb - kb0) * PQ;
      if (e.res) {
        // Residual add (and the ReLU after it): all rows' residual runs are
        // requested before any is used.
        uint4 rr[PASSES];
        const uint16_t* rp = reinterpret_cast<const uint16_t*>(e.res);
        if (r.full) {
#pragma unroll
          for (int it = 0; it < PASSES; ++it) {
            const int row = rrow + RPI * it;
            rr[it] = make_uint4(0u, 0u, 0u, 0u);
            if (kb + row < e.K) __builtin_memcpy(&rr[it], rp + ob + static_cast<int64_t>(row) * PQ, 16);
          }
        }
#pragma unroll
        for (int it = 0; it < PASSES; ++it) {
          const int row = rrow + RPI * it;
          if (kb + row >= e.K || r.nvalid <= 0) continue;
          const int64_t o = ob + static_cast<int64_t>(row) * PQ;
          const uint32_t w[4] = {d[it].x, d[it].y, d[it].z, d[it].w};
          float v[8];
#pragma unroll
          for (int t = 0; t < 8; ++t) v[t] = __uint_as_float((w[t >> 1] >> (16 * (t & 1))) << 16);
          if (r.full) {
            const uint32_t q[4] = {rr[it].x, rr[it].y, rr[it].z, rr[it].w};
#pragma unroll
            for (int t = 0; t < 8; ++t) v[t] += __uint_as_float((q[t >> 1] >> (16 * (t & 1))) << 16);
          } else {
            add_residual_run<bf16_t>(v, e, o, false, r.nvalid, r.wrap, PQ, next_img);
          }
          if (e.relu)
#pragma unroll
            for (int t = 0; t < 8; ++t) v[t] = fmaxf(v[t], 0.f);
          d[it].x = f32x2_to_bf16x2(v[0], v[1]);
          d[it].y = f32x2_to_bf16x2(v[2], v[3]);
          d[it].z = f32x2_to_bf16x2(v[4], v[5]);
          d[it].w = f32x2_to_bf16x2(v[6], v[7]);
        }
      }
#pragma unroll
      for (int it = 0; it < PASSES; ++it) {
        const int row = rrow + RPI * it;
        if (kb + row >= e.K || r.nvalid <= 0) continue;
        const int64_t o = ob + static_cast<int64_t>(row) * PQ;
        if (r.full) {
          __builtin_memcpy(y + o, &d[it], 16);
        } else if (r.wrap >= 8) {
          k3_store_head(y + o, d[it].x, d[it].y, d[it].z, d[it].w, r.nvalid);
        } else {
          const uint32_t wd[4] = {d[it].x, d[it].y, d[it].z, d[it].w};
#pragma unroll
          for (int t = 0; t < 8; ++t)
            if (t < r.nvalid)
              y[o + t + (t >= r.wrap ? next_img : 0)] = static_cast<uint16_t>(wd[t >> 1] >> (16 * (t & 1)));
        }
      }
      __builtin_amdgcn_wave_barrier();  // the next block reuses the staging rows
    }
    return;
  }
  // fp32 partial sums: rows of 32 MB floats (8 MB units), one 8-pixel run
  // (two units) per lane and pass.
  constexpr int U = MB * 8;
  constexpr int LPR = MB * 4;        // lanes per row
  constexpr int RPI = 64 / LPR;
  constexpr int PASSES = 32 / RPI;
  float* part = e.partial + static_cast<int64_t>(split) * e.slab;
  const int rrow = lane / LPR, c = lane % LPR;
  const Run128t r = k3_run(e, m, kb0, col0, c * 8);
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int kb = kb0 + 32 * nb;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int px0 = mb * 32 + 8 * g + 4 * h;
        const float4 v = make_float4(acc[mb][nb][4 * g], acc[mb][nb][4 * g + 1], acc[mb][nb][4 * g + 2],
                                     acc[mb][nb][4 * g + 3]);
        *reinterpret_cast<float4*>(stage + l32 * (U * 16) + (((px0 >> 2) ^ (l32 & (U - 1))) << 4)) = v;
      }
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();
    float4 lo[PASSES], hi[PASSES];
#pragma unroll
    for (int it = 0; it < PASSES; ++it) {
      const int row = rrow + RPI * it;
      lo[it] = *reinterpret_cast<const float4*>(stage + row * (U * 16) + (((2 * c) ^ (row & (U - 1))) << 4));
      hi[it] = *reinterpret_cast<const float4*>(stage + row * (U * 16) + (((2 * c + 1) ^ (row & (U - 1))) << 4));
    }
    const int64_t ob = r.o + static_cast<int64_t>(kb - kb0) * PQ;
#pragma unroll
    for (int it = 0; it < PASSES; ++it) {
      const int row = rrow + RPI * it;
      if (kb + row >= e.K || r.nvalid <= 0) continue;
      const int64_t o = ob + static_cast<int64_t>(row) * PQ;
      if (r.full) {
        __builtin_memcpy(part + o, &lo[it], 16);
        __builtin_memcpy(part + o + 4, &hi[it], 16);
      } else if (r.wrap >= 8) {
        // the first nvalid floats: 4 (16 bytes), then 2, then 1
        const int nv = r.nvalid;
        const bool b4 = nv >= 4;
        if (b4) __builtin_memcpy(part + o, &lo[it], 16);
        const float qx = b4 ? hi[it].x : lo[it].x, qy = b4 ? hi[it].y : lo[it].y;
        const float qz = b4 ? hi[it].z : lo[it].z;
        const int t2 = b4 ? 4 : 0;
        const bool b2 = nv - t2 >= 2;
        if (b2) {
          const float2 q2 = make_float2(qx, qy);
          __builtin_memcpy(part + o + t2, &q2, 8);
        }
        if (nv - t2 - (b2 ? 2 : 0) >= 1) part[o + t2 + (b2 ? 2 : 0)] = b2 ? qz : qx;
      } else {
        const float vals[8] = {lo[it].x, lo[it].y, lo[it].z, lo[it].w, hi[it].x, hi[it].y, hi[it].z, hi[it].w};
#pragma unroll
        for (int t = 0; t < 8; ++t)
          if (t < r.nvalid) part[o + t + (t >= r.wrap ? next_img : 0)] = vals[t];
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
}

template <int CH, int WP, int WK, int MB, int NB, bool S2, int UPX, int HS, bool PK, bool BG>
__global__ __launch_bounds__((WP * WK + kLoaders) * 64) void conv3x3_kernel(K3Args a) {
  constexpr int NC = WP * WK;                 // compute waves
  constexpr int TP = WP * MB * 32, TK = WK * NB * 32;
  constexpr int UP = CH / 8;                  // 16-byte units per pixel / filter row
  constexpr int KS = CH / 16;                 // MFMA steps per tap and chunk
  static_assert(CH == 16 || CH == 32, "channel chunk");
  static_assert(UPX == 8 || UPX == 4, "column window");
  static_assert(!(PK && BG), "one filter path");
  constexpr bool FL = !PK && !BG;             // the loader waves stage the filters from KCRS
  extern __shared__ __align__(16) vec16 smem[];
  char* lds = reinterpret_cast<char*>(smem);

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // Work units (pixel tile, channel tile, split) are dealt to the eight XCDs
  // in contiguous ranges, channel tile outermost: workgroup b runs on XCD
  // b % 8, so each XCD reads a contiguous range of pixel tiles and (for
  // many channel tiles) only its own slice of the filters, which its L2
  // then holds for all of its workgroups.
  const int units = a.ptiles * a.ktiles * a.e.splits;
  const int per_xcd = (units + 7) >> 3;
  const int unit = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (unit >= units || (blockIdx.x >> 3) >= per_xcd) return;  // uniform over the workgroup
  const int split = unit % a.e.splits;
  const int tile = unit / a.e.splits;
  const int ktile = tile / a.ptiles, ptile = tile - ktile * a.ptiles;
  const int j0 = ptile * TP, k0 = ktile * TK;
  const int ch_begin = split * a.chunks_per_split;
  const int nchunks = min(a.nch, ch_begin + a.chunks_per_split) - ch_begin;
  const int npairs = (nchunks + 1) >> 1;  // barrier steps run in pairs
  auto vrow = [&](int j) {
    const int n = j / a.PE, pq = j - n * a.PE;
    return n * a.Hp + (pq / a.E) * a.sh;
  };
  const int v_lo = vrow(j0);

  if (wave >= NC) {
    // ---------------- loader waves ----------------
    const int lt = tid - NC * 64;
    const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, a.x_bytes);
    const __amdgpu_buffer_rsrc_t wr = make_rsrc(a.w, a.w_bytes);
    const uint32_t plane = static_cast<uint32_t>(a.H * a.W * 2);
    // With a filter package (PK) loader waves 0-1 load the halo and waves 2-3
    // copy the filter tiles by DMA; otherwise all four do both.
    constexpr int HL = PK ? 128 : 256;  // halo lanes
    // Halo items: (channel group g, halo row vr, column window gc).  The
    // per-lane offset is that of channel 8g; the chunk's channels go into
    // the scalar offset.  Rows outside the image read zeros.
    uint32_t hvo[HS];
    int hrow[HS];    // LDS slot of the item's halo row, -1: no item
    int hcol[HS];    // padded column of the window's first pixel
    int hg[HS];
#pragma unroll
    for (int t = 0; t < HS; ++t) {
      const int it = lt + t * HL;
      hvo[t] = a.x_bytes;
      hrow[t] = -1;
      hcol[t] = 0;
      hg[t] = 0;
      if (lt < HL && it < a.halo_items) {
        // Channel groups fastest, then column windows, then rows: the UP
        // lanes of one window write distinct units of the same slots, and
        // windows and rows spread the rest over the banks (the bank groups
        // of 16 consecutive slots are taken by the compute waves' reads, so
        // the writes' pattern can only be chosen by the item order).
        const int g = it % UP, rest = it / UP;
        const int vr = rest / a.NG, gc = rest - vr * a.NG;
        const int ws = min(gc * UPX, a.W - UPX);
        const int v = v_lo + vr;
        const int n = v / a.Hp, h = v - n * a.Hp - a.ph;
        if (n < a.N && h >= 0 && h < a.H)
          hvo[t] = static_cast<uint32_t>(((n * a.C + 8 * g) * a.H + h) * a.W + ws) * 2;
        hg[t] = g;
        hrow[t] = vr * a.RS;
        hcol[t] = ws + a.pw;
      }
    }
    // LDS byte offset (within a stage) of each pixel unit of each item: the
    // same in every chunk.
    uint32_t hoff[HS][UPX];
#pragma unroll
    for (int t = 0; t < HS; ++t)
#pragma unroll
      for (int px = 0; px < UPX; ++px) {
        const int pc = hcol[t] + px;
        const int slot = S2 ? hrow[t] + (pc & 1) * a.PS + (pc >> 1) : hrow[t] + pc;
        hoff[t][px] = static_cast<uint32_t>(slot * (CH * 2) + ((hg[t] ^ k3_swz<UP>(slot)) * 16));
      }
    constexpr int HD = UPX / 2;  // dwords per channel of a window
    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    // Chunks past the last re-read the last one (never written to LDS), so
    // the issue sequence does not depend on the chunk count.
    auto chunk_of = [&](int ch) { return ch < nchunks ? ch : nchunks - 1; };
    if constexpr (PK) {
      constexpr int NST = 3;
      if (lt >= HL) {
        // ---- filter DMA waves: chunk i's tile lands in stage i % 3 ----
        // The package holds each (chunk, channel tile) filter tile as
        // [tap][TK][CH], FU 16-byte units; DMA instruction j of wave dw
        // fills LDS units (dw FI + j) 64 + lane, and a lane fetches the
        // package unit that the bank swizzle puts there.
        constexpr int FU = kK3Taps * TK * CH / 8;
        constexpr int FI = FU / 128;
        static_assert(FU % 128 == 0 && FI <= 31, "DMA split");
        const int dw = wave - NC - 2;
        uint32_t dvo[FI];
#pragma unroll
        for (int j = 0; j < FI; ++j) {
          const int u = (dw * FI + j) * 64 + lane;
          const int row = u / UP, phys = u - (u / UP) * UP;
          dvo[j] = static_cast<uint32_t>(row * UP + (phys ^ k3_swz<UP>(row % TK))) * 16;
        }
        auto dma = [&](int ch, int st) {
          const uint32_t so = static_cast<uint32_t>(((ch_begin + ch) * a.ktiles + ktile) * FU) * 16;
          char __attribute__((address_space(3)))* Fs =
              (char __attribute__((address_space(3)))*)(lds + st * a.stage_bytes + a.halo_bytes);
#pragma unroll
          for (int j = 0; j < FI; ++j) {
            // (The offset goes through a scalar: with the array element as the
            // operand, hipcc's host pass silently drops the kernel's stub.)
            const uint32_t vo = dvo[j];
            __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (lds_void_t*)(Fs + (dw * FI + j) * 1024), 16, vo, so, 0, 0);
          }
        };
        dma(0, 0);
        if (nchunks > 1) dma(1, 1);
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();  // the padding is clear
        int st2 = 2;                   // stage of chunk i + 2
        for (int i = 0; i < npairs * 2; ++i) {
          if (i < nchunks) {
            // chunk i's tile must have landed; chunk i+1's may stay in flight
            if (i + 1 < nchunks) CONVSEL_WAIT_VMCNT(FI); else CONVSEL_WAIT_VMCNT(0);
          }
          asm volatile("" ::: "memory");
          __builtin_amdgcn_s_barrier();  // A(i)
          asm volatile("" ::: "memory");
          if (i + 2 < nchunks) dma(i + 2, st2);  // its stage held chunk i-1, freed at B(i-1)
          st2 = st2 == NST - 1 ? 0 : st2 + 1;
          asm volatile("" ::: "memory");
          __builtin_amdgcn_s_barrier();  // B(i)
          asm volatile("" ::: "memory");
        }
        return;
      }
      // ---- halo waves: register path, two sets, three stages ----
      uint32_t hd[2][HS][8][HD];
      auto issue_h = [&](int ch, auto set_c) {
        constexpr int SET = decltype(set_c)::value;
        const int c0 = (ch_begin + ch) * CH;
#pragma unroll
        for (int t = 0; t < HS; ++t) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const uint32_t so = static_cast<uint32_t>(c0 + e) * plane;
            if constexpr (UPX == 8) {
              const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(xr, hvo[t], so, 0);
              hd[SET][t][e][0] = v[0]; hd[SET][t][e][1] = v[1]; hd[SET][t][e][2] = v[2]; hd[SET][t][e][3] = v[3];
            } else {
              const auto v = __builtin_amdgcn_raw_buffer_load_b64(xr, hvo[t], so, 0);
              hd[SET][t][e][0] = v[0]; hd[SET][t][e][1] = v[1];
            }
          }
        }
      };
      auto write_h = [&](int st, auto set_c) {
        constexpr int SET = decltype(set_c)::value;
        char* Hs = lds + st * a.stage_bytes;
#pragma unroll
        for (int t = 0; t < HS; ++t) {
          if (hrow[t] >= 0) {
#pragma unroll
            for (int px = 0; px < UPX; ++px) {
              // pixel px of the window: channels 8g .. 8g+7, the px-th bf16 of
              // each channel's loaded dword pair, as one 16-byte unit
              u32x4_t o;
#pragma unroll
              for (int m = 0; m < 4; ++m)
                o[m] = __builtin_amdgcn_perm(hd[SET][t][2 * m + 1][px >> 1], hd[SET][t][2 * m][px >> 1],
                                             (px & 1) ? 0x07060302u : 0x05040100u);
              *reinterpret_cast<u32x4_t*>(Hs + hoff[t][px]) = o;
            }
          }
        }
      };
      constexpr int PH = HS * 8;
      issue_h(0, S0{});
      issue_h(chunk_of(1), S1{});
      for (int i = lt; i < a.halo_bytes / 16; i += HL) {
#pragma unroll
        for (int st = 0; st < NST; ++st) reinterpret_cast<u32x4_t*>(lds + st * a.stage_bytes)[i] = u32x4_t{0u, 0u, 0u, 0u};
      }
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_waitcnt(0xc07f);
      __builtin_amdgcn_s_barrier();  // the padding is clear
      asm volatile("" ::: "memory");
      CONVSEL_WAIT_VMCNT(PH);  // chunk 0 (chunk 1's loads may stay in flight)
      write_h(0, S0{});
      issue_h(chunk_of(2), S0{});
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_waitcnt(0xc07f);
      int st1 = 1;  // stage of chunk i + 1
      auto hstep = [&](int i, auto set_c) {  // set_c: (i + 1) & 1
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();  // A(i)
        asm volatile("" ::: "memory");
        CONVSEL_WAIT_VMCNT(PH);
        if (i + 1 < nchunks) write_h(st1, set_c);  // its stage held chunk i-2, freed at B(i-2)
        issue_h(chunk_of(i + 3), set_c);
        st1 = st1 == NST - 1 ? 0 : st1 + 1;
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_waitcnt(0xc07f);
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();  // B(i)
        asm volatile("" ::: "memory");
      };
      for (int i = 0; i < npairs * 2; i += 2) {
        hstep(i, S1{});
        hstep(i + 1, S0{});
      }
      CONVSEL_WAIT_VMCNT(0);
      return;
    }
    // Filter items: (filter row kl, channel group g); rows past K read zeros.
    const int kl = lt / UP, fg = lt - (lt / UP) * UP;
    const bool f_on = kl < TK;
    const uint32_t fvo = (f_on && k0 + kl < a.K)
                             ? static_cast<uint32_t>(((k0 + kl) * a.C + 8 * fg) * kK3Taps) * 2
                             : a.w_bytes;
    // Every chunk issues the same HS * 8 (+ 9 filter) loads per lane (unused
    // halo slots read zeros past the buffer), so the compiler's own count of
    // the loads in flight matches the explicit waits below.  With BG the
    // compute waves read the filters themselves and the loaders only stage
    // the halo.
    constexpr int PER = HS * 8 + (FL ? kK3Taps : 0);
    static_assert(2 * PER <= 63, "vmcnt range");
    // Two register sets, by chunk parity: chunk i+2's loads stay in flight
    // while chunk i+1 is written to LDS.
    uint32_t hd[2][HS][8][HD];
    u32x4_t fd[2][kK3Taps];

    auto issue = [&](int ch, auto set_c) {
      constexpr int SET = decltype(set_c)::value;
      const int c0 = (ch_begin + ch) * CH;
#pragma unroll
      for (int t = 0; t < HS; ++t) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint32_t so = static_cast<uint32_t>(c0 + e) * plane;
          if constexpr (UPX == 8) {
            const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(xr, hvo[t], so, 0);
            hd[SET][t][e][0] = v[0]; hd[SET][t][e][1] = v[1]; hd[SET][t][e][2] = v[2]; hd[SET][t][e][3] = v[3];
          } else {
            const auto v = __builtin_amdgcn_raw_buffer_load_b64(xr, hvo[t], so, 0);
            hd[SET][t][e][0] = v[0]; hd[SET][t][e][1] = v[1];
          }
        }
      }
      if constexpr (FL) {
        const uint32_t fso = static_cast<uint32_t>(c0 * kK3Taps * 2);
#pragma unroll
        for (int q = 0; q < kK3Taps; ++q)
          fd[SET][q] = __builtin_amdgcn_raw_buffer_load_b128(wr, fvo, fso + 16 * q, 0);
      }
    };
    auto write = [&](int st, auto set_c) {
      constexpr int SET = decltype(set_c)::value;
      char* Hs = lds + st * a.stage_bytes;
      char* Fs = Hs + a.halo_bytes;
#pragma unroll
      for (int t = 0; t < HS; ++t) {
        if (hrow[t] >= 0) {
#pragma unroll
          for (int px = 0; px < UPX; ++px) {
            // pixel px of the window: channels 8g .. 8g+7 as one 16-byte unit
            u32x4_t o;
#pragma unroll
            for (int m = 0; m < 4; ++m)
              o[m] = __builtin_amdgcn_perm(hd[SET][t][2 * m + 1][px >> 1], hd[SET][t][2 * m][px >> 1],
                                           (px & 1) ? 0x07060302u : 0x05040100u);
            *reinterpret_cast<u32x4_t*>(Hs + hoff[t][px]) = o;
          }
        }
      }
      if (FL && f_on) {
        // element i = c * 9 + tap of the 72 loaded values (c = 0..7): the
        // (i & 1) half of dword (i >> 1) & 3 of load i >> 3.  Output dword m
        // of a tap unit pairs elements 2m * 9 + tap and (2m + 1) * 9 + tap.
        const int unit_ = fg ^ k3_swz<UP>(kl);
#pragma unroll
        for (int tap = 0; tap < kK3Taps; ++tap) {
          u32x4_t o;
#pragma unroll
          for (int m = 0; m < 4; ++m) {
            const int i0 = 2 * m * kK3Taps + tap, i1 = (2 * m + 1) * kK3Taps + tap;
            const uint32_t sel = (2u * (i0 & 1)) | ((2u * (i0 & 1) + 1u) << 8) | ((4u + 2u * (i1 & 1)) << 16) |
                                 ((5u + 2u * (i1 & 1)) << 24);
            o[m] = __builtin_amdgcn_perm(fd[SET][i1 >> 3][(i1 >> 1) & 3], fd[SET][i0 >> 3][(i0 >> 1) & 3], sel);
          }
          *reinterpret_cast<u32x4_t*>(Fs + (tap * TK + kl) * (CH * 2) + unit_ * 16) = o;
        }
      }
    };
    // The first two chunks' loads go out before the workgroup clears the
    // halo padding, so the clearing and the wave launches overlap them.
    issue(0, S0{});
    issue(chunk_of(1), S1{});
    for (int i = lt; i < a.halo_bytes / 16; i += 256) {
      reinterpret_cast<u32x4_t*>(lds)[i] = u32x4_t{0u, 0u, 0u, 0u};
      reinterpret_cast<u32x4_t*>(lds + a.stage_bytes)[i] = u32x4_t{0u, 0u, 0u, 0u};
    }
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_s_barrier();  // the padding is clear
    asm volatile("" ::: "memory");
    CONVSEL_WAIT_VMCNT(PER);  // chunk 0 (chunk 1's loads may stay in flight)
    write(0, S0{});
    issue(chunk_of(2), S0{});
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this lane's LDS writes are done
    // Chunk i+1 comes from register set (i+1) & 1, and chunk i+3's loads
    // refill that set; chunk i+2's (the PER loads issued after chunk i+1's)
    // stay in flight.  Steps run in pairs (an odd chunk count gets an empty
    // last step, matched by the compute waves) and every step issues its
    // loads, so the loop carries the same loads in flight on every path.
    auto step = [&](int i, auto set_c) {  // set_c: (i + 1) & 1
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_barrier();  // A(i): chunk i visible to the compute waves
      asm volatile("" ::: "memory");
      CONVSEL_WAIT_VMCNT(PER);
      if (i + 1 < nchunks) write((i + 1) & 1, set_c);  // its stage was freed at B(i-1)
      issue(chunk_of(i + 3), set_c);
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_waitcnt(0xc07f);
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_barrier();  // B(i): the compute waves are done with stage i & 1
      asm volatile("" ::: "memory");
    };
    for (int i = 0; i < npairs * 2; i += 2) {
      step(i, S1{});
      step(i + 1, S0{});
    }
    CONVSEL_WAIT_VMCNT(0);  // the re-reads past the last chunk
    return;
  }

  // ---------------- compute waves ----------------
  __builtin_amdgcn_s_barrier();  // the loaders have cleared the halo padding
  const int wp = wave % WP, wk = wave / WP;
  const int half = lane >> 5, l32 = lane & 31;
  const int jl = min(j0 + TP, a.NPQ) - 1;
  // Slot of each pixel fragment row (clamped to the tile's last pixel).
  int apos[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int j = min(j0 + (wp * MB + mb) * 32 + l32, jl);
    const int pq = j - (j / a.PE) * a.PE;
    const int q = pq - (pq / a.E) * a.E;
    apos[mb] = (vrow(j) - v_lo) * a.RS + q;
  }
  // Tap offsets in slots: row r, column s (stride 2: parity plane s & 1, s >> 1 further).
  auto tapoff = [&](int t) {
    const int r = t / 3, s = t - (t / 3) * 3;
    return S2 ? r * a.RS + (s & 1) * a.PS + (s >> 1) : r * a.RS + s;
  };
  // Filter fragment offsets within a tap (bytes): row kr, unit 2u + half.
  int boff[NB][KS];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int kr = (wk * NB + nb) * 32 + l32;
#pragma unroll
    for (int u = 0; u < KS; ++u) boff[nb][u] = kr * (CH * 2) + (((2 * u + half) ^ k3_swz<UP>(kr)) * 16);
  }

  f32x16_t acc[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = zero16();

  // BG: every filter fragment of a chunk lives in registers, read straight
  // from the package ([chunk][channel tile][tap][TK][CH] units) by the wave
  // that multiplies it: the fragment of step S is reloaded with the next
  // chunk's right after its last MFMA, a whole chunk ahead of its use, and
  // the LDS carries only the halo.  (The last chunk reloads itself.)
  constexpr int NSTEP_ALL = kK3Taps * KS;
  constexpr int NBG = BG ? NSTEP_ALL : 1;
  bf16x8_t bq[NBG][NB];
  uint32_t bvo[NB];
  const __amdgpu_buffer_rsrc_t pr = make_rsrc(a.w, a.w_bytes);
  if constexpr (BG) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) bvo[nb] = static_cast<uint32_t>(((wk * NB + nb) * 32 + l32) * UP + half) * 16;
  }
  auto bload = [&](int ch, auto s_c) {
    constexpr int S = decltype(s_c)::value;
    constexpr int t = S / KS, u = S % KS;
    const uint32_t so = static_cast<uint32_t>((((ch_begin + ch) * a.ktiles + ktile) * kK3Taps + t) * TK * UP + 2 * u) * 16;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(pr, bvo[nb], so, 0);
      __builtin_memcpy(&bq[S][nb], &v, 16);
    }
  };
  if constexpr (BG) static_for<NSTEP_ALL>([&](auto s_c) { bload(0, s_c); });

  // A chunk is 9 KS steps (tap t, 16-channel slice u), each MB pixel and NB
  // filter fragment reads and MB x NB MFMAs.  The reads run D steps ahead of
  // the MFMAs (at most 15 LDS reads in flight per wave), and a wave with a
  // single 32 x 32 block alternates two accumulators by step parity, so that
  // neither an LDS round trip nor a dependent MFMA sits between two MFMAs.
  constexpr int NSTEP = kK3Taps * KS;
  constexpr int RD = MB + (BG ? 0 : NB);      // LDS reads per step
  constexpr int D0 = 15 / RD - 1;
  constexpr int D = D0 < 1 ? 1 : (D0 > NSTEP - 1 ? NSTEP - 1 : D0);
  constexpr int NACC = MB * NB == 1 ? 2 : 1;
  f32x16_t acc2[1];  // the second accumulator (NACC == 2)
  acc2[0] = zero16();
  int cst = 0;  // stage of chunk i
  for (int i = 0; i < nchunks; ++i) {
    lds_sync();  // A(i)
    const char* Hs = lds + cst * a.stage_bytes;
    cst = cst == (PK ? 2 : 1) ? 0 : cst + 1;
    const char* Fs = Hs + a.halo_bytes;
    bf16x8_t fa[D + 1][MB], fb[D + 1][NB];
    auto read = [&](auto s_c) {
      constexpr int S = decltype(s_c)::value;
      constexpr int t = S / KS, u = S % KS, slot = S % (D + 1);
      const int to = tapoff(t);
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const int pos = apos[mb] + to;
        fa[slot][mb] =
            *reinterpret_cast<const bf16x8_t*>(Hs + pos * (CH * 2) + (((2 * u + half) ^ k3_swz<UP>(pos)) * 16));
      }
      if constexpr (!BG)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
          fb[slot][nb] = *reinterpret_cast<const bf16x8_t*>(Fs + t * (TK * CH * 2) + boff[nb][u]);
    };
    const int nxt = i + 1 < nchunks ? i + 1 : i;
    static_for<D>([&](auto s_c) { read(s_c); });
    static_for<NSTEP>([&](auto s_c) {
      constexpr int S = decltype(s_c)::value;
      if constexpr (S + D < NSTEP) read(std::integral_constant<int, S + D>{});
      // Keep the program order: the scheduler would otherwise sink each read
      // next to its MFMA.
      __builtin_amdgcn_sched_barrier(0);
      constexpr int slot = S % (D + 1);
      auto bfrag = [&](int nb) -> const bf16x8_t& { return BG ? bq[BG ? S : 0][nb] : fb[slot][nb]; };
      if constexpr (NACC == 2 && (S & 1)) {
        acc2[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[slot][0], bfrag(0), acc2[0], 0, 0, 0);
      } else {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
          for (int nb = 0; nb < NB; ++nb)
            acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[slot][mb], bfrag(nb), acc[mb][nb], 0, 0, 0);
      }
      if constexpr (BG) bload(nxt, s_c);
      __builtin_amdgcn_sched_barrier(0);
    });
    lds_sync();  // B(i)
  }
  if constexpr (NACC == 2) acc[0][0] += acc2[0];
  if (nchunks & 1) {  // the loaders' empty last step of an odd chunk count
    lds_sync();
    lds_sync();
  }

  // ---------------- epilogue ----------------
  // After B of the last chunk no wave reads the stages again: each compute
  // wave stages its output in its own region at the start of LDS.
  char* stage = lds + wave * (MB * 32 * 32 * 4);
  const K3Map m{a.E, a.PE, a.Q, a.NPQ};
  k3_epilogue<MB, NB>(acc, stage, a.e, m, k0 + wk * NB * 32, j0 + wp * MB * 32, split);
}

// ---------------------------------------------------------------------------
// Host side: tile configurations and planning.
// ---------------------------------------------------------------------------
struct K3Config {
  int CH, WP, WK, MB, NB;
  int tp() const { return WP * MB * 32; }
  int tk() const { return WK * NB * 32; }
  int nc() const { return WP * WK; }
};

// The instantiated tile shapes (pixels x channels per workgroup, wave tile):
// 512 x 64 (waves 128 x 64), 128 x 128 (64 x 64), 128 x 64 (64 x 32),
// 64 x 64 (32 x 32).
constexpr K3Config kK3Configs[] = {
    {16, 4, 1, 4, 2},
    {16, 2, 2, 2, 2},
    {32, 2, 2, 2, 1},
    {32, 2, 2, 1, 1},
};
constexpr int kNumK3Configs = sizeof(kK3Configs) / sizeof(kK3Configs[0]);

struct K3Plan {
  int cfg;
  bool pk;   // filters from the tile-ordered package (by DMA, three LDS stages; or, with bg, into registers)
  bool bg;   // the compute waves read their filter fragments from the package into registers
  bool aligned;  // pixel layout with bank-aligned rows (E >= Q), else E = Q
  int nsplit;    // ways the channel reduction is split
  bool s2;
  int upx;
  int64_t images_per_launch;
  size_t part_bytes, lds;
  K3Args a;
};

// Largest halo span (virtual rows) of any TP-pixel tile of N images
// (pixels enumerated with E columns per output row).
int k3_halo_rows(const Shape& s, int64_t N, int Hp, int TP, int E) {
  const int64_t PQ = s.P * E, NPQ = N * PQ;
  const int64_t tiles = (NPQ + TP - 1) / TP;
  auto vrow = [&](int64_t j) {
    const int64_t n = j / PQ, pq = j % PQ;
    return n * Hp + (pq / E) * s.sh;
  };
  // A tile's span depends only on where it starts within an image, which
  // repeats every PQ / gcd(TP, PQ) tiles.
  int64_t a = TP, b = PQ;
  while (b) {
    const int64_t t = a % b;
    a = b;
    b = t;
  }
  const int64_t period = PQ / a;
  int64_t best = 0;
  for (int64_t t = 0; t < tiles && t <= period; ++t) {
    const int64_t j1 = ((t + 1) * TP < NPQ ? (t + 1) * TP : NPQ) - 1;
    best = std::max(best, vrow(j1) - vrow(t * TP) + 3);
  }
  best = std::max(best, vrow(NPQ - 1) - vrow((tiles - 1) * TP) + 3);
  return (int)best;
}

bool k3_shape_ok(const Shape& s) {
  if (s.dtype != DT_BF16 || s.G != 1 || s.R != 3 || s.S != 3) return false;
  if (s.sh != s.sw || (s.sh != 1 && s.sh != 2) || s.dh != 1 || s.dw != 1) return false;
  if (s.C % 16 != 0 || s.W < 4 || s.P * s.Q < 8) return false;
  if (s.ph > 2 || s.pw > 2) return false;
  return true;
}

// Pixel layouts.  The compute waves read the halo in 16-lane groups of 16
// consecutive tile pixels; the reads are free of bank conflicts when those
// pixels' slots are 16 consecutive slots (mod 16).  Along an output row they
// are; across a row end the slot jumps by sh * RS - Q, across an image by
// Hp * RS - P * Q.  The aligned layout pads each output row to E columns (a
// multiple of 8; the padding pixels are computed and not stored) and picks
// RS and Hp so that both jumps are 0 mod 16.  At stride 1 consecutive halo
// rows share their padding columns (the right padding of row v is the left
// padding of row v + 1: both are zeros), which keeps RS small.  The plain
// layout (E = Q) is used where the aligned one does not fit.
void k3_layout(const Shape& s, bool aligned, int& E, int& RS, int& PS, int& Hp) {
  // Padded columns read: q * sh + tap column < (Q - 1) * sh + 3; written: [pw, W + pw).
  const int cols = (int)std::max<int64_t>((s.Q - 1) * s.sh + 3, s.W + s.pw);
  const int hmin = (int)((s.P - 1) * s.sh + 3);
  PS = s.sh == 2 ? (cols + 1) / 2 : 0;
  if (!aligned) {
    E = (int)s.Q;
    RS = s.sh == 2 ? 2 * PS : cols;
    Hp = hmin;
    return;
  }
  E = (int)((s.Q + 7) / 8 * 8);
  RS = s.sh == 2 ? 2 * PS : (int)std::max<int64_t>(s.W + s.pw, (s.Q - 1) + 3 - s.pw);
  while (((s.sh * RS - E) % 16 + 16) % 16 != 0) ++RS;
  Hp = hmin;
  for (int h = hmin; h < hmin + 16; ++h)
    if (((h * RS - (int)s.P * E) % 16 + 16) % 16 == 0) {
      Hp = h;
      break;
    }
}

bool make_k3_plan_cfg(const Shape& s, int cfg, K3Plan& pl, int64_t N1, bool pk, bool aligned, int nsplit,
                      bool bg = false) {
  const K3Config c = kK3Configs[cfg];
  if (s.C % c.CH != 0) return false;
  // The register copy of a chunk's filter fragments fits next to the
  // accumulators only for the tiles with at most 72 fragment registers and
  // 32 or 64 accumulators.
  if (bg && (!pk || kK3Taps * (c.CH / 16) * c.NB * 4 > 72 || c.MB * c.NB > 4)) return false;
  pl.cfg = cfg;
  pl.pk = pk;
  pl.bg = bg;
  pl.aligned = aligned;
  pl.s2 = s.sh == 2;
  pl.upx = s.W >= 8 ? 8 : 4;
  pl.images_per_launch = N1;
  K3Args& a = pl.a;
  a.N = (int)N1; a.C = (int)s.C; a.H = (int)s.H; a.W = (int)s.W; a.K = (int)s.K;
  a.P = (int)s.P; a.Q = (int)s.Q;
  a.sh = s.sh; a.ph = s.ph; a.pw = s.pw;
  k3_layout(s, aligned, a.E, a.RS, a.PS, a.Hp);
  a.PE = (int)(s.P * a.E);
  if (N1 * a.PE >= ((int64_t)1 << 31)) return false;
  a.NPQ = (int)(N1 * a.PE);
  a.ptiles = (a.NPQ + c.tp() - 1) / c.tp();
  a.ktiles = (int)((s.K + c.tk() - 1) / c.tk());
  a.nch = (int)(s.C / c.CH);
  a.VR = k3_halo_rows(s, N1, a.Hp, c.tp(), a.E);
  a.NG = (int)((s.W + pl.upx - 1) / pl.upx);
  a.halo_items = a.VR * a.NG * (c.CH / 8);
  const int halo_lanes = pk && !bg ? 128 : 256;
  if (a.halo_items > kHSMax * halo_lanes) return false;
  // 16 spare zero slots after the last row: taps of the last row's final
  // pixels (and of padding pixels) read past it.
  a.halo_bytes = (int)((((size_t)a.VR * a.RS + 16) * c.CH * 2 + 255) / 256 * 256);
  const size_t filt = bg ? 0 : (size_t)kK3Taps * c.tk() * c.CH * 2;
  a.stage_bytes = (int)(a.halo_bytes + filt);
  pl.lds = (size_t)(pk && !bg ? 3 : 2) * a.stage_bytes;
  // The epilogue stages each compute wave's fp32 or bf16 rows in LDS.
  const size_t staging = (size_t)c.nc() * c.MB * 32 * 32 * 4;
  if (pl.lds < staging) pl.lds = staging;
  if (pl.lds > kLdsLimit) return false;
  // The channel chunks are split nsplit ways (fewer when the chunks do not
  // go round).
  if (nsplit < 1 || nsplit > a.nch) return false;
  a.chunks_per_split = (a.nch + nsplit - 1) / nsplit;
  a.e.splits = (a.nch + a.chunks_per_split - 1) / a.chunks_per_split;
  if (a.e.splits != nsplit) return false;
  pl.nsplit = nsplit;
  a.e.K = (int)s.K; a.e.Kg = (int)s.K; a.e.relu = s.relu ? 1 : 0; a.e.PQ = (int)(s.P * s.Q);
  a.e.span = a.e.PQ;
  a.e.NPQ = a.NPQ;
  a.e.slab = (int)((N1 * s.K * s.P * s.Q + 3) & ~(int64_t)3);
  pl.part_bytes = a.e.splits > 1 ? (size_t)a.e.splits * a.e.slab * sizeof(float) : 0;
  return true;
}

// Estimated time of a plan, in microseconds:
//
//   a + rounds * chunks * max(b[tile] * MFMAs per chunk, c * halo items per
//   loader lane * CH / 16 + d * filter bytes regrouped per chunk / 1024)
//     + g * rounds + (split: e + f * splits * N*K*P*Q * 8 bytes / 1e6)
//
// rounds = workgroups over the 256 CUs, chunks per workgroup, MFMAs of one
// compute wave.  A chunk is bound either by the compute waves (their MFMAs
// and operand reads, per tile shape) or by the loader waves (halo rows
// transposed per lane, filters regrouped); a and g are the launch and the
// per-round pipeline fill and drain; split partial sums cost their fp32
// round trip and the reduction kernel.  The constants are least-squares fits
// (relative error) to measured times of the bf16 3x3 layers of ResNet-50 at
// batch 32 over every tile shape and split of 1, 2 and 4; one set for the
// per-call kernel (filters regrouped by the loaders), one for the package
// kernel with filters by DMA, one for the package kernel with filters in
// the compute waves' registers (the loaders then stage only the halo, with
// all 256 lanes).  Median error about 6% (per call), 12% (DMA) and 5%
// (registers).  The register path wins where the halo is the loaders'
// bottleneck (the stride-2 layers: their halo holds four input pixels per
// output pixel).
struct K3CostParams {
  double a, b[kNumK3Configs], c, d, e, f, g;
};
constexpr K3CostParams kK3CostCall = {7.18, {0.0180, 0.0252, 0.0307, 0.0534}, 0.500, 0.0, 2.99, 0.168, 4.85};
constexpr K3CostParams kK3CostPack = {4.90, {0.0180, 0.0278, 0.0175, 0.0094}, 0.315, 0.0, 0.90, 0.204, 4.39};
constexpr K3CostParams kK3CostBg = {4.41, {1.0, 0.0226, 0.0333, 0.0482}, 0.543, 0.0, 3.29, 0.128, 4.59};

double k3_cost(const K3Plan& pl, const Shape& s) {
  const K3CostParams& m = pl.bg ? kK3CostBg : pl.pk ? kK3CostPack : kK3CostCall;
  const K3Config c = kK3Configs[pl.cfg];
  const K3Args& a = pl.a;
  const int64_t wgs = (int64_t)a.ptiles * a.ktiles * a.e.splits;
  const double rounds = (double)((wgs + kCUs - 1) / kCUs);
  const double mfma = (double)kK3Taps * (c.CH / 16) * c.MB * c.NB;
  const int HL = pl.pk && !pl.bg ? 128 : 256;
  const double hs = (double)((a.halo_items + HL - 1) / HL);
  const double filt = pl.pk ? 0.0 : (double)c.tk() * c.CH / 1024.0;
  const double chunk = std::max(m.b[pl.cfg] * mfma, m.c * hs * c.CH / 16.0 + m.d * filt);
  double t = m.a + rounds * a.chunks_per_split * chunk + m.g * rounds;
  if (a.e.splits > 1) t += m.e + m.f * a.e.splits * (double)(a.N * s.P * s.Q) * s.K * 8.0 / 1e6;
  return t;
}

bool make_k3_plan(const Shape& s, K3Plan& pl, int64_t N1 = -1, bool prepacked = false) {
  if (!k3_shape_ok(s)) return false;
  const int64_t img_bytes = s.C * s.H * s.W * 2;
  if (img_bytes > kMaxLaunchBytes) return false;
  if (N1 < 0) {
    N1 = kMaxLaunchBytes / img_bytes;
    if (N1 > s.N) N1 = s.N;
    if (N1 < 1) N1 = 1;
  }
  if ((int64_t)s.K * s.C * 9 * 2 >= ((int64_t)1 << 31)) return false;
  // Every tile shape and split of 1, 2, 4 or 8, in the aligned layout where
  // it fits (else the plain one), scored by the per-call estimate plus the
  // package kernel's estimate (or the per-call one again where the package
  // kernel does not fit): both calls of a layer run the same tiles and split,
  // so their results are the same bits, and the choice serves both.  The
  // remainder launch (N not a multiple of the images per launch) must fit the
  // same choice.
  const int64_t r = s.N % N1;
  auto build = [&](int cfg, bool pk, bool al, int S, K3Plan& out, bool bg = false) {
    K3Plan rest;
    return make_k3_plan_cfg(s, cfg, out, N1, pk, al, S, bg) &&
           (r == 0 || make_k3_plan_cfg(s, cfg, rest, r, pk, al, S, bg));
  };
  bool found = false;
  double best = 0;
  K3Plan best_call, best_pack;
  bool best_has_pack = false;
  for (int cfg = 0; cfg < kNumK3Configs; ++cfg) {
    for (int S = 1; S <= 8; S *= 2) {
      K3Plan call;
      bool al = true;
      if (!build(cfg, false, true, S, call)) {
        al = false;
        if (!build(cfg, false, false, S, call)) continue;
      }
      // The package kernels: filters by DMA (not for the 512-pixel tile,
      // where the register path measured as fast) or read into registers by
      // the compute waves, whichever is estimated faster.
      K3Plan pack, pack_bg;
      bool has_pack = cfg != 0 && build(cfg, true, al, S, pack);
      if (build(cfg, true, al, S, pack_bg, true) && (!has_pack || k3_cost(pack_bg, s) < k3_cost(pack, s))) {
        pack = pack_bg;
        has_pack = true;
      }
      const double t = k3_cost(call, s) + (has_pack ? k3_cost(pack, s) : k3_cost(call, s));
      if (!found || t < best) {
        best = t;
        best_call = call;
        best_pack = pack;
        best_has_pack = has_pack;
        found = true;
      }
    }
  }
  if (!found) return false;
  // Prepacked filters (built once, outside the call) go in by DMA from the
  // package in every launch of the layer (the package's layout follows the
  // tile shape).  A per-call package would cost its own launch, which
  // measured more than the DMA saves, so conv2d() regroups the filters in
  // the kernel.
  pl = prepacked && best_has_pack ? best_pack : best_call;
  return true;
}

// Plan of a launch of `cnt` images with the tile shape and filter path of
// the layer's plan.
bool k3_plan_for_launch(const Shape& s, const K3Plan& pl, int64_t cnt, K3Plan& cur) {
  if (cnt == pl.images_per_launch) {
    cur = pl;
    return true;
  }
  return make_k3_plan_cfg(s, pl.cfg, cur, cnt, pl.pk, pl.aligned, pl.nsplit, pl.bg);
}

// Filter package: for chunk cg (CH channels) and channel tile kt, the LDS
// image of the tile's filters, [tap][TK][CH], zero past K.  One thread per
// (chunk, filter row, 8-channel group) reads the group's 8 x 9 values (72
// consecutive bf16 of the KCRS filter) and writes its nine tap units.
constexpr int kK3PackThreads = 128;
__global__ __launch_bounds__(kK3PackThreads) void k3_pack_kernel(const uint16_t* __restrict__ w,
                                                                 u32x4_t* __restrict__ pk, int K, int C, int Kpad,
                                                                 int TK, int CH, int items, int vec) {
  const int item = blockIdx.x * kK3PackThreads + threadIdx.x;
  if (item >= items) return;
  const int UP = CH / 8;
  const int g = item % UP, rest = item / UP;
  const int k = rest % Kpad, cg = rest / Kpad;
  uint32_t v[72];  // element i = c * 9 + tap, c = 0..7
  if (k < K && vec) {
    const u32x4_t* src = reinterpret_cast<const u32x4_t*>(w + (static_cast<int64_t>(k) * C + cg * CH + 8 * g) * 9);
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
    for (int i = 0; i < 72; ++i)
      v[i] = k < K ? w[(static_cast<int64_t>(k) * C + cg * CH + 8 * g + i / 9) * 9 + i % 9] : 0u;
  }
  const int ktiles = Kpad / TK;
  const int64_t FU = (int64_t)9 * TK * UP;
  u32x4_t* dst = pk + (static_cast<int64_t>(cg) * ktiles + k / TK) * FU + (k % TK) * UP + g;
#pragma unroll
  for (int tap = 0; tap < 9; ++tap) {
    u32x4_t o;
#pragma unroll
    for (int m = 0; m < 4; ++m) o[m] = v[(2 * m) * 9 + tap] | (v[(2 * m + 1) * 9 + tap] << 16);
    dst[static_cast<int64_t>(tap) * TK * UP] = o;
  }
}

template <int CH, int WP, int WK, int MB, int NB, bool S2, int UPX, int HS, bool PK, bool BG>
hipError_t k3_launch(const K3Plan& pl, const K3Args& a, hipStream_t stream) {
  const auto kern = conv3x3_kernel<CH, WP, WK, MB, NB, S2, UPX, HS, PK, BG>;
  static std::atomic<int> lds_limit{64 * 1024};
  if ((int)pl.lds > lds_limit.load()) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsLimit);
    if (e != hipSuccess) return e;
    lds_limit.store((int)kLdsLimit);
  }
  const int units = a.ptiles * a.ktiles * a.e.splits;
  const dim3 grid((unsigned)(8 * ((units + 7) / 8)));
  hipLaunchKernelGGL(kern, grid, dim3((WP * WK + kLoaders) * 64), pl.lds, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.e.splits == 1) return e;
  const int total = a.N * a.K * a.P * a.Q;
  hipLaunchKernelGGL(splitk_reduce_kernel<bf16_t>, dim3(reduce_blocks(total)), dim3(256), 0, stream,
                     a.e.partial, reinterpret_cast<const bf16_t*>(a.e.b), reinterpret_cast<bf16_t*>(a.e.y), total,
                     a.e.slab, a.P * a.Q, a.K, a.e.splits, a.e.relu, reinterpret_cast<const bf16_t*>(a.e.res));
  return hipGetLastError();
}

template <int CH, int WP, int WK, int MB, int NB, bool S2, int UPX>
hipError_t k3_dispatch_hs(const K3Plan& pl, const K3Args& a, hipStream_t st) {
  if (pl.bg) {
    // only the tiles whose fragments fit in registers (make_k3_plan_cfg)
    if constexpr (kK3Taps * (CH / 16) * NB * 4 <= 72 && MB * NB <= 4)
      return a.halo_items > 256 ? k3_launch<CH, WP, WK, MB, NB, S2, UPX, 2, false, true>(pl, a, st)
                                : k3_launch<CH, WP, WK, MB, NB, S2, UPX, 1, false, true>(pl, a, st);
    return hipErrorInvalidValue;
  }
  if (pl.pk)
    return a.halo_items > 128 ? k3_launch<CH, WP, WK, MB, NB, S2, UPX, 2, true, false>(pl, a, st)
                              : k3_launch<CH, WP, WK, MB, NB, S2, UPX, 1, true, false>(pl, a, st);
  return a.halo_items > 256 ? k3_launch<CH, WP, WK, MB, NB, S2, UPX, 2, false, false>(pl, a, st)
                            : k3_launch<CH, WP, WK, MB, NB, S2, UPX, 1, false, false>(pl, a, st);
}

template <int CH, int WP, int WK, int MB, int NB>
hipError_t k3_dispatch_cfg(const K3Plan& pl, const K3Args& a, hipStream_t st) {
  if (pl.s2)
    return pl.upx == 8 ? k3_dispatch_hs<CH, WP, WK, MB, NB, true, 8>(pl, a, st)
                       : k3_dispatch_hs<CH, WP, WK, MB, NB, true, 4>(pl, a, st);
  return pl.upx == 8 ? k3_dispatch_hs<CH, WP, WK, MB, NB, false, 8>(pl, a, st)
                     : k3_dispatch_hs<CH, WP, WK, MB, NB, false, 4>(pl, a, st);
}

hipError_t k3_dispatch(const K3Plan& pl, const K3Args& a, hipStream_t st) {
  switch (pl.cfg) {
    case 0: return k3_dispatch_cfg<16, 4, 1, 4, 2>(pl, a, st);
    case 1: return k3_dispatch_cfg<16, 2, 2, 2, 2>(pl, a, st);
    case 2: return k3_dispatch_cfg<32, 2, 2, 2, 1>(pl, a, st);
    case 3: return k3_dispatch_cfg<32, 2, 2, 1, 1>(pl, a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

bool k3_applies(const Shape& s) {
  K3Plan pl;
  return make_k3_plan(s, pl);
}

size_t k3_split_bytes(const Shape& s) {
  K3Plan pl;
  if (!make_k3_plan(s, pl)) return 0;
  size_t m = pl.part_bytes;
  const int64_t rest = s.N % pl.images_per_launch;
  if (rest) {
    K3Plan last;
    if (k3_plan_for_launch(s, pl, rest, last) && last.part_bytes > m) m = last.part_bytes;
  }
  return m;
}

bool k3_uses_package(const Shape& s) {
  K3Plan pl;
  return make_k3_plan(s, pl, -1, true) && pl.pk;
}

size_t k3_package_bytes(const Shape& s) {
  K3Plan pl;
  if (!make_k3_plan(s, pl, -1, true) || !pl.pk) return 0;
  return (size_t)pl.a.ktiles * kK3Configs[pl.cfg].tk() * s.C * 9 * 2;
}

hipError_t k3_pack(const Shape& s, const void* w, void* pk, hipStream_t stream) {
  K3Plan pl;
  if (!make_k3_plan(s, pl, -1, true) || !pl.pk) return hipErrorInvalidValue;
  const K3Config c = kK3Configs[pl.cfg];
  const int Kpad = pl.a.ktiles * c.tk();
  const int items = (int)(s.C / c.CH) * Kpad * (c.CH / 8);
  const int vec = reinterpret_cast<uintptr_t>(w) % 16 == 0;
  hipLaunchKernelGGL(k3_pack_kernel, dim3((unsigned)((items + kK3PackThreads - 1) / kK3PackThreads)),
                     dim3(kK3PackThreads), 0, stream, reinterpret_cast<const uint16_t*>(w),
                     reinterpret_cast<u32x4_t*>(pk), (int)s.K, (int)s.C, Kpad, c.tk(), c.CH, items, vec);
  return hipGetLastError();
}

hipError_t k3_main(const Shape& s, const void* x, const void* w, const void* b, void* y, void* part_ws,
                   hipStream_t stream, const void* res, bool prepacked) {
  K3Plan pl;
  if (!make_k3_plan(s, pl, -1, prepacked)) return hipErrorInvalidValue;
  const int64_t img_elems = s.C * s.H * s.W, out_elems = s.K * s.P * s.Q;
  for (int64_t n0 = 0; n0 < s.N; n0 += pl.images_per_launch) {
    const int64_t cnt = s.N - n0 < pl.images_per_launch ? s.N - n0 : pl.images_per_launch;
    K3Plan cur;
    if (!k3_plan_for_launch(s, pl, cnt, cur)) return hipErrorInvalidValue;
    if (cur.a.e.splits > 1 && !part_ws) return hipErrorInvalidValue;
    K3Args a = cur.a;
    a.x = reinterpret_cast<const uint16_t*>(x) + n0 * img_elems;
    a.x_bytes = (uint32_t)(cnt * img_elems * 2);
    a.w = w;  // the package when pl.pk, else the KCRS filters
    a.w_bytes = pl.pk ? (uint32_t)((size_t)pl.a.ktiles * kK3Configs[pl.cfg].tk() * s.C * 9 * 2)
                      : (uint32_t)(s.K * s.C * 9 * 2);
    a.e.y = reinterpret_cast<uint16_t*>(y) + n0 * out_elems;
    a.e.res = res ? reinterpret_cast<const uint16_t*>(res) + n0 * out_elems : nullptr;
    a.e.b = b;
    a.e.partial = reinterpret_cast<float*>(part_ws);
    a.e.vec = 1;
    const hipError_t e = k3_dispatch(cur, a, stream);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

std::string k3_describe(const Shape& s, bool prepacked) {
  K3Plan pl;
  if (!make_k3_plan(s, pl, -1, prepacked)) return "implicit_gemm (3x3 halo/filter tiles): not applicable";
  const K3Config c = kK3Configs[pl.cfg];
  char buf[512];
  snprintf(buf, sizeof(buf),
           "implicit_gemm kernels=%sconv3x3_kernel<%d,%d,%d,%d,%d,%d,%d,%d,%d,%d>%s tile=%dx%d grid=%dx%d chunk=%d "
           "halo_rows=%d halo_items=%d row_slots=%d cols=%d lds=%zu images_per_launch=%lld (loader waves: halo "
           "rows transposed to pixel-major LDS, %s; compute waves: MFMA %dx%d per wave)",
           pl.pk ? "k3_pack_kernel;" : "", c.CH, c.WP, c.WK, c.MB, c.NB, pl.s2 ? 1 : 0, pl.upx,
           pl.a.halo_items > (pl.pk && !pl.bg ? 128 : 256) ? 2 : 1, pl.pk && !pl.bg ? 1 : 0, pl.bg ? 1 : 0,
           pl.a.e.splits > 1 ? ";splitk_reduce_kernel" : "",
           c.tp(), c.tk(), pl.a.ptiles * pl.a.ktiles, pl.a.e.splits, c.CH, pl.a.VR, pl.a.halo_items, pl.a.RS,
           pl.a.E, pl.lds,
           (long long)pl.images_per_launch,
           pl.bg   ? "filter fragments read from the package into the compute waves' registers, halo only in "
                     "LDS, two LDS stages"
           : pl.pk ? "filter tiles copied by DMA from the package, three LDS stages"
                   : "KCRS filters regrouped to tap-major LDS, two LDS stages",
           32 * c.MB, 32 * c.NB);
  return buf;
}

}  // namespace convsel
