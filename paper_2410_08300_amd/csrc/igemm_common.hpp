// Pieces shared by the implicit GEMM kernels: tile constants, buffer-load
// helpers, the tile epilogue, the split-K reduction and host-side planning
// helpers.
#pragma once

#include <stdint.h>

#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace convsel {
namespace igemm {

constexpr int kThreads = 256;
constexpr int BN = 128;
constexpr uint32_t kRsrcWord3 = 0x00020000u;  // raw buffer, 32-bit data format (gfx9 family)

typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

// Output side of a tile, shared by the implicit GEMM kernels.
struct EpiArgs {
  const void* b;
  void* y;             // first image of this launch
  float* partial;      // splits > 1: fp32 partial sums, [split][N][K][P][Q]
  int K, Kg, NPQ, PQ, relu;
  int span;            // pixels per image in the tile index space: P*Q, or a padded plane (a multiple of 8)
  int splits;          // workgroups sharing one output tile along the channels
  int slab;            // floats per split of `partial` (N*K*P*Q rounded up to 4)
  int vec;             // store piece in elements (8, 4, 2 or 1; see store_tile)
  uint32_t y_bytes = 0;  // bytes of y in this launch when below 2^31 (buffer stores), else 0
  // Residual added after the bias and before the ReLU (same layout and type
  // as y; NULL: none).  With bf16 the convolution's value is rounded to bf16
  // first, so y = round(relu(round(conv + b) + res)) -- the rounding steps
  // of a convolution followed by a separate add.
  const void* res = nullptr;
};

// Adds the residual to the 8 values of a run (offsets as for its stores).
template <typename T>
__device__ __forceinline__ void add_residual_run(float (&v)[8], const EpiArgs& e, int64_t o, bool full, int nvalid,
                                                 int wrap, int PQ, int64_t next_img) {
  const T* rp = reinterpret_cast<const T*>(e.res);
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int t = 0; t < 8; ++t) v[t] = bf16_to_f32(f32_to_bf16(v[t]));
  }
  if (full) {
    if constexpr (sizeof(T) == 2) {
      uint4 r;
      __builtin_memcpy(&r, rp + o, 16);
      const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
      for (int t = 0; t < 8; ++t) v[t] += __uint_as_float((w[t >> 1] >> (16 * (t & 1))) << 16);
    } else {
      float4 a, b;
      __builtin_memcpy(&a, rp + o, 16);
      __builtin_memcpy(&b, rp + o + 4, 16);
      v[0] += a.x; v[1] += a.y; v[2] += a.z; v[3] += a.w;
      v[4] += b.x; v[5] += b.y; v[6] += b.z; v[7] += b.w;
    }
    return;
  }
  int64_t add = 0;
  int next = wrap;
#pragma unroll
  for (int t = 0; t < 8; ++t) {
    if (t == next) {
      add += next_img;
      next += PQ;
    }
    if (t < nvalid) v[t] += elem<T>::load(rp + o + t + add);
  }
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

// Calls f(std::integral_constant<int, i>{}) for i = 0 .. N-1 (compile-time
// indices, so register arrays indexed by i stay in registers).
template <int N, typename F, int I = 0>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, F, I + 1>(static_cast<F&&>(f));
  }
}

// Element offsets of a run of 8 tile pixels that crosses into the next
// image after `wrap` pixels, and then again every PQ pixels: each crossing
// moves the destination (K-1)*PQ elements further than the pixel count
// alone.  With PQ >= 8 a run crosses at most once and the stores use that
// directly; planes smaller than a run use this cursor, per element t = 0..7
// in order:  RunCursor c(wrap, PQ, next_img);  ...  dst[o + c.at(t)] = v[t];
struct RunCursor {
  int64_t add;
  int next;
  const int PQ;
  const int64_t step;
  __device__ __forceinline__ RunCursor(int wrap, int pq, int64_t next_img) : add(0), next(wrap), PQ(pq), step(next_img) {}
  __device__ __forceinline__ int64_t at(int t) {
    if (t == next) {
      add += step;
      next += PQ;
    }
    return t + add;
  }
};

// Bias, ReLU and the NCHW store of one wave's MI x NJ blocks of 32 x 32
// accumulators (NJ even): rows row0 + 32 mi + .. of group g, pixels col0 +
// 32 nj + .., or their raw fp32 partial sums when the channels are split.
// The accumulators go through LDS (`stage`: this wave's 8 KiB), 32 rows x 64
// pixels at a time, so that a lane then holds a run of 8 consecutive pixels
// of one output channel: lane l takes pixels (l % 8) * 8 .. +7 of the 64 and
// rows l / 8 + 8 * it, it = 0..3.  A run inside one image leaves as one
// 16-byte store (2-byte alignment is enough on gfx950; the compiler emits
// these for any 16-byte copy); a run that crosses an image boundary or ends
// at the last pixel is stored element by element.  Bias values are loaded
// before any store: loads and stores share one counter, so a load issued
// after stores would wait for all of them.
template <typename T, int MI, int NJ>
__device__ __forceinline__ void store_block(const f32x16_t (&acc)[MI][NJ], float* stage, const EpiArgs& e, int row0,
                                            int col0, int g, int split) {
  static_assert(NJ % 2 == 0, "blocks of 64 pixels");
  constexpr int EW = 64;  // pixels per staged row
  const int lane = threadIdx.x & 63;
  const int l32 = lane & 31, h = lane >> 5;
  const int PQ = e.PQ, span = e.span;
  const bool split_out = e.splits > 1;
  const T* bias = reinterpret_cast<const T*>(e.b);
  const bool has_bias = bias != nullptr;

  // Staging layout: float4 f of row r sits at f ^ ((r & 1) | 8 ((r >> 2) & 1)),
  // so the writes of two half-waves (rows r and r+4) and the reads of four
  // quarter-waves (rows 2q, 2q+1) touch distinct banks.  For the row of
  // accumulator v of this lane (8 (v/4) + 4 h + v % 4) the XOR term is
  // (v & 1) | 8 h, so the write address is a per-lane base (one per parity
  // of v and per 32-pixel half) plus a constant.
  int wbase[2][2];
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int par = 0; par < 2; ++par) {
      const int px = q * 32 + l32;
      wbase[q][par] = 4 * h * EW + ((((px >> 2) ^ par ^ (h << 3))) << 2) + (px & 3);
    }
  const int rrow = lane >> 3, cb = (lane & 7) * 8;
  const int rsw = (rrow & 1) | (((rrow >> 2) & 1) << 3);
  const int rbase_lo = rrow * EW + (((cb >> 2) ^ rsw) << 2);
  const int rbase_hi = rrow * EW + ((((cb + 4) >> 2) ^ rsw) << 2);

  float bv[MI][4];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int i = row0 + mi * 32 + rrow + 8 * it;
      bv[mi][it] = (!split_out && bias && i < e.Kg) ? elem<T>::load(bias + g * e.Kg + i) : 0.f;
    }

#pragma unroll
  for (int hb = 0; hb < NJ / 2; ++hb) {
    // Pixel j of the tile index space is pixel pq of image n; with a padded
    // plane (span > P*Q) the pixels past P*Q are padding.
    const int j = col0 + hb * EW + cb;
    const int n = j / span, pq = j - n * span;
    // Pixels of this run's image from j on (<= 0: none; j >= NPQ lies past the last image).
    const int last = j >= e.NPQ ? 0 : span == PQ ? e.NPQ - j : PQ - pq;
    const int wrap = span == PQ ? PQ - pq : 8;           // a run crosses into the next image after `wrap` pixels
    const bool full = last >= 8 && wrap >= 8;
    const int nvalid = last < 8 ? last : 8;
    const int64_t next_img = static_cast<int64_t>(e.K - 1) * PQ;
    const int64_t obase = (static_cast<int64_t>(n) * e.K + g * e.Kg + row0 + rrow) * PQ + pq;
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) {
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          stage[wbase[q][v & 1] + (8 * (v >> 2) + (v & 3)) * EW] = acc[mi][2 * hb + q][v];
      __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes are done
      __builtin_amdgcn_wave_barrier();
      float4 lo[4], hi[4];
#pragma unroll
      for (int it = 0; it < 4; ++it) {
        lo[it] = *reinterpret_cast<const float4*>(stage + rbase_lo + it * 8 * EW);
        hi[it] = *reinterpret_cast<const float4*>(stage + rbase_hi + it * 8 * EW);
      }
#pragma unroll
      for (int it = 0; it < 4; ++it) {
        const int i = row0 + mi * 32 + rrow + 8 * it;
        if (i >= e.Kg || nvalid <= 0) continue;
        const int64_t o = obase + static_cast<int64_t>(mi * 32 + 8 * it) * PQ;
        float vals[8] = {lo[it].x, lo[it].y, lo[it].z, lo[it].w, hi[it].x, hi[it].y, hi[it].z, hi[it].w};
        if (split_out) {
          float* part = e.partial + static_cast<int64_t>(split) * e.slab;
          if (full) {
            __builtin_memcpy(part + o, &lo[it], 16);
            __builtin_memcpy(part + o + 4, &hi[it], 16);
          } else {
            if (PQ >= 8) {
#pragma unroll
              for (int t = 0; t < 8; ++t)
                if (t < nvalid) part[o + t + (t >= wrap ? next_img : 0)] = vals[t];
            } else {
              RunCursor rc(wrap, PQ, next_img);
#pragma unroll
              for (int t = 0; t < 8; ++t) {
                const int64_t ot = rc.at(t);
                if (t < nvalid) part[o + ot] = vals[t];
              }
            }
          }
          continue;
        }
        if (has_bias)  // uniform
#pragma unroll
          for (int t = 0; t < 8; ++t) vals[t] += bv[mi][it];
        if (e.res)  // uniform
          add_residual_run<T>(vals, e, o, full, nvalid, wrap, PQ, next_img);
        if (e.relu)  // uniform
#pragma unroll
          for (int t = 0; t < 8; ++t) vals[t] = fmaxf(vals[t], 0.f);
        T* y = reinterpret_cast<T*>(e.y);
        if constexpr (sizeof(T) == 2) {
          if (full) {
            uint4 w;
            w.x = f32x2_to_bf16x2(vals[0], vals[1]);
            w.y = f32x2_to_bf16x2(vals[2], vals[3]);
            w.z = f32x2_to_bf16x2(vals[4], vals[5]);
            w.w = f32x2_to_bf16x2(vals[6], vals[7]);
            __builtin_memcpy(y + o, &w, 16);
          } else {
            if (PQ >= 8) {
#pragma unroll
              for (int t = 0; t < 8; ++t)
                if (t < nvalid) elem<T>::store(y + o + t + (t >= wrap ? next_img : 0), vals[t]);
            } else {
              RunCursor rc(wrap, PQ, next_img);
#pragma unroll
              for (int t = 0; t < 8; ++t) {
                const int64_t ot = rc.at(t);
                if (t < nvalid) elem<T>::store(y + o + ot, vals[t]);
              }
            }
          }
        } else {
          if (full) {
            const float4 a = make_float4(vals[0], vals[1], vals[2], vals[3]);
            const float4 b = make_float4(vals[4], vals[5], vals[6], vals[7]);
            __builtin_memcpy(y + o, &a, 16);
            __builtin_memcpy(y + o + 4, &b, 16);
          } else {
            if (PQ >= 8) {
#pragma unroll
              for (int t = 0; t < 8; ++t)
                if (t < nvalid) elem<T>::store(y + o + t + (t >= wrap ? next_img : 0), vals[t]);
            } else {
              RunCursor rc(wrap, PQ, next_img);
#pragma unroll
              for (int t = 0; t < 8; ++t) {
                const int64_t ot = rc.at(t);
                if (t < nvalid) elem<T>::store(y + o + ot, vals[t]);
              }
            }
          }
        }
      }
      __builtin_amdgcn_wave_barrier();  // the next block reuses this wave's stage
    }
  }
}

// A run of 8 pixels starting at tile pixel `px` (tile origin col0, channel
// block row0 of group g): where its first channel row goes and whether it is
// whole.
struct Run128t {
  int64_t o;
  int nvalid, wrap;
  bool full;
};
__device__ __forceinline__ Run128t run128t(const EpiArgs& e, int row0, int col0, int g, int px) {
  Run128t r;
  const int PQ = e.PQ, span = e.span;
  const int j = col0 + px;
  const int n = j / span, pq = j - n * span;
  const int last = j >= e.NPQ ? 0 : span == PQ ? e.NPQ - j : PQ - pq;
  r.wrap = span == PQ ? PQ - pq : 8;
  r.full = last >= 8 && r.wrap >= 8;
  r.nvalid = last < 8 ? last : 8;
  r.o = (static_cast<int64_t>(n) * e.K + g * e.Kg + row0) * PQ + pq;
  return r;
}

// Epilogue of a wave that holds 32 output channels x 128 pixels as four
// transposed 32 x 32 blocks (the MFMA computed pixels x channels: block nj,
// accumulator v of lane l is channel l % 32, pixel nj*32 + 8 (v/4) +
// 4 (l/32) + v % 4, so a lane holds runs of 4 consecutive pixels of one
// channel).  Bias, ReLU and the rounding to T happen in registers; the block
// is staged once in LDS (`stage`: 8 KiB, [channel][128 pixels] in 16-byte
// units XOR-swizzled by the channel) and leaves as whole 256-byte channel
// rows, four per store instruction, the pattern that reaches the HBM write
// rate.  A run of 8 pixels inside one image is one 16-byte store (2-byte
// alignment is enough on gfx950); a run that crosses an image boundary or
// passes the last pixel is stored element by element.  Split-K partials
// (fp32) are staged in two halves of 64 pixels.  Precondition (the callers'
// plans guarantee it): a run crosses at most one image boundary, i.e.
// P*Q >= 8 or the tile index space pads planes to a multiple of 8.
template <typename T>
__device__ __forceinline__ void store_block128t(const f32x16_t (&acc)[1][4], float* stage_f, const EpiArgs& e,
                                                int row0, int col0, int g, int split, bool bias_in_acc = false) {
  const int lane = threadIdx.x & 63;
  const int l32 = lane & 31, h = lane >> 5;
  const int PQ = e.PQ;
  char* stage = reinterpret_cast<char*>(stage_f);
  const int64_t next_img = static_cast<int64_t>(e.K - 1) * PQ;
  using Run = Run128t;
  auto run_at = [&](int px) { return run128t(e, row0, col0, g, px); };

  if (e.splits <= 1) {
    // (bias_in_acc: the accumulators started from the bias.)
    const T* bias = bias_in_acc ? nullptr : reinterpret_cast<const T*>(e.b);
    const int i_own = row0 + l32;
    const float bv = (bias && i_own < e.Kg) ? elem<T>::load(bias + g * e.Kg + i_own) : 0.f;
    // Channel l32, pixels px0 .. px0 + 3 (8 bytes of T = bf16; fp32 goes
    // through the partial path's layout below).  Bias and ReLU are uniform
    // choices: without them the 64 values per lane only need rounding, and
    // the per-value add and select are not issued at all.
    static_assert(sizeof(T) == 2, "bf16 output");
    auto stage_all = [&](auto with_bias, auto with_relu) {
#pragma unroll
      for (int nj = 0; nj < 4; ++nj)
#pragma unroll
        for (int gg = 0; gg < 4; ++gg) {
          float v4[4];
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            v4[k] = acc[0][nj][4 * gg + k];
            if constexpr (decltype(with_bias)::value) v4[k] += bv;
            if constexpr (decltype(with_relu)::value) v4[k] = fmaxf(v4[k], 0.f);
          }
          uint2 w;
          w.x = f32x2_to_bf16x2(v4[0], v4[1]);
          w.y = f32x2_to_bf16x2(v4[2], v4[3]);
          const int px0 = nj * 32 + 8 * gg + 4 * h;
          *reinterpret_cast<uint2*>(stage + l32 * 256 + ((((px0 >> 3) ^ (l32 & 15))) << 4) + ((px0 >> 2) & 1) * 8) = w;
        }
    };
    using F = std::false_type;
    using Tr = std::true_type;
    if (bias) {
      if (e.relu && !e.res) stage_all(Tr{}, Tr{}); else stage_all(Tr{}, F{});
    } else {
      if (e.relu && !e.res) stage_all(F{}, Tr{}); else stage_all(F{}, F{});
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes are done
    __builtin_amdgcn_wave_barrier();
    // Lane l: channel rows l/16 + 4 it (it = 0..7), 16-byte unit l % 16.
    const int rrow = lane >> 4, u = lane & 15;
    const Run r = run_at(u * 8);
    uint4 d[8];
#pragma unroll
    for (int it = 0; it < 8; ++it) {
      const int row = rrow + 4 * it;
      d[it] = *reinterpret_cast<const uint4*>(stage + row * 256 + ((u ^ (row & 15)) << 4));
    }
    T* y = reinterpret_cast<T*>(e.y);
    // Common case: no residual, every lane's run is whole and the launch's
    // output fits a buffer resource.  Then each row is one buffer store
    // whose scalar offset steps by four channel rows, and rows past Kg get
    // an offset past the buffer (the store is dropped): no per-row address
    // arithmetic and no branches.
    if (!e.res && e.y_bytes != 0 && __builtin_amdgcn_ballot_w64(!r.full) == 0) {
      const __amdgpu_buffer_rsrc_t yr = make_rsrc(e.y, e.y_bytes);
      const uint32_t vo = static_cast<uint32_t>((r.o + static_cast<int64_t>(rrow) * PQ) * 2);
      const uint32_t step = static_cast<uint32_t>(4 * PQ * 2);
      const int rows_left = e.Kg - row0 - rrow;  // rows of this lane below Kg: it < ceil(rows_left / 4)
#pragma unroll
      for (int it = 0; it < 8; ++it) {
        const uint32_t v = 4 * it < rows_left ? vo : 0x80000000u;
        __builtin_amdgcn_raw_buffer_store_b128(*reinterpret_cast<const u32x4_t*>(&d[it]), yr, v, step * it, 0);
      }
      __builtin_amdgcn_wave_barrier();
      return;
    }
    if (e.res) {  // uniform: residual add (and the ReLU after it), then the same stores
      // Whole runs: all eight rows are requested before any is used, so the
      // loads overlap (one memory round trip per tile, not one per row).
      uint4 rr[8];
      if (r.full) {
        const uint16_t* rp = reinterpret_cast<const uint16_t*>(e.res);
#pragma unroll
        for (int it = 0; it < 8; ++it) {
          const int row = rrow + 4 * it;
          rr[it] = make_uint4(0u, 0u, 0u, 0u);
          if (row0 + row < e.Kg) __builtin_memcpy(&rr[it], rp + r.o + static_cast<int64_t>(row) * PQ, 16);
        }
      }
#pragma unroll
      for (int it = 0; it < 8; ++it) {
        const int row = rrow + 4 * it;
        if (row0 + row >= e.Kg || r.nvalid <= 0) continue;
        const int64_t o = r.o + static_cast<int64_t>(row) * PQ;
        const uint32_t w[4] = {d[it].x, d[it].y, d[it].z, d[it].w};
        float v[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) v[t] = __uint_as_float((w[t >> 1] >> (16 * (t & 1))) << 16);
        if (r.full) {  // the staged values are bf16 already
          const uint32_t q[4] = {rr[it].x, rr[it].y, rr[it].z, rr[it].w};
#pragma unroll
          for (int t = 0; t < 8; ++t) v[t] += __uint_as_float((q[t >> 1] >> (16 * (t & 1))) << 16);
        } else {
          add_residual_run<T>(v, e, o, false, r.nvalid, r.wrap, PQ, next_img);
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
    for (int it = 0; it < 8; ++it) {
      const int row = rrow + 4 * it;
      if (row0 + row >= e.Kg || r.nvalid <= 0) continue;
      const int64_t o = r.o + static_cast<int64_t>(row) * PQ;
      if (r.full) {
        __builtin_memcpy(y + o, &d[it], 16);
      } else {
        const uint32_t wd[4] = {d[it].x, d[it].y, d[it].z, d[it].w};
#pragma unroll
        for (int t = 0; t < 8; ++t)
          if (t < r.nvalid)
            reinterpret_cast<uint16_t*>(y)[o + t + (t >= r.wrap ? next_img : 0)] =
                static_cast<uint16_t>(wd[t >> 1] >> (16 * (t & 1)));
      }
    }
    __builtin_amdgcn_wave_barrier();
    return;
  }

  // fp32 partial sums: two passes of 32 channels x 64 pixels (256 bytes per
  // channel row, 16-byte units swizzled by the channel).
  float* part = e.partial + static_cast<int64_t>(split) * e.slab;
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int gg = 0; gg < 4; ++gg) {
        const int px0 = q * 32 + 8 * gg + 4 * h;  // within the 64-pixel half
        const float4 v = make_float4(acc[0][2 * pass + q][4 * gg], acc[0][2 * pass + q][4 * gg + 1],
                                     acc[0][2 * pass + q][4 * gg + 2], acc[0][2 * pass + q][4 * gg + 3]);
        *reinterpret_cast<float4*>(stage + l32 * 256 + (((px0 >> 2) ^ (l32 & 15)) << 4)) = v;
      }
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();
    // Lane l: channel rows l/8 + 8 it (it = 0..3), pixels 8 (l % 8) .. +7 of the half.
    const int rrow = lane >> 3, c = lane & 7;
    const Run r = run_at(pass * 64 + c * 8);
    float4 lo[4], hi[4];
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int row = rrow + 8 * it;
      lo[it] = *reinterpret_cast<const float4*>(stage + row * 256 + (((2 * c) ^ (row & 15)) << 4));
      hi[it] = *reinterpret_cast<const float4*>(stage + row * 256 + (((2 * c + 1) ^ (row & 15)) << 4));
    }
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int row = rrow + 8 * it;
      if (row0 + row >= e.Kg || r.nvalid <= 0) continue;
      const int64_t o = r.o + static_cast<int64_t>(row) * PQ;
      if (r.full) {
        __builtin_memcpy(part + o, &lo[it], 16);
        __builtin_memcpy(part + o + 4, &hi[it], 16);
      } else {
        const float vals[8] = {lo[it].x, lo[it].y, lo[it].z, lo[it].w, hi[it].x, hi[it].y, hi[it].z, hi[it].w};
#pragma unroll
        for (int t = 0; t < 8; ++t)
          if (t < r.nvalid) part[o + t + (t >= r.wrap ? next_img : 0)] = vals[t];
      }
    }
    __builtin_amdgcn_wave_barrier();  // the next pass reuses this wave's stage
  }
}

// The epilogue of one BM x BN tile (rows k0.. of group g, pixels j0..)
// computed by four waves in a 2 x 2 layout, each holding (BM/2) x 64; the
// caller provides 32 KiB of LDS (8 KiB per wave).
template <typename T, int BM>
__device__ __forceinline__ void store_tile(const f32x16_t (&acc)[BM / 64][BN / 64], vec16* smem, const EpiArgs& e,
                                           int j0, int k0, int g, int split) {
  static_assert(BN / 2 == 64, "staging layout assumes 64 pixels per wave row");
  const int wave = (threadIdx.x >> 6) & 3;
  const int wm = wave >> 1, wn = wave & 1;
  float* stage = reinterpret_cast<float*>(smem) + wave * 32 * 64;
  store_block<T, BM / 64, BN / 64>(acc, stage, e, k0 + wm * (BM / 2), j0 + wn * (BN / 2), g, split);
}

// s_waitcnt with vmcnt = n and the other counters at their maximum (gfx9 encoding).
#define CONVSEL_WAIT_VMCNT(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (((n) >> 4) << 14) | (7 << 4) | (15 << 8))

// The same for a count known only at run time (0 .. 63; uniform).
__device__ __forceinline__ void wait_vmcnt(int n) {
  static_for<64>([&](auto m) {
    if (n == decltype(m)::value) CONVSEL_WAIT_VMCNT(decltype(m)::value);
  });
}

typedef short v4s_t __attribute__((ext_vector_type(4)));
typedef short v8s_t __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v4s_t lds_v4s_t;
typedef __attribute__((address_space(3))) void lds_void_t;

// Sum of the split partials, plus bias, ReLU, rounding to the output type;
// kReducePer consecutive outputs per thread (flat index: outputs stay below
// 2^31), read and written as vectors when all of them exist; the channel of
// each output is found with one division per thread, then stepped.
constexpr int kReducePer = 4;
inline unsigned reduce_blocks(int total) { return (unsigned)((total + 256 * kReducePer - 1) / (256 * kReducePer)); }

template <typename T>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part, const T* __restrict__ bias,
                                                            T* __restrict__ y, int total, int slab, int PQ, int K,
                                                            int splits, int relu, const T* __restrict__ res) {
  constexpr int R = kReducePer;
  static_assert(R % 4 == 0, "whole float4 partial loads");
  const int64_t i0l = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * R;
  if (i0l >= total) return;
  const int i0 = static_cast<int>(i0l);
  const int nr = total - i0 < R ? total - i0 : R;
  float sum[R];
#pragma unroll
  for (int e = 0; e < R; ++e) sum[e] = 0.f;
  for (int s = 0; s < splits; ++s) {
    const float* p = part + static_cast<int64_t>(s) * slab + i0;
    if (nr == R) {
#pragma unroll
      for (int e = 0; e < R; e += 4) {
        const float4 v = *reinterpret_cast<const float4*>(p + e);  // slabs and i0 are multiples of 4 floats
        sum[e] += v.x; sum[e + 1] += v.y; sum[e + 2] += v.z; sum[e + 3] += v.w;
      }
    } else {
      for (int e = 0; e < nr; ++e) sum[e] += p[e];
    }
  }
  if (bias) {
    const int plane = i0 / PQ;
    int q = i0 - plane * PQ, ch = plane % K;
#pragma unroll
    for (int e = 0; e < R; ++e) {
      if (e > 0 && ++q == PQ) {
        q = 0;
        if (++ch == K) ch = 0;
      }
      sum[e] += elem<T>::load(bias + ch);
    }
  }
  typedef typename elem<T>::storage S;
  if (nr == R) {
    if (res) {  // see EpiArgs::res
      S r[R];
      __builtin_memcpy(r, res + i0, sizeof(r));
#pragma unroll
      for (int e = 0; e < R; ++e) {
        T re;
        __builtin_memcpy(&re, &r[e], sizeof(T));
        sum[e] = elem<T>::to_f32(elem<T>::from_f32(sum[e])) + elem<T>::to_f32(re);
      }
    }
    S o[R];
#pragma unroll
    for (int e = 0; e < R; ++e) {
      const T t = elem<T>::from_f32(relu ? fmaxf(sum[e], 0.f) : sum[e]);
      __builtin_memcpy(&o[e], &t, sizeof(T));
    }
    __builtin_memcpy(y + i0, o, sizeof(o));
    return;
  }
  for (int e = 0; e < nr; ++e) {
    const int i = i0 + e;
    float v = sum[e];
    if (res) v = elem<T>::to_f32(elem<T>::from_f32(v)) + elem<T>::load(res + i);  // see EpiArgs::res
    if (relu) v = fmaxf(v, 0.f);
    elem<T>::store(y + i, v);
  }
}

// Largest halo span (in virtual rows) over all pixel tiles of N images.  The
// span of a tile depends only on where it starts within an image, which
// repeats every PQ / gcd(BN, PQ) tiles, so one period is scanned.
inline int halo_rows(const Shape& s, int64_t N, int Hv) {
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

inline void split_chunks(int64_t tiles, int nch, int* splits, int* chunks_per_split) {
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
  *chunks_per_split = (nch + best - 1) / best;
  *splits = (nch + *chunks_per_split - 1) / *chunks_per_split;
}

inline size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// Store piece of the epilogue (store_tile): the largest of 8, 4, 2, 1
// elements that divides P*Q and whose stores stay aligned in y.
inline int store_piece(const Shape& s, const void* y) {
  const int64_t PQ = s.P * s.Q;
  for (int r = 8; r > 1; r >>= 1) {
    const int64_t align = r * s.esize() < 16 ? r * s.esize() : 16;
    if (PQ % r == 0 && reinterpret_cast<uintptr_t>(y) % align == 0) return r;
  }
  return 1;
}




}  // namespace igemm
}  // namespace convsel
