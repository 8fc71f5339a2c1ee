// Device-side helpers shared by the gfx950 kernels: element types, bf16
// conversion, 16-byte vector moves and the MFMA wrappers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace convsel {

// bf16 is carried as its 16-bit pattern.
struct bf16_t {
  uint16_t bits;
};

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// fp32 -> bf16, round to nearest, ties to even (the hardware conversion,
// v_cvt_pk_bf16_f32 on gfx950; NaN stays a quiet NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  const __bf16 h = static_cast<__bf16>(f);
  return __builtin_bit_cast(uint16_t, h);
}

// Two fp32 -> two bf16 packed in one word (first value in the low half).
__device__ __forceinline__ uint32_t f32x2_to_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  bf16x2_t v;
  v[0] = static_cast<__bf16>(lo);
  v[1] = static_cast<__bf16>(hi);
  return __builtin_bit_cast(uint32_t, v);
}

// Element-type traits: how one element is loaded as fp32 and stored from fp32.
template <typename T> struct elem;

template <> struct elem<float> {
  typedef float storage;
  static constexpr int bytes = 4;
  static constexpr int per16 = 4;  // elements in 16 bytes
  __device__ static __forceinline__ float load(const float* p) { return *p; }
  __device__ static __forceinline__ void store(float* p, float v) { *p = v; }
  __device__ static __forceinline__ float to_f32(float v) { return v; }
  __device__ static __forceinline__ float from_f32(float v) { return v; }
};

template <> struct elem<bf16_t> {
  typedef uint16_t storage;
  static constexpr int bytes = 2;
  static constexpr int per16 = 8;
  __device__ static __forceinline__ float load(const bf16_t* p) { return bf16_to_f32(p->bits); }
  __device__ static __forceinline__ void store(bf16_t* p, float v) { p->bits = f32_to_bf16(v); }
  __device__ static __forceinline__ float to_f32(bf16_t v) { return bf16_to_f32(v.bits); }
  __device__ static __forceinline__ bf16_t from_f32(float v) {
    bf16_t r;
    r.bits = f32_to_bf16(v);
    return r;
  }
};

// Raw element bits as a 32-bit integer (for packing into 16-byte vectors).
__device__ __forceinline__ uint32_t raw_bits(float v) { return __float_as_uint(v); }
__device__ __forceinline__ uint32_t raw_bits(bf16_t v) { return v.bits; }

// 16 bytes holding `elem<T>::per16` consecutive elements.
struct vec16 {
  uint32_t d[4];
};

template <typename T>
__device__ __forceinline__ void vec16_set(vec16& v, int i, T e);

template <>
__device__ __forceinline__ void vec16_set<float>(vec16& v, int i, float e) {
  v.d[i] = __float_as_uint(e);
}

template <>
__device__ __forceinline__ void vec16_set<bf16_t>(vec16& v, int i, bf16_t e) {
  const int w = i >> 1;
  if (i & 1)
    v.d[w] = (v.d[w] & 0x0000ffffu) | (static_cast<uint32_t>(e.bits) << 16);
  else
    v.d[w] = (v.d[w] & 0xffff0000u) | static_cast<uint32_t>(e.bits);
}

template <typename T>
__device__ __forceinline__ T vec16_get(const vec16& v, int i);

template <>
__device__ __forceinline__ float vec16_get<float>(const vec16& v, int i) {
  return __uint_as_float(v.d[i]);
}

template <>
__device__ __forceinline__ bf16_t vec16_get<bf16_t>(const vec16& v, int i) {
  bf16_t r;
  r.bits = static_cast<uint16_t>((i & 1) ? (v.d[i >> 1] >> 16) : (v.d[i >> 1] & 0xffffu));
  return r;
}

// Raw bits of one element, zero-extended to 32 bits.
__device__ __forceinline__ uint32_t load_bits(const float* p) { return __float_as_uint(*p); }
__device__ __forceinline__ uint32_t load_bits(const bf16_t* p) {
  return static_cast<uint32_t>(*reinterpret_cast<const uint16_t*>(p));
}

// Packs per16 element bit patterns (low bits of each word) into 16 bytes.
template <typename T>
__device__ __forceinline__ void pack16(vec16& v, const uint32_t* e);

template <>
__device__ __forceinline__ void pack16<float>(vec16& v, const uint32_t* e) {
  v.d[0] = e[0];
  v.d[1] = e[1];
  v.d[2] = e[2];
  v.d[3] = e[3];
}

template <>
__device__ __forceinline__ void pack16<bf16_t>(vec16& v, const uint32_t* e) {
  v.d[0] = e[0] | (e[1] << 16);
  v.d[1] = e[2] | (e[3] << 16);
  v.d[2] = e[4] | (e[5] << 16);
  v.d[3] = e[6] | (e[7] << 16);
}

__device__ __forceinline__ vec16 vec16_zero() {
  vec16 v;
  v.d[0] = v.d[1] = v.d[2] = v.d[3] = 0u;
  return v;
}

__device__ __forceinline__ vec16 load16(const void* p) {
  const uint4 u = *reinterpret_cast<const uint4*>(p);
  vec16 v;
  v.d[0] = u.x;
  v.d[1] = u.y;
  v.d[2] = u.z;
  v.d[3] = u.w;
  return v;
}

__device__ __forceinline__ void store16(void* p, const vec16& v) {
  *reinterpret_cast<uint4*>(p) = make_uint4(v.d[0], v.d[1], v.d[2], v.d[3]);
}

// ---------------------------------------------------------------------------
// MFMA.  A 32x32 output block per wave; `a` and `b` are one lane's 16-byte
// slice of the A row / B column (8 bf16 or 4 fp32 consecutive reduction
// elements).  For lane l: row/column index l % 32, reduction slice l / 32.
//
// bf16: one v_mfma_f32_32x32x16_bf16 consumes the 2 x 8 reduction elements.
// fp32: v_mfma_f32_32x32x2_f32 takes one element per lane, so four of them,
//       taking element t of both halves in step t, consume the same 2 x 4
//       elements (the pairing is identical for A and B, so the sum is the
//       full dot product over the slice).
// Accumulator layout (both): lane l, register v holds row
//   8*(v/4) + 4*(l/32) + (v%4) and column l % 32 of the 32x32 block.
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ void mfma_32x32(f32x16_t& acc, const vec16& a, const vec16& b);

template <>
__device__ __forceinline__ void mfma_32x32<bf16_t>(f32x16_t& acc, const vec16& a, const vec16& b) {
  bf16x8_t av, bv;
  __builtin_memcpy(&av, &a, 16);
  __builtin_memcpy(&bv, &b, 16);
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc, 0, 0, 0);
}

template <>
__device__ __forceinline__ void mfma_32x32<float>(f32x16_t& acc, const vec16& a, const vec16& b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.d[0]), __uint_as_float(b.d[0]), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.d[1]), __uint_as_float(b.d[1]), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.d[2]), __uint_as_float(b.d[2]), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.d[3]), __uint_as_float(b.d[3]), acc, 0, 0, 0);
}

// Row of the 32x32 block held by accumulator register v of lane `lane`.
__device__ __forceinline__ int mfma_row(int v, int lane) { return 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3); }

// Workgroup barrier that orders LDS accesses only.  __syncthreads() also
// waits for every outstanding global load and store of the wave
// (s_waitcnt vmcnt(0)), which would drain the prefetches and LDS-DMA loads
// the kernels keep in flight across their barriers; those are waited for
// explicitly where their data is used.
__device__ __forceinline__ void lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ f32x16_t zero16() {
  f32x16_t z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

}  // namespace convsel
