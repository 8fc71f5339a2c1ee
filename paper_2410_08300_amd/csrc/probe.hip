// Measurement probes for the roofline denominators: the MFMA rate with the
// operands in registers, and a plain 16-byte copy.  Neither is part of a
// convolution; bench.py times them beside the step so that each fraction of
// peak can also be read against what this machine delivers.
#include "common.hpp"
#include "kernels.hpp"
#include "convsel.h"

namespace convsel {

namespace {

// Every wave issues `iters` rounds of eight independent 32 x 32 MFMAs (eight
// accumulators, so no MFMA waits for the previous one's result), then folds
// its accumulators into one float per lane.
template <bool BF16>
__global__ __launch_bounds__(256) void mfma_probe_kernel(int iters, float* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  f32x16_t acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = zero16();
  const float av = 1e-3f * static_cast<float>(lane + 1), bv = 1e-3f * static_cast<float>(64 - lane);
  if constexpr (BF16) {
    bf16x8_t a, b;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      a[e] = static_cast<__bf16>(av);
      b[e] = static_cast<__bf16>(bv);
    }
    for (int i = 0; i < iters; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
  } else {
    for (int i = 0; i < iters; ++i)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc[j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int v = 0; v < 16; ++v) s += acc[j][v];
  sink[static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x] = s;
}

}  // namespace

}  // namespace convsel

extern "C" {

conv_status_t conv2d_probe_mfma(int32_t dtype, int32_t blocks, int32_t iters, float* sink, void* stream) {
  if (!sink || blocks <= 0 || iters <= 0 || (dtype != CONV_F32 && dtype != CONV_BF16)) return CONV_ERR_INVALID_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (dtype == CONV_BF16)
    hipLaunchKernelGGL(convsel::mfma_probe_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, st, (int)iters, sink);
  else
    hipLaunchKernelGGL(convsel::mfma_probe_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, st, (int)iters, sink);
  return hipGetLastError() == hipSuccess ? CONV_OK : CONV_ERR_DEVICE;
}

conv_status_t conv2d_probe_copy(const void* src, void* dst, size_t bytes, void* stream) {
  if ((!src || !dst) && bytes) return CONV_ERR_INVALID_ARG;
  if (bytes == 0) return CONV_OK;
  const hipError_t e = convsel::launch_copy(src, dst, bytes, static_cast<hipStream_t>(stream));
  return e == hipSuccess ? CONV_OK : CONV_ERR_DEVICE;
}

}  // extern "C"
