// Host-side interface between the C ABI (api.hip) and the kernel launchers.
// Every launcher enqueues on `stream` and returns the HIP status of its last
// launch; shapes are validated by the caller before any launcher runs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

namespace convsel {

enum { DT_F32 = 0, DT_BF16 = 1 };

// A validated layer with its derived sizes.
struct Shape {
  int64_t N, C, H, W, K, R, S, P, Q;
  int64_t Cg, Kg;
  int sh, sw, ph, pw, dh, dw, G;
  int dtype;
  bool bias, relu;
  int64_t esize() const { return dtype == DT_F32 ? 4 : 2; }
};

// Batched "NT" GEMM on MFMA:  C[b][i][j] = sum_k A[b][i][k] * B[b][j][k]
// (+ bias[b1*sBias1 + i], then ReLU), i < M, j < N, k < Kred.  Both operands
// are reduction-contiguous (row-major with leading dimensions lda / ldb),
// unless b_kmajor is set: then B is read as B[b][k][j] (leading dimension
// ldb along k).
// Batch b is split as b0 = b / bdiv, b1 = b % bdiv and every operand is
// offset by b0*s?0 + b1*s?1 elements.  C is stored in the data type, or in
// fp32 when out_f32 is set.
struct GemmArgs {
  const void* A;
  const void* B;
  void* C;
  const void* bias;
  int M, N, Kred;
  int64_t lda, ldb, ldc;
  int batch, bdiv;
  int64_t sA0, sA1, sB0, sB1, sC0, sC1;
  int64_t sBias1;
  int relu;
  int out_f32;
  int b_kmajor;
  // Set inside launch_gemm_nt only: with jspan > 0, column j of C is column
  // j % jspan of batch item j / jspan (sCj apart), for a batch folded into N.
  int jspan = 0;
  int64_t sCj = 0;
};

hipError_t launch_gemm_nt(int dtype, const GemmArgs& g, hipStream_t stream);

// Byte copy of `bytes` from src to dst (dst 16-byte aligned).
hipError_t launch_copy(const void* src, void* dst, size_t bytes, hipStream_t stream);

// Implicit GEMM over filter rows (bf16, one group, 5 <= S <= 8, S + (pw % 2)
// <= 8, even column stride, C*R <= 64: the wide-filter, few-channel layers
// such as a 7x7 stem).  The filter package (rows_packed_bytes) is the LDS
// image of each 64-channel tile; no other workspace.
bool rows_applies(const Shape& s);
size_t rows_packed_bytes(const Shape& s);
hipError_t rows_pack(const Shape& s, const void* w, void* wp, hipStream_t stream);
hipError_t rows_main(const Shape& s, const void* x, const void* wp, const void* b, void* y, hipStream_t stream,
                     const void* res = nullptr);
std::string rows_describe(const Shape& s);

// Implicit GEMM for bf16 3x3 layers, stride 1 or 2, dilation 1, one group,
// C a multiple of 16, W >= 4, P*Q >= 8; workspace: the filter package (when
// used) and split-K partials (k3_split_bytes).
bool k3_applies(const Shape& s);
// Whether prepacked calls copy the filter tiles by DMA from a package
// (k3_package_bytes, built by k3_pack from the KCRS filters); otherwise, and
// in every per-call conv2d(), the kernel reads the KCRS filters as given.
bool k3_uses_package(const Shape& s);
size_t k3_package_bytes(const Shape& s);
hipError_t k3_pack(const Shape& s, const void* w, void* pk, hipStream_t stream);
size_t k3_split_bytes(const Shape& s);
hipError_t k3_main(const Shape& s, const void* x, const void* w, const void* b, void* y, void* part_ws,
                   hipStream_t stream, const void* res = nullptr, bool prepacked = false);
std::string k3_describe(const Shape& s, bool prepacked = false);

// Implicit GEMM with loader and compute waves (bf16, one group, nine taps,
// C > 8): its own filter package ([16-channel chunk][K padded][19 units]),
// plus split-K partials.
bool ws_applies(const Shape& s);
size_t ws_packed_bytes(const Shape& s);
size_t ws_split_bytes(const Shape& s);
hipError_t ws_pack(const Shape& s, const void* w, void* wp, hipStream_t stream);
hipError_t ws_main(const Shape& s, const void* x, const void* wp, const void* b, void* y, void* part_ws,
                   hipStream_t stream, const void* res = nullptr);
std::string ws_describe(const Shape& s);

// direct convolution (VALU), all N images.
std::string direct_describe(const Shape& s);
hipError_t launch_direct(const Shape& s, const void* x, const void* w, const void* b, void* y,
                         hipStream_t stream);

// implicit GEMM (MFMA), all N images.  Layers whose output tiles alone
// would leave CUs idle split the channel reduction over several workgroups;
// they need implicit_gemm_workspace(s) bytes of fp32 partial sums in ws.
// The filters are first repacked (launch_implicit_pack, packed_bytes of
// space); the main kernel then reads only the packed copy.
bool implicit_gemm_fits(const Shape& s);
size_t implicit_gemm_packed_bytes(const Shape& s);
size_t implicit_gemm_split_bytes(const Shape& s);
size_t implicit_gemm_workspace(const Shape& s);  // packed filters (256-aligned) + split partials
hipError_t launch_implicit_pack(const Shape& s, const void* w, void* wp, hipStream_t stream);
hipError_t launch_implicit_main(const Shape& s, const void* x, const void* wp, const void* b, void* y, void* part,
                                hipStream_t stream, const void* res = nullptr);
hipError_t launch_implicit_gemm(const Shape& s, const void* x, const void* w, const void* b, void* y, void* ws,
                                hipStream_t stream);
std::string implicit_gemm_describe(const Shape& s);


// Implicit precomputed-index GEMM: the package holds the zero-padded
// filters and the reduction and pixel index tables; no other workspace.
bool precomp_applies(const Shape& s);
size_t precomp_packed_bytes(const Shape& s);
hipError_t precomp_pack(const Shape& s, const void* w, void* pkg, hipStream_t stream);
hipError_t precomp_main(const Shape& s, const void* x, const void* pkg, const void* b, void* y, hipStream_t stream);
std::string precomp_describe(const Shape& s);

// KN2ROW: the package is the tap-stacked filter matrix; the workspace holds
// the fp32 partial planes Z of a batch of images (kn2row_z_bytes).
bool kn2row_applies(const Shape& s);
size_t kn2row_packed_bytes(const Shape& s);
size_t kn2row_z_bytes(const Shape& s);
hipError_t kn2row_pack(const Shape& s, const void* w, void* wst, hipStream_t stream);
hipError_t kn2row_main(const Shape& s, const void* x, const void* wst, const void* b, void* y, void* z,
                       hipStream_t stream);
std::string kn2row_describe(const Shape& s);

// SMM: the package holds the filters in blocks of output channels; the
// workspace holds the zero-packed input of a batch of images.
bool smm_applies(const Shape& s);
size_t smm_packed_bytes(const Shape& s);
size_t smm_zero_pack_bytes(const Shape& s);
hipError_t smm_pack(const Shape& s, const void* w, void* wp, hipStream_t stream);
hipError_t smm_main(const Shape& s, const void* x, const void* wp, const void* b, void* y, void* zp,
                    hipStream_t stream);
std::string smm_describe(const Shape& s);

// Column matrix [nb][G][P*Q][Cg*R*S] of images n0 .. n0+nb-1.
hipError_t launch_im2col(const Shape& s, const void* x, void* col, int64_t n0, int64_t nb,
                         hipStream_t stream);

// Winograd F(2x2,3x3) pieces.  U: 16 x K x C.  V: 16 x Tc x C and M: 16 x K x Tc
// (fp32) for the Tc = nb*TP*TQ tiles of images n0 .. n0+nb-1.
hipError_t launch_wino_filter(const Shape& s, const void* w, void* U, hipStream_t stream);
hipError_t launch_wino_input(const Shape& s, const void* x, void* V, int64_t n0, int64_t nb,
                             hipStream_t stream);
hipError_t launch_wino_output(const Shape& s, const float* M, const void* b, void* y, int64_t n0,
                              int64_t nb, hipStream_t stream);

}  // namespace convsel
