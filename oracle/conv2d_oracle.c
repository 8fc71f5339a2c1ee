/*
 * Test infrastructure only.  This is the CPU oracle for the forward 2-D
 * convolution that every algorithm of the library must reproduce.  Only the
 * test suite, the smoke entry point and the benchmark's CPU-baseline leg may
 * load it; the product path never does.
 *
 * What it computes (paper, Sec. II-B and Sec. IV: every algorithm the
 * framework offers must give the same output as PyTorch's Conv2d, so the
 * operation is the plain definition of that layer's forward pass):
 *
 *   P = floor((H + 2*ph - dh*(R-1) - 1) / sh) + 1
 *   Q = floor((W + 2*pw - dw*(S-1) - 1) / sw) + 1
 *   y[n,k,p,q] = b[k] + sum_{c<C/G} sum_{r<R} sum_{s<S}
 *                xpad[n, g*C/G + c, p*sh - ph + r*dh, q*sw - pw + s*dw] * w[k,c,r,s]
 *   with g = k / (K/G) and xpad = x inside the image, 0 outside
 *   (cross-correlation: the filter is not flipped), then max(0, y) when the
 *   ReLU flag is set.
 *
 * Everything is fp64.  Callers widen fp32 / bf16 data exactly before the call,
 * so the oracle computes the exact convolution (up to fp64 rounding) of the very
 * values the GPU receives.  The order of the sum for every output element is
 * fixed (c, then r, then s), so the result does not depend on the thread count.
 * Build without -ffast-math.
 */
#include <stdint.h>
#include <stddef.h>

static int64_t out_extent(int64_t in, int64_t pad, int64_t dil, int64_t ker, int64_t stride) {
  int64_t span = in + 2 * pad - dil * (ker - 1) - 1;
  if (span < 0) return 0;
  return span / stride + 1;
}

/* Shape check shared by both entry points; returns 0 when the arguments
 * describe a valid convolution and writes P and Q. */
static int check_shape(int64_t N, int64_t C, int64_t H, int64_t W, int64_t K, int64_t R, int64_t S,
                       int64_t sh, int64_t sw, int64_t ph, int64_t pw, int64_t dh, int64_t dw,
                       int64_t G, int64_t* P, int64_t* Q) {
  if (N < 0 || C < 1 || H < 1 || W < 1 || K < 1 || R < 1 || S < 1) return 1;
  if (sh < 1 || sw < 1 || dh < 1 || dw < 1 || ph < 0 || pw < 0 || G < 1) return 1;
  if (C % G != 0 || K % G != 0) return 1;
  *P = out_extent(H, ph, dh, R, sh);
  *Q = out_extent(W, pw, dw, S, sw);
  if (*P < 1 || *Q < 1) return 1;
  return 0;
}

/* Full output: x is N*C*H*W, w is K*(C/G)*R*S, b is K values or NULL,
 * y is N*K*P*Q.  All row-major (NCHW / KCRS / NKPQ). */
int oracle_conv2d_f64(const double* x, const double* w, const double* b, double* y,
                      int64_t N, int64_t C, int64_t H, int64_t W, int64_t K, int64_t R, int64_t S,
                      int64_t sh, int64_t sw, int64_t ph, int64_t pw, int64_t dh, int64_t dw,
                      int64_t G, int32_t relu) {
  int64_t P, Q;
  if (check_shape(N, C, H, W, K, R, S, sh, sw, ph, pw, dh, dw, G, &P, &Q)) return 1;
  const int64_t Cg = C / G, Kg = K / G;
  int64_t nk;
#pragma omp parallel for schedule(static)
  for (nk = 0; nk < N * K; ++nk) {
    const int64_t n = nk / K, k = nk % K, g = k / Kg;
    double* out = y + nk * P * Q;
    const double init = b ? b[k] : 0.0;
    for (int64_t i = 0; i < P * Q; ++i) out[i] = init;
    for (int64_t c = 0; c < Cg; ++c) {
      const double* plane = x + (n * C + g * Cg + c) * H * W;
      for (int64_t r = 0; r < R; ++r) {
        for (int64_t s = 0; s < S; ++s) {
          const double wv = w[((k * Cg + c) * R + r) * S + s];
          for (int64_t p = 0; p < P; ++p) {
            const int64_t h = p * sh - ph + r * dh;
            if (h < 0 || h >= H) continue;
            double* orow = out + p * Q;
            const double* irow = plane + h * W;
            for (int64_t q = 0; q < Q; ++q) {
              const int64_t ww = q * sw - pw + s * dw;
              if (ww < 0 || ww >= W) continue;
              orow[q] += irow[ww] * wv;
            }
          }
        }
      }
    }
    if (relu)
      for (int64_t i = 0; i < P * Q; ++i) out[i] = out[i] > 0.0 ? out[i] : 0.0;
  }
  return 0;
}

/* Selected outputs only: idx holds npts rows of (n, k, p, q); out[i] receives
 * y[n,k,p,q] computed from the same definition, term by term in the same
 * (c, r, s) order as the full version.  Used for spot checks at sizes where
 * the full output would take too long on the host. */
int oracle_conv2d_points_f64(const double* x, const double* w, const double* b,
                             int64_t N, int64_t C, int64_t H, int64_t W, int64_t K, int64_t R, int64_t S,
                             int64_t sh, int64_t sw, int64_t ph, int64_t pw, int64_t dh, int64_t dw,
                             int64_t G, int32_t relu, const int64_t* idx, int64_t npts, double* out) {
  int64_t P, Q;
  if (check_shape(N, C, H, W, K, R, S, sh, sw, ph, pw, dh, dw, G, &P, &Q)) return 1;
  for (int64_t i = 0; i < npts; ++i) {
    const int64_t n = idx[4 * i], k = idx[4 * i + 1], p = idx[4 * i + 2], q = idx[4 * i + 3];
    if (n < 0 || n >= N || k < 0 || k >= K || p < 0 || p >= P || q < 0 || q >= Q) return 2;
  }
  const int64_t Cg = C / G, Kg = K / G;
  int64_t i;
#pragma omp parallel for schedule(static)
  for (i = 0; i < npts; ++i) {
    const int64_t n = idx[4 * i], k = idx[4 * i + 1], p = idx[4 * i + 2], q = idx[4 * i + 3];
    const int64_t g = k / Kg;
    double acc = b ? b[k] : 0.0;
    for (int64_t c = 0; c < Cg; ++c) {
      const double* plane = x + (n * C + g * Cg + c) * H * W;
      for (int64_t r = 0; r < R; ++r) {
        const int64_t h = p * sh - ph + r * dh;
        if (h < 0 || h >= H) continue;
        for (int64_t s = 0; s < S; ++s) {
          const int64_t ww = q * sw - pw + s * dw;
          if (ww < 0 || ww >= W) continue;
          acc += plane[h * W + ww] * w[((k * Cg + c) * R + r) * S + s];
        }
      }
    }
    out[i] = (relu && acc < 0.0) ? 0.0 : acc;
  }
  return 0;
}
