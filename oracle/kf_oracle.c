/*
 * Plain fp64 reference contractions for the fused-chain oracle.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header or table with the HIP
 * library.
 *
 * What is computed (paper, Methodology / Overview and Appendix A "Operator
 * Fusion": the task is a PyTorch operator given as a reference computation,
 * and a candidate must reproduce it exactly up to rounding):
 *
 *   kfo_gemm_rows   h[i][j] = sum_k a[i][k] * b(k, j)
 *                   b(k, j) = b[k*N + j] (layout KN) or b[j*K + k] (layout NK)
 *   kfo_conv2d_3x3  PyTorch Conv2d cross-correlation, stride 1, zero padding 1,
 *                   dilation 1, groups 1, NCHW input / OIHW weight:
 *                   out[n][co][oh][ow] = sum_{ci,kh,kw}
 *                       in[n][ci][oh+kh-1][ow+kw-1] * w[co][ci][kh][kw]
 *                   with in[...] = 0 outside [0,H) x [0,W).
 *   kfo_conv3d_3x3x3 PyTorch Conv3d cross-correlation, 3x3x3 kernel, stride 1,
 *                   no padding, NCDHW input / OIDHW weight (the conv of the
 *                   paper's Conv3d -> softmax -> max-pool case study,
 *                   Appendix C):
 *                   out[n][co][od][oh][ow] = sum_{ci,kd,kh,kw}
 *                       in[n][ci][od+kd][oh+kh][ow+kw] * w[co][ci][kd][kh][kw].
 *
 * Every sum runs over its index in ascending order in double precision; no
 * blocking, reordering or fusion is applied.  Rows (GEMM) or images (conv)
 * are independent and are spread over OpenMP threads.
 */
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int kfo_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* rows[r] selects which row of a to use; out is nrows x N, row-major. */
void kfo_gemm_rows(const double* a, const double* b, int64_t M, int64_t N,
                   int64_t K, int b_layout_nk, const int64_t* rows,
                   int64_t nrows, double* out) {
  (void)M;
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < nrows; ++r) {
    const double* ai = a + rows[r] * K;
    double* hi = out + r * N;
    if (!b_layout_nk) {
      /* h[i][j] accumulates a[i][k]*b[k][j] for k = 0, 1, ..., K-1. */
      memset(hi, 0, sizeof(double) * (size_t)N);
      for (int64_t k = 0; k < K; ++k) {
        const double aik = ai[k];
        const double* bk = b + k * N;
        for (int64_t j = 0; j < N; ++j) hi[j] += aik * bk[j];
      }
    } else {
      for (int64_t j = 0; j < N; ++j) {
        const double* bj = b + j * K;
        double s = 0.0;
        for (int64_t k = 0; k < K; ++k) s += ai[k] * bj[k];
        hi[j] = s;
      }
    }
  }
}

/* images[t] selects which batch entry to compute; out is nimg x Cout x H x W. */
void kfo_conv2d_3x3(const double* in, const double* w, int64_t Nb,
                    int64_t Cin, int64_t H, int64_t W, int64_t Cout,
                    const int64_t* images, int64_t nimg, double* out) {
  (void)Nb;
  const int64_t plane = H * W;
#pragma omp parallel for collapse(2) schedule(static)
  for (int64_t t = 0; t < nimg; ++t) {
    for (int64_t co = 0; co < Cout; ++co) {
      const double* img = in + images[t] * Cin * plane;
      double* o = out + (t * Cout + co) * plane;
      for (int64_t oh = 0; oh < H; ++oh) {
        for (int64_t ow = 0; ow < W; ++ow) {
          double s = 0.0;
          for (int64_t ci = 0; ci < Cin; ++ci) {
            for (int64_t kh = 0; kh < 3; ++kh) {
              const int64_t ih = oh + kh - 1;
              if (ih < 0 || ih >= H) continue;
              for (int64_t kw = 0; kw < 3; ++kw) {
                const int64_t iw = ow + kw - 1;
                if (iw < 0 || iw >= W) continue;
                s += img[ci * plane + ih * W + iw] *
                     w[((co * Cin + ci) * 3 + kh) * 3 + kw];
              }
            }
          }
          o[oh * W + ow] = s;
        }
      }
    }
  }
}

/* images[t] selects which batch entry to compute; out is nimg x Cout x Do x
 * Ho x Wo with Do = D-2, Ho = H-2, Wo = W-2.  PyTorch Conv3d (the 3-D
 * cross-correlation) with a 3x3x3 kernel, stride 1, no padding, dilation 1,
 * groups 1, NCDHW input / OIDHW weight:
 *   out[n][co][od][oh][ow] = sum_{ci,kd,kh,kw}
 *       in[n][ci][od+kd][oh+kh][ow+kw] * w[co][ci][kd][kh][kw]
 * Every input index stays inside the volume, so no padding value enters. */
void kfo_conv3d_3x3x3(const double* in, const double* w, int64_t Nb,
                      int64_t Cin, int64_t D, int64_t H, int64_t W,
                      int64_t Cout, const int64_t* images, int64_t nimg,
                      double* out) {
  (void)Nb;
  const int64_t Do = D - 2, Ho = H - 2, Wo = W - 2;
  const int64_t vol = D * H * W, ovol = Do * Ho * Wo;
#pragma omp parallel for collapse(2) schedule(static)
  for (int64_t t = 0; t < nimg; ++t) {
    for (int64_t co = 0; co < Cout; ++co) {
      const double* img = in + images[t] * Cin * vol;
      double* o = out + (t * Cout + co) * ovol;
      for (int64_t od = 0; od < Do; ++od) {
        for (int64_t oh = 0; oh < Ho; ++oh) {
          for (int64_t ow = 0; ow < Wo; ++ow) {
            double s = 0.0;
            for (int64_t ci = 0; ci < Cin; ++ci) {
              for (int64_t kd = 0; kd < 3; ++kd) {
                for (int64_t kh = 0; kh < 3; ++kh) {
                  for (int64_t kw = 0; kw < 3; ++kw) {
                    s += img[ci * vol + ((od + kd) * H + (oh + kh)) * W + (ow + kw)] *
                         w[(((co * Cin + ci) * 3 + kd) * 3 + kh) * 3 + kw];
                  }
                }
              }
            }
            o[(od * Ho + oh) * Wo + ow] = s;
          }
        }
      }
    }
  }
}
