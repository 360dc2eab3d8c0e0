/*
 * WBMM oracle — TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.
 *
 * Plain, slow, fp64 CPU definition of the Windowed Batch Matrix Multiplication
 * operator (WBMM, "Windowed Batch Matrix Multiplication for Efficient Large
 * Receptive Field Convolution").  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark may build, load or call this file.  It
 * shares no source, header, table or helper with the HIP library.
 *
 * Every function is the operator's definition written out as loops, in the
 * paper's notation:
 *   X[B,C,H,W]   input feature map (Notation and Definitions, Sec. 3.1)
 *   R[C,(2wh-1)(2ww-1)]  relative position bias table (the "table" T)
 *   I[i,j] = (dh + wh - 1)(2ww - 1) + (dw + ww - 1),  dh = h_i - h_j,
 *            dw = w_i - w_j  (eq. index_computation, Sec. 3.4.2)
 *   M_c = R[c, I]  (eq. index_select)
 *   Y_batch = X_batch M  (Alg. 1, step 3) in the row-vector convention of
 *            Theorem 3.2: Y[.., j] = sum_i X[.., i] M[i, j], i = input
 *            position, j = output position, so dh/dw = input - output.
 *   Zero padding of H, W up to window multiples, output cropped afterwards
 *   (Sec. 3.4.1, "Handling Arbitrary Input Sizes"); padding sits at the
 *   bottom/right (the paper does not say where; this is the reading taken).
 *
 * The backward passes are not written out in the paper (it states only that
 * gradients flow through R, Sec. 3.4.5); they are the chain rule applied to the
 * forward loops below:
 *   dX[in]    = sum_{out in same window} dY[out] * R[c, I(in, out)]
 *   dR[c, k]  = sum_{b, windows} sum_{(in,out): I(in,out)=k} X[in] * dY[out]
 * with positions outside the image contributing zero (they are padding).
 *
 * Parallelism: OpenMP over (b, c) planes / channels only; the arithmetic of
 * every output element is a single sequential fp64 sum in loop order.
 */
#include <stdint.h>
#include <stddef.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Mutants for the test that shows the pins catch plausible mistakes.  Each is
 * selected at compile time with -DWBMM_ORACLE_MUTANT=k; the default build has
 * none.  1: transposed orientation (dh = output - input); 2: last input column
 * of each window dropped from the sum; 3: table row stride 2w instead of 2w-1;
 * 4: backward-table ignores the image boundary (reads padded outputs). */
#ifndef WBMM_ORACLE_MUTANT
#define WBMM_ORACLE_MUTANT 0
#endif

void wbmm_oracle_set_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

int wbmm_oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Table index of the offset (dh, dw) = input - output, eq. index_computation. */
static int64_t rel_index(int wh, int ww, int dh, int dw) {
#if WBMM_ORACLE_MUTANT == 1
  dh = -dh;
  dw = -dw;
#endif
#if WBMM_ORACLE_MUTANT == 3
  /* wrong row stride, wrapped into the table so the mutant stays in bounds */
  return ((int64_t)(dh + wh - 1) * (2 * ww) + (dw + ww - 1)) % ((int64_t)(2 * wh - 1) * (2 * ww - 1));
#else
  return (int64_t)(dh + wh - 1) * (2 * ww - 1) + (dw + ww - 1);
#endif
}

/* I[i, j] for window positions i, j in row-major order (i = h_i*ww + w_i),
 * eq. index_computation.  Writes d*d int32 values, d = wh*ww. */
void wbmm_oracle_relative_index(int wh, int ww, int32_t *I) {
  const int d = wh * ww;
  for (int i = 0; i < d; ++i) {
    const int hi = i / ww, xi = i % ww;
    for (int j = 0; j < d; ++j) {
      const int hj = j / ww, xj = j % ww;
      I[(int64_t)i * d + j] = (int32_t)rel_index(wh, ww, hi - hj, xi - xj);
    }
  }
}

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

/* Forward, Alg. 1: Y[b,c,h,x] = sum over input positions (hi, xi) of the
 * same window of X[b,c,hi,xi] * R[c, I(in, out)]; out-of-image inputs are the
 * zero padding and contribute nothing. */
void wbmm_oracle_forward(const double *x, const double *t, double *y, int64_t B,
                         int64_t C, int64_t H, int64_t W, int wh, int ww) {
  const int64_t K = (int64_t)(2 * wh - 1) * (2 * ww - 1);
  int64_t bc;
#pragma omp parallel for schedule(static)
  for (bc = 0; bc < B * C; ++bc) {
    const int64_t c = bc % C;
    const double *xp = x + bc * H * W;
    const double *tc = t + c * K;
    double *yp = y + bc * H * W;
    for (int64_t h = 0; h < H; ++h) {
      for (int64_t w = 0; w < W; ++w) {
        const int64_t wy = h / wh, wx = w / ww;
        const int ho = (int)(h % wh), xo = (int)(w % ww);
        double s = 0.0;
        for (int hi = 0; hi < wh; ++hi) {
          const int64_t gh = wy * wh + hi;
          if (gh >= H) continue;
#if WBMM_ORACLE_MUTANT == 2
          for (int xi = 0; xi < ww - 1; ++xi) {
#else
          for (int xi = 0; xi < ww; ++xi) {
#endif
            const int64_t gw = wx * ww + xi;
            if (gw >= W) continue;
            s += xp[gh * W + gw] * tc[rel_index(wh, ww, hi - ho, xi - xo)];
          }
        }
        yp[h * W + w] = s;
      }
    }
  }
}

/* Backward with respect to the input: chain rule on the forward loop.  Every
 * in-image input position receives the sum over the in-image output positions
 * of its window of dY[out] * R[c, I(in, out)]. */
void wbmm_oracle_backward_input(const double *dy, const double *t, double *dx,
                                int64_t B, int64_t C, int64_t H, int64_t W,
                                int wh, int ww) {
  const int64_t K = (int64_t)(2 * wh - 1) * (2 * ww - 1);
  int64_t bc;
#pragma omp parallel for schedule(static)
  for (bc = 0; bc < B * C; ++bc) {
    const int64_t c = bc % C;
    const double *gp = dy + bc * H * W;
    const double *tc = t + c * K;
    double *dp = dx + bc * H * W;
    for (int64_t h = 0; h < H; ++h) {
      for (int64_t w = 0; w < W; ++w) {
        const int64_t wy = h / wh, wx = w / ww;
        const int hi = (int)(h % wh), xi = (int)(w % ww);
        double s = 0.0;
        for (int ho = 0; ho < wh; ++ho) {
          const int64_t gh = wy * wh + ho;
          if (gh >= H) continue;
          for (int xo = 0; xo < ww; ++xo) {
            const int64_t gw = wx * ww + xo;
            if (gw >= W) continue;
            s += gp[gh * W + gw] * tc[rel_index(wh, ww, hi - ho, xi - xo)];
          }
        }
        dp[h * W + w] = s;
      }
    }
  }
}

/* Backward with respect to the table: dR[c, k] collects X[in] * dY[out] over
 * every batch image, every window and every in-image (in, out) pair whose
 * offset maps to k.  Written as one sequential sum per channel. */
void wbmm_oracle_backward_table(const double *x, const double *dy, double *dt,
                                int64_t B, int64_t C, int64_t H, int64_t W,
                                int wh, int ww) {
  const int64_t K = (int64_t)(2 * wh - 1) * (2 * ww - 1);
  const int64_t NH = ceil_div(H, wh), NW = ceil_div(W, ww);
  int64_t c;
#pragma omp parallel for schedule(static)
  for (c = 0; c < C; ++c) {
    double *dc = dt + c * K;
    for (int64_t k = 0; k < K; ++k) dc[k] = 0.0;
    for (int64_t b = 0; b < B; ++b) {
      const double *xp = x + (b * C + c) * H * W;
      const double *gp = dy + (b * C + c) * H * W;
      for (int64_t wy = 0; wy < NH; ++wy)
        for (int64_t wx = 0; wx < NW; ++wx)
          for (int hi = 0; hi < wh; ++hi)
            for (int xi = 0; xi < ww; ++xi) {
              const int64_t ih = wy * wh + hi, iw = wx * ww + xi;
              if (ih >= H || iw >= W) continue;
              const double xv = xp[ih * W + iw];
              for (int ho = 0; ho < wh; ++ho)
                for (int xo = 0; xo < ww; ++xo) {
                  const int64_t oh = wy * wh + ho, ow = wx * ww + xo;
#if WBMM_ORACLE_MUTANT == 4
                  const double gv = (oh < H && ow < W) ? gp[oh * W + ow] : 1.0;
#else
                  if (oh >= H || ow >= W) continue;
                  const double gv = gp[oh * W + ow];
#endif
                  dc[rel_index(wh, ww, hi - ho, xi - xo)] += xv * gv;
                }
            }
    }
  }
}

/* Hierarchical window reparameterisation, inference form (Sec. 3.6 and the
 * appendix algorithm "Inference Mode with Fused Hierarchical Matrix"):
 * global windows of size wg = 2*wl with table Rg[C,(2wg-1)^2], local 2x2
 * sub-windows of size wl with table Rl[C,(2wl-1)^2], and
 *   M_fused = M_g + diag_blocks(M_l + I_{wl^2}) + I_{wg^2}
 * where the local term links only positions of the same sub-window.  Y is
 * X_w M_fused per global window, padded and cropped like the plain forward.
 * The fused matrix of each channel is built explicitly (d x d, d = wg^2). */
void wbmm_oracle_hier_fused_matrix(const double *tg, const double *tl,
                                   double *m, int64_t C, int wl) {
  const int wg = 2 * wl;
  const int d = wg * wg;
  const int64_t Kg = (int64_t)(2 * wg - 1) * (2 * wg - 1);
  const int64_t Kl = (int64_t)(2 * wl - 1) * (2 * wl - 1);
  for (int64_t c = 0; c < C; ++c) {
    double *mc = m + c * (int64_t)d * d;
    for (int i = 0; i < d; ++i) {
      const int hi = i / wg, xi = i % wg;
      for (int j = 0; j < d; ++j) {
        const int hj = j / wg, xj = j % wg;
        double v = tg[c * Kg + rel_index(wg, wg, hi - hj, xi - xj)];
        const int same_sub = (hi / wl == hj / wl) && (xi / wl == xj / wl);
        if (same_sub) {
          /* local table indexed by the offset inside the sub-window */
          v += tl[c * Kl + rel_index(wl, wl, (hi % wl) - (hj % wl),
                                     (xi % wl) - (xj % wl))];
          if (i == j) v += 1.0; /* local identity shortcut */
        }
        if (i == j) v += 1.0; /* global identity shortcut */
        mc[(int64_t)i * d + j] = v;
      }
    }
  }
}

/* Y = X_w M_fused with the fused matrix given explicitly ([C, d, d], d =
 * wg^2); windows of size wg, zero padding to multiples of wg, crop after. */
void wbmm_oracle_dense_forward(const double *x, const double *m, double *y,
                               int64_t B, int64_t C, int64_t H, int64_t W,
                               int wh, int ww) {
  const int d = wh * ww;
  int64_t bc;
#pragma omp parallel for schedule(static)
  for (bc = 0; bc < B * C; ++bc) {
    const int64_t c = bc % C;
    const double *xp = x + bc * H * W;
    const double *mc = m + c * (int64_t)d * d;
    double *yp = y + bc * H * W;
    for (int64_t h = 0; h < H; ++h)
      for (int64_t w = 0; w < W; ++w) {
        const int64_t wy = h / wh, wx = w / ww;
        const int j = (int)(h % wh) * ww + (int)(w % ww);
        double s = 0.0;
        for (int hi = 0; hi < wh; ++hi) {
          const int64_t gh = wy * wh + hi;
          if (gh >= H) continue;
          for (int xi = 0; xi < ww; ++xi) {
            const int64_t gw = wx * ww + xi;
            if (gw >= W) continue;
            s += xp[gh * W + gw] * mc[(int64_t)(hi * ww + xi) * d + j];
          }
        }
        yp[h * W + w] = s;
      }
  }
}

/* Gradient of the dense form with respect to the per-channel matrix:
 * dM[c, i, j] = sum over images and windows of X[.., i] * dY[.., j], the
 * positions taken row-major inside each (zero-padded) window. */
void wbmm_oracle_dense_backward_matrix(const double *x, const double *dy, double *dm,
                                       int64_t B, int64_t C, int64_t H, int64_t W,
                                       int wh, int ww) {
  const int d = wh * ww;
  const int64_t NH = ceil_div(H, wh), NW = ceil_div(W, ww);
  int64_t c;
#pragma omp parallel for schedule(static)
  for (c = 0; c < C; ++c) {
    double *mc = dm + c * (int64_t)d * d;
    for (int64_t k = 0; k < (int64_t)d * d; ++k) mc[k] = 0.0;
    for (int64_t b = 0; b < B; ++b) {
      const double *xp = x + (b * C + c) * H * W;
      const double *gp = dy + (b * C + c) * H * W;
      for (int64_t wy = 0; wy < NH; ++wy)
        for (int64_t wx = 0; wx < NW; ++wx)
          for (int i = 0; i < d; ++i) {
            const int64_t hi = wy * wh + i / ww, xi = wx * ww + i % ww;
            if (hi >= H || xi >= W) continue;
            const double xv = xp[hi * W + xi];
            for (int j = 0; j < d; ++j) {
              const int64_t ho = wy * wh + j / ww, xo = wx * ww + j % ww;
              if (ho >= H || xo >= W) continue;
              mc[(int64_t)i * d + j] += xv * gp[ho * W + xo];
            }
          }
    }
  }
}
