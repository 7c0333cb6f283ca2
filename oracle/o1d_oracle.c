/*
 * Reference oracle for depthwise convolution with oriented 1D kernels.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the library's product path may link,
 * load or call this file. It exists so that tests, the smoke check and the
 * benchmark's CPU baseline can compare the GPU kernels against a plain,
 * slow, obviously correct implementation of the paper's definition.
 *
 * Source: Kirchmeyer & Deng, "Convolutional Networks with Oriented 1D
 * Kernels" (ICCV 2023).
 *   - Definition 1, Eq. (1): y[n,p,q,c] = sum_k x[n,h,w,c] * w[k,c].
 *   - Eq. (2) and the 1D coordinate equation of the appendix ("1D
 *     formulation"):  h = str*p + floor(-(k-pad) * sin(theta_c)),
 *                     w = str*q + floor( (k-pad) * cos(theta_c)).
 *   - Appendix "Padding": odd K only, pad = floor(K/2), the pad sits
 *     inside the floor (the de-centred variant with "- pad" outside the
 *     floor is explicitly rejected).
 *
 * Readings taken where the paper is silent (each is also listed in the
 * design notes of the repository):
 *   R1  theta is given in degrees (the paper quotes all angles in degrees);
 *       it is converted to radians in double precision.
 *   R2  a product that is within 1e-9 of an integer is treated as that
 *       integer before the floor.  Without this, theta = 90 deg gives
 *       cos = 6e-17 and floor(-j*cos) = -1 for j > 0, and theta = 30 deg
 *       gives 2*sin = 0.99999999999999989 -> 0 instead of 1.
 *   R5  stride 1, output size P = H and Q = W; taps that fall outside
 *       the H x W plane read zero (zero padding).
 *   R7  tensors are NCHW, weights are [C][K] (Definition 1 writes NHWC and
 *       K x C; only the memory order differs).
 *   R8  duplicate taps (two k giving the same (dh, dw)) are summed, as the
 *       plain sum over k in Eq. (1) says.
 *
 * Everything is computed in double precision.  The backward passes are the
 * literal adjoint of Eq. (1) written in scatter form: for every term of the
 * forward sum that reads x[n,c,h,w] for output (p,q) through tap k,
 *     dx[n,c,h,w] += dy[n,c,p,q] * w[c,k]
 *     dw[c,k]     += dy[n,c,p,q] * x[n,c,h,w].
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_SNAP_EPS 1e-9

/* Real-valued filter offsets before rounding (appendix "Rotation vs
 * Shearing": (dh^k, dw^k) = R_theta (0, k - pad)^T), for an explicit pad. */
void oracle_offsets_real(double theta_deg, int K, int pad, double* dh_real, double* dw_real) {
  const double t = theta_deg * (M_PI / 180.0);
  const double s = sin(t), c = cos(t);
  for (int k = 0; k < K; ++k) {
    const double j = (double)(k - pad);
    dh_real[k] = -j * s;
    dw_real[k] = j * c;
  }
}

static double floor_snapped(double v) {
  const double r = nearbyint(v);
  if (fabs(v - r) <= ORACLE_SNAP_EPS) return r;
  return floor(v);
}

/* Integer filter offsets: floor of the real offsets (Eq. 2), with the
 * near-integer reading R2. */
void oracle_offsets(double theta_deg, int K, int pad, int* dh, int* dw) {
  double* vh = (double*)malloc(sizeof(double) * (size_t)K);
  double* vw = (double*)malloc(sizeof(double) * (size_t)K);
  oracle_offsets_real(theta_deg, K, pad, vh, vw);
  for (int k = 0; k < K; ++k) {
    dh[k] = (int)floor_snapped(vh[k]);
    dw[k] = (int)floor_snapped(vw[k]);
  }
  free(vh);
  free(vw);
}

/* Forward pass, Definition 1 with str = 1, pad = K/2. */
void oracle_fwd(const double* x, const double* wt, const double* theta_deg, double* y,
                int N, int C, int H, int W, int K, int nthreads) {
  const int pad = K / 2;
  const long planes = (long)N * C;
#pragma omp parallel for schedule(dynamic) num_threads(nthreads)
  for (long nc = 0; nc < planes; ++nc) {
    const int c = (int)(nc % C);
    int* dh = (int*)malloc(sizeof(int) * (size_t)K);
    int* dw = (int*)malloc(sizeof(int) * (size_t)K);
    oracle_offsets(theta_deg[c], K, pad, dh, dw);
    const double* xp = x + (size_t)nc * H * W;
    double* yp = y + (size_t)nc * H * W;
    for (int p = 0; p < H; ++p) {
      for (int q = 0; q < W; ++q) {
        double acc = 0.0;
        for (int k = 0; k < K; ++k) {
          const int h = p + dh[k];
          const int w = q + dw[k];
          if (h >= 0 && h < H && w >= 0 && w < W) acc += xp[(size_t)h * W + w] * wt[(size_t)c * K + k];
        }
        yp[(size_t)p * W + q] = acc;
      }
    }
    free(dh);
    free(dw);
  }
}

/* Gradient with respect to the input, scatter form of the adjoint. */
void oracle_bwd_input(const double* dy, const double* wt, const double* theta_deg, double* dx,
                      int N, int C, int H, int W, int K, int nthreads) {
  const int pad = K / 2;
  const long planes = (long)N * C;
#pragma omp parallel for schedule(dynamic) num_threads(nthreads)
  for (long nc = 0; nc < planes; ++nc) {
    const int c = (int)(nc % C);
    int* dh = (int*)malloc(sizeof(int) * (size_t)K);
    int* dw = (int*)malloc(sizeof(int) * (size_t)K);
    oracle_offsets(theta_deg[c], K, pad, dh, dw);
    const double* gp = dy + (size_t)nc * H * W;
    double* xp = dx + (size_t)nc * H * W;
    memset(xp, 0, sizeof(double) * (size_t)H * W);
    for (int p = 0; p < H; ++p) {
      for (int q = 0; q < W; ++q) {
        const double g = gp[(size_t)p * W + q];
        for (int k = 0; k < K; ++k) {
          const int h = p + dh[k];
          const int w = q + dw[k];
          if (h >= 0 && h < H && w >= 0 && w < W) xp[(size_t)h * W + w] += g * wt[(size_t)c * K + k];
        }
      }
    }
    free(dh);
    free(dw);
  }
}

/* Gradient with respect to the weights, scatter form of the adjoint.
 * Parallel over channels so that every dw[c][:] has a single writer. */
void oracle_bwd_weight(const double* x, const double* dy, const double* theta_deg, double* dwt,
                       int N, int C, int H, int W, int K, int nthreads) {
  const int pad = K / 2;
#pragma omp parallel for schedule(dynamic) num_threads(nthreads)
  for (int c = 0; c < C; ++c) {
    int* dh = (int*)malloc(sizeof(int) * (size_t)K);
    int* dw = (int*)malloc(sizeof(int) * (size_t)K);
    oracle_offsets(theta_deg[c], K, pad, dh, dw);
    double* g = dwt + (size_t)c * K;
    for (int k = 0; k < K; ++k) g[k] = 0.0;
    for (int n = 0; n < N; ++n) {
      const double* xp = x + ((size_t)n * C + c) * H * W;
      const double* gp = dy + ((size_t)n * C + c) * H * W;
      for (int p = 0; p < H; ++p) {
        for (int q = 0; q < W; ++q) {
          const double gy = gp[(size_t)p * W + q];
          for (int k = 0; k < K; ++k) {
            const int h = p + dh[k];
            const int w = q + dw[k];
            if (h >= 0 && h < H && w >= 0 && w < W) g[k] += gy * xp[(size_t)h * W + w];
          }
        }
      }
    }
    free(dh);
    free(dw);
  }
}

/* ------------------------------------------------------------------------
 * Extensions: stride and the bilinear-interpolation variant.
 *
 * Stride (Definition 1, Eq. 2): the output position (p, q) samples the input
 * at (str*p + dh_k, str*q + dw_k).  The paper does not give P and Q; the
 * reading taken here is the usual one for a centred odd kernel,
 * P = floor((H - 1) / str) + 1 and Q = floor((W - 1) / str) + 1, so that
 * output (p, q) is centred on input (str*p, str*q).
 *
 * Bilinear variant (section "Discretization and Interpolation", where the
 * paper weighs it against rounding down): tap k samples the input at the
 * unrounded position (str*p + rh_k, str*q + rw_k), (rh_k, rw_k) =
 * (-(k - pad) sin theta, (k - pad) cos theta), by bilinear interpolation of
 * the four surrounding pixels, each read as zero outside the plane:
 *   h0 = floor(rh), fh = rh - h0, w0 = floor(rw), fw = rw - w0,
 *   sample = (1-fh)(1-fw) x[h0][w0] + (1-fh) fw x[h0][w0+1]
 *          + fh (1-fw) x[h0+1][w0] + fh fw x[h0+1][w0+1].
 * The floor takes reading R2 (a product within 1e-9 of an integer is that
 * integer, with a zero fraction), which only matters at the 1e-16 level
 * here since the result is continuous in the fraction.
 *
 * Both are written as a list of (row offset, column offset, coefficient)
 * samples per tap: one sample with coefficient 1 for rounding down, four
 * for bilinear.  y sums w[c,k] * coefficient * x over every sample; the
 * backward passes are again the literal adjoints in scatter form.
 * ------------------------------------------------------------------------ */

/* Samples of the K taps: sh, sw, sc hold 4 entries per tap (unused entries
 * have coefficient 0).  mode 0 = round down (Eq. 2), 1 = bilinear. */
static void tap_samples(double theta_deg, int K, int mode, int* sh, int* sw, double* sc) {
  const int pad = K / 2;
  double* rh = (double*)malloc(sizeof(double) * (size_t)K);
  double* rw = (double*)malloc(sizeof(double) * (size_t)K);
  oracle_offsets_real(theta_deg, K, pad, rh, rw);
  for (int k = 0; k < K; ++k) {
    const double h0 = floor_snapped(rh[k]), w0 = floor_snapped(rw[k]);
    for (int s = 0; s < 4; ++s) {
      sh[4 * k + s] = (int)h0 + (s >> 1);
      sw[4 * k + s] = (int)w0 + (s & 1);
      sc[4 * k + s] = 0.0;
    }
    if (mode == 0) {
      sc[4 * k] = 1.0;
    } else {
      /* a snapped coordinate is exactly the integer h0: zero fraction */
      const double fh = (fabs(rh[k] - h0) <= ORACLE_SNAP_EPS) ? 0.0 : rh[k] - h0;
      const double fw = (fabs(rw[k] - w0) <= ORACLE_SNAP_EPS) ? 0.0 : rw[k] - w0;
      sc[4 * k + 0] = (1.0 - fh) * (1.0 - fw);
      sc[4 * k + 1] = (1.0 - fh) * fw;
      sc[4 * k + 2] = fh * (1.0 - fw);
      sc[4 * k + 3] = fh * fw;
    }
  }
  free(rh);
  free(rw);
}

/* Exposed for the tests: the sample list of one channel. */
void oracle_tap_samples(double theta_deg, int K, int mode, int* sh, int* sw, double* sc) {
  tap_samples(theta_deg, K, mode, sh, sw, sc);
}

int oracle_out_size(int n, int str) { return (n - 1) / str + 1; }

/* Forward pass with stride and discretisation mode; y is N x C x P x Q. */
void oracle_fwd_ex(const double* x, const double* wt, const double* theta_deg, double* y,
                   int N, int C, int H, int W, int K, int str, int mode, int nthreads) {
  const int P = oracle_out_size(H, str), Q = oracle_out_size(W, str);
  const long planes = (long)N * C;
#pragma omp parallel for schedule(dynamic) num_threads(nthreads)
  for (long nc = 0; nc < planes; ++nc) {
    const int c = (int)(nc % C);
    int* sh = (int*)malloc(sizeof(int) * 4 * (size_t)K);
    int* sw = (int*)malloc(sizeof(int) * 4 * (size_t)K);
    double* sc = (double*)malloc(sizeof(double) * 4 * (size_t)K);
    tap_samples(theta_deg[c], K, mode, sh, sw, sc);
    const double* xp = x + (size_t)nc * H * W;
    double* yp = y + (size_t)nc * P * Q;
    for (int p = 0; p < P; ++p) {
      for (int q = 0; q < Q; ++q) {
        double acc = 0.0;
        for (int k = 0; k < K; ++k) {
          for (int s = 0; s < 4; ++s) {
            if (sc[4 * k + s] == 0.0) continue;
            const int h = str * p + sh[4 * k + s];
            const int w = str * q + sw[4 * k + s];
            if (h >= 0 && h < H && w >= 0 && w < W)
              acc += xp[(size_t)h * W + w] * sc[4 * k + s] * wt[(size_t)c * K + k];
          }
        }
        yp[(size_t)p * Q + q] = acc;
      }
    }
    free(sh);
    free(sw);
    free(sc);
  }
}

/* Gradient with respect to the input (N x C x H x W) given dy (N x C x P x Q). */
void oracle_bwd_input_ex(const double* dy, const double* wt, const double* theta_deg, double* dx,
                         int N, int C, int H, int W, int K, int str, int mode, int nthreads) {
  const int P = oracle_out_size(H, str), Q = oracle_out_size(W, str);
  const long planes = (long)N * C;
#pragma omp parallel for schedule(dynamic) num_threads(nthreads)
  for (long nc = 0; nc < planes; ++nc) {
    const int c = (int)(nc % C);
    int* sh = (int*)malloc(sizeof(int) * 4 * (size_t)K);
    int* sw = (int*)malloc(sizeof(int) * 4 * (size_t)K);
    double* sc = (double*)malloc(sizeof(double) * 4 * (size_t)K);
    tap_samples(theta_deg[c], K, mode, sh, sw, sc);
    const double* gp = dy + (size_t)nc * P * Q;
    double* xp = dx + (size_t)nc * H * W;
    memset(xp, 0, sizeof(double) * (size_t)H * W);
    for (int p = 0; p < P; ++p) {
      for (int q = 0; q < Q; ++q) {
        const double g = gp[(size_t)p * Q + q];
        for (int k = 0; k < K; ++k) {
          for (int s = 0; s < 4; ++s) {
            if (sc[4 * k + s] == 0.0) continue;
            const int h = str * p + sh[4 * k + s];
            const int w = str * q + sw[4 * k + s];
            if (h >= 0 && h < H && w >= 0 && w < W)
              xp[(size_t)h * W + w] += g * sc[4 * k + s] * wt[(size_t)c * K + k];
          }
        }
      }
    }
    free(sh);
    free(sw);
    free(sc);
  }
}

/* Gradient with respect to the weights (C x K). */
void oracle_bwd_weight_ex(const double* x, const double* dy, const double* theta_deg, double* dwt,
                          int N, int C, int H, int W, int K, int str, int mode, int nthreads) {
  const int P = oracle_out_size(H, str), Q = oracle_out_size(W, str);
#pragma omp parallel for schedule(dynamic) num_threads(nthreads)
  for (int c = 0; c < C; ++c) {
    int* sh = (int*)malloc(sizeof(int) * 4 * (size_t)K);
    int* sw = (int*)malloc(sizeof(int) * 4 * (size_t)K);
    double* sc = (double*)malloc(sizeof(double) * 4 * (size_t)K);
    tap_samples(theta_deg[c], K, mode, sh, sw, sc);
    double* g = dwt + (size_t)c * K;
    for (int k = 0; k < K; ++k) g[k] = 0.0;
    for (int n = 0; n < N; ++n) {
      const double* xp = x + ((size_t)n * C + c) * H * W;
      const double* gp = dy + ((size_t)n * C + c) * P * Q;
      for (int p = 0; p < P; ++p) {
        for (int q = 0; q < Q; ++q) {
          const double gy = gp[(size_t)p * Q + q];
          for (int k = 0; k < K; ++k) {
            for (int s = 0; s < 4; ++s) {
              if (sc[4 * k + s] == 0.0) continue;
              const int h = str * p + sh[4 * k + s];
              const int w = str * q + sw[4 * k + s];
              if (h >= 0 && h < H && w >= 0 && w < W) g[k] += gy * sc[4 * k + s] * xp[(size_t)h * W + w];
            }
          }
        }
      }
    }
    free(sh);
    free(sw);
    free(sc);
  }
}
