/*
 * qcnn_oracle.c -- TEST INFRASTRUCTURE ONLY.  Not part of the product path.
 *
 * Only tests/, the smoke check (__graft_entry__.smoke) and the benchmark's
 * cpu_baseline leg may load or call this file.  It shares no code, header,
 * table or constant with the HIP library under paper_1512_06473_amd/csrc.
 *
 * A plain, slow, obviously correct CPU implementation of the test-phase
 * forward of a product-quantized (PQ) layer, from
 *   J. Wu, C. Leng, Y. Wang, Q. Hu, J. Cheng, "Quantized Convolutional Neural
 *   Networks for Mobile Devices", CVPR 2016 (arXiv 1512.06473).
 *
 * What it computes (paper notation):
 *   - Sec. 2, Eq. (3): an inner product split over M subspaces; each sub-vector
 *     of the weights is replaced by a sub-codeword c^(m)_{k_m}.
 *   - Sec. 3.1, Eq. (5) and the test-phase paragraph after it: for a
 *     fully-connected layer, the input S is split into M sub-vectors S^(m);
 *     the inner products of S^(m) with every sub-codeword of D^(m) go into a
 *     look-up table; each response T(c_t) is then the sum over m of the table
 *     entry selected by k_m(c_t).
 *   - Sec. 3.2, Eq. (7): for a convolutional layer the split is along input
 *     channels, one sub-codebook D^(m) is shared by all kernel offsets p_k,
 *     the table is pre-computed at every input position p_s, and T_{p_t}(c_t)
 *     sums the table entry selected by k_m(c_t, p_k) over the receptive-field
 *     pairs (p_k, p_s) and over m.
 *
 * Every floating-point sum is taken in double precision from the fp32 inputs.
 *
 * Readings of points the paper leaves open (each is stated where it is used):
 *   R1 layouts: x [N][C_s][H][W]; codebooks D [M][K][C'_s] (row k of D[m] is
 *      the sub-codeword D^(m)_k); conv codes [C_t][d_k][d_k][M] holding
 *      k_m(c_t, p_k) for p_k = (ky, kx); FC codes [C_t][M] holding k_m(c_t).
 *   R2 the (p_k, p_s) pairing of Eq. (1) is cross-correlation with stride s
 *      and zero padding p: p_s = p_t * s - p + p_k, no kernel flip.
 *   R3 positions in the zero padding hold S = 0, so <D_k, 0> = 0: they add
 *      nothing and are skipped.
 *   R4 subspace m covers input channels [m C'_s, (m+1) C'_s) (the "even split"
 *      of Sec. 3.1), so C_s = M C'_s.
 *   R5 optional per-output-channel bias and ReLU are applied after the sum;
 *      neither is part of Eq. (5) or Eq. (7), a NULL bias and relu = 0 give
 *      exactly those equations.
 *
 * Return value of every entry point: 0 on success, otherwise one of the
 * negative QO_E* codes below; on error nothing is written.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

#define QO_EARG   (-1) /* null pointer or non-positive size */
#define QO_ESHAPE (-2) /* C_s != M C'_s, or an empty output */
#define QO_EK     (-3) /* K outside [1, 256] */
#define QO_ECODE  (-4) /* a code >= K */
#define QO_ENOMEM (-5)

static int out_size(int in, int k, int s, int p) {
  int span = in + 2 * p - k;
  if (span < 0) return 0;
  return span / s + 1;
}

static int check_pq(int N, int Cs, int M, int K, int Csp) {
  if (N < 1 || Cs < 1 || M < 1 || Csp < 1) return QO_EARG;
  if (K < 1 || K > 256) return QO_EK;
  if (Cs != M * Csp) return QO_ESHAPE;
  return 0;
}

static int check_codes(const uint8_t* codes, size_t n, int K) {
  for (size_t i = 0; i < n; ++i)
    if ((int)codes[i] >= K) return QO_ECODE;
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Look-up table (Sec. 3.1 test phase; Sec. 3.2 last paragraph):
 *   lut[n][m][k][y][x] = < D^(m)_k , S^(m)_{(y,x)} >
 *                      = sum_{j < C'_s} D[m][k][j] * x[n][m C'_s + j][y][x]
 * over the real (unpadded) input positions only (R3).
 * absb, if non-NULL, receives sum_j |D[m][k][j] * x[...]| (the sum of the
 * absolute values of the terms, used for the rounding-error bound).        */
int qo_lut(const float* x, int N, int Cs, int H, int W,
           const float* D, int M, int K, int Csp,
           double* lut, double* absb) {
  int e;
  if (!x || !D || !lut) return QO_EARG;
  if ((e = check_pq(N, Cs, M, K, Csp))) return e;
  if (H < 1 || W < 1) return QO_EARG;
  const size_t HW = (size_t)H * W;
#pragma omp parallel for schedule(static)
  for (int n = 0; n < N; ++n)
    for (int m = 0; m < M; ++m)
      for (int k = 0; k < K; ++k)
        for (size_t p = 0; p < HW; ++p) {
          double s = 0.0, a = 0.0;
          for (int j = 0; j < Csp; ++j) {
            double term = (double)D[((size_t)m * K + k) * Csp + j] *
                          (double)x[((size_t)n * Cs + (size_t)m * Csp + j) * HW + p];
            s += term;
            a += fabs(term);
          }
          size_t o = (((size_t)n * M + m) * K + k) * HW + p;
          lut[o] = s;
          if (absb) absb[o] = a;
        }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Convolutional layer through the table, Eq. (7) third line:
 *   T_{p_t}(c_t) = sum_{(p_k, p_s)} sum_m lut[m][ k_m(c_t, p_k) ][p_s]
 * with p_t = (yo, xo), p_k = (ky, kx), p_s = (yo s - p + ky, xo s - p + kx)
 * (R2); pairs whose p_s falls in the padding contribute 0 and are skipped
 * (R3).  Then + bias[c_t] and ReLU if requested (R5).
 * y: [N][C_t][H_o][W_o].  absb (nullable): the bound sum over every product
 * |D * x| that enters the response, plus |bias|.                            */
int qo_conv_lut(const float* x, int N, int Cs, int H, int W,
                const float* D, int M, int K, int Csp,
                const uint8_t* codes, int Ct, int dk, int stride, int pad,
                const float* bias, int relu, double* y, double* absb) {
  int e;
  if (!x || !D || !codes || !y) return QO_EARG;
  if ((e = check_pq(N, Cs, M, K, Csp))) return e;
  if (H < 1 || W < 1 || Ct < 1 || dk < 1 || stride < 1 || pad < 0) return QO_EARG;
  const int Ho = out_size(H, dk, stride, pad), Wo = out_size(W, dk, stride, pad);
  if (Ho < 1 || Wo < 1) return QO_ESHAPE;
  if ((e = check_codes(codes, (size_t)Ct * dk * dk * M, K))) return e;
  const size_t HW = (size_t)H * W;
  const size_t per_img = (size_t)M * K * HW;
  int failed = 0;
#pragma omp parallel for schedule(dynamic, 1)
  for (int n = 0; n < N; ++n) {
    /* Table for one image: step 1. */
    double* lut = (double*)malloc(per_img * sizeof(double));
    double* alut = absb ? (double*)malloc(per_img * sizeof(double)) : NULL;
    if (!lut || (absb && !alut)) { free(lut); free(alut); failed = 1; continue; }
    qo_lut(x + (size_t)n * Cs * HW, 1, Cs, H, W, D, M, K, Csp, lut, alut);
    /* Step 2: sum of selected entries. */
    for (int t = 0; t < Ct; ++t)
      for (int yo = 0; yo < Ho; ++yo)
        for (int xo = 0; xo < Wo; ++xo) {
          double s = 0.0, a = 0.0;
          for (int ky = 0; ky < dk; ++ky) {
            int yi = yo * stride - pad + ky;
            if (yi < 0 || yi >= H) continue;
            for (int kx = 0; kx < dk; ++kx) {
              int xi = xo * stride - pad + kx;
              if (xi < 0 || xi >= W) continue;
              for (int m = 0; m < M; ++m) {
                int k = codes[(((size_t)t * dk + ky) * dk + kx) * M + m];
                size_t o = ((size_t)m * K + k) * HW + (size_t)yi * W + xi;
                s += lut[o];
                if (alut) a += alut[o];
              }
            }
          }
          if (bias) { s += (double)bias[t]; a += fabs((double)bias[t]); }
          if (relu && s < 0.0) s = 0.0;
          size_t oi = (((size_t)n * Ct + t) * Ho + yo) * Wo + xo;
          y[oi] = s;
          if (absb) absb[oi] = a;
        }
    free(lut);
    free(alut);
  }
  return failed ? QO_ENOMEM : 0;
}

/* ------------------------------------------------------------------------ */
/* Independent route for the same layer, Eq. (7) second line read with
 * D^(m) B^(m)_{c_t,p_k} = D^(m)_{k_m(c_t,p_k)}: rebuild the dense kernel
 *   What[c_t][m C'_s + j][ky][kx] = D[m][ k_m(c_t,(ky,kx)) ][j]
 * and evaluate Eq. (1), the plain receptive-field sum of <W_{c_t,p_k}, S_{p_s}>,
 * with no table.  Shares nothing with qo_conv_lut but the layouts.          */
int qo_conv_direct(const float* x, int N, int Cs, int H, int W,
                   const float* D, int M, int K, int Csp,
                   const uint8_t* codes, int Ct, int dk, int stride, int pad,
                   const float* bias, int relu, double* y) {
  int e;
  if (!x || !D || !codes || !y) return QO_EARG;
  if ((e = check_pq(N, Cs, M, K, Csp))) return e;
  if (H < 1 || W < 1 || Ct < 1 || dk < 1 || stride < 1 || pad < 0) return QO_EARG;
  const int Ho = out_size(H, dk, stride, pad), Wo = out_size(W, dk, stride, pad);
  if (Ho < 1 || Wo < 1) return QO_ESHAPE;
  if ((e = check_codes(codes, (size_t)Ct * dk * dk * M, K))) return e;
  const size_t wsz = (size_t)Ct * Cs * dk * dk;
  double* What = (double*)malloc(wsz * sizeof(double));
  if (!What) return QO_ENOMEM;
  for (int t = 0; t < Ct; ++t)
    for (int ky = 0; ky < dk; ++ky)
      for (int kx = 0; kx < dk; ++kx)
        for (int m = 0; m < M; ++m) {
          int k = codes[(((size_t)t * dk + ky) * dk + kx) * M + m];
          for (int j = 0; j < Csp; ++j)
            What[(((size_t)t * Cs + (size_t)m * Csp + j) * dk + ky) * dk + kx] =
                (double)D[((size_t)m * K + k) * Csp + j];
        }
  const size_t HW = (size_t)H * W;
#pragma omp parallel for schedule(static)
  for (int n = 0; n < N; ++n)
    for (int t = 0; t < Ct; ++t)
      for (int yo = 0; yo < Ho; ++yo)
        for (int xo = 0; xo < Wo; ++xo) {
          double s = 0.0;
          for (int c = 0; c < Cs; ++c)
            for (int ky = 0; ky < dk; ++ky) {
              int yi = yo * stride - pad + ky;
              if (yi < 0 || yi >= H) continue;
              for (int kx = 0; kx < dk; ++kx) {
                int xi = xo * stride - pad + kx;
                if (xi < 0 || xi >= W) continue;
                s += What[(((size_t)t * Cs + c) * dk + ky) * dk + kx] *
                     (double)x[((size_t)n * Cs + c) * HW + (size_t)yi * W + xi];
              }
            }
          if (bias) s += (double)bias[t];
          if (relu && s < 0.0) s = 0.0;
          y[(((size_t)n * Ct + t) * Ho + yo) * Wo + xo] = s;
        }
  free(What);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Single responses of the conv layer, for spot checks at sizes where a whole
 * table would be too slow: pts is [P][4] = (n, c_t, yo, xo).  Each response
 * is Eq. (7) with every table entry it selects evaluated from its definition
 * (the C'_s-term inner product) on the spot.                                */
int qo_conv_points(const float* x, int N, int Cs, int H, int W,
                   const float* D, int M, int K, int Csp,
                   const uint8_t* codes, int Ct, int dk, int stride, int pad,
                   const float* bias, int relu,
                   const int32_t* pts, int P, double* y, double* absb) {
  int e;
  if (!x || !D || !codes || !pts || !y || P < 0) return QO_EARG;
  if ((e = check_pq(N, Cs, M, K, Csp))) return e;
  if (H < 1 || W < 1 || Ct < 1 || dk < 1 || stride < 1 || pad < 0) return QO_EARG;
  const int Ho = out_size(H, dk, stride, pad), Wo = out_size(W, dk, stride, pad);
  if (Ho < 1 || Wo < 1) return QO_ESHAPE;
  for (int i = 0; i < P; ++i) {
    const int32_t* q = pts + 4 * (size_t)i;
    if (q[0] < 0 || q[0] >= N || q[1] < 0 || q[1] >= Ct || q[2] < 0 || q[2] >= Ho ||
        q[3] < 0 || q[3] >= Wo) return QO_EARG;
  }
  const size_t HW = (size_t)H * W;
#pragma omp parallel for schedule(dynamic, 4)
  for (int i = 0; i < P; ++i) {
    const int n = pts[4 * (size_t)i], t = pts[4 * (size_t)i + 1];
    const int yo = pts[4 * (size_t)i + 2], xo = pts[4 * (size_t)i + 3];
    double s = 0.0, a = 0.0;
    for (int ky = 0; ky < dk; ++ky) {
      int yi = yo * stride - pad + ky;
      if (yi < 0 || yi >= H) continue;
      for (int kx = 0; kx < dk; ++kx) {
        int xi = xo * stride - pad + kx;
        if (xi < 0 || xi >= W) continue;
        for (int m = 0; m < M; ++m) {
          int k = codes[(((size_t)t * dk + ky) * dk + kx) * M + m];
          for (int j = 0; j < Csp; ++j) {
            double term = (double)D[((size_t)m * K + k) * Csp + j] *
                          (double)x[((size_t)n * Cs + (size_t)m * Csp + j) * HW +
                                    (size_t)yi * W + xi];
            s += term;
            a += fabs(term);
          }
        }
      }
    }
    if (bias) { s += (double)bias[t]; a += fabs((double)bias[t]); }
    if (relu && s < 0.0) s = 0.0;
    y[i] = s;
    if (absb) absb[i] = a;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Fully-connected layer through the table, Eq. (5) last line and the
 * test-phase paragraph of Sec. 3.1:
 *   lut[m][k] = < D^(m)_k , S^(m) > = sum_j D[m][k][j] * x[n][m C'_s + j]
 *   T(c_t)    = sum_m lut[m][ k_m(c_t) ]
 * x: [N][C_s], codes: [C_t][M], y: [N][C_t].  absb as for the conv layer.  */
int qo_fc_lut(const float* x, int N, int Cs,
              const float* D, int M, int K, int Csp,
              const uint8_t* codes, int Ct,
              const float* bias, int relu, double* y, double* absb) {
  int e;
  if (!x || !D || !codes || !y) return QO_EARG;
  if ((e = check_pq(N, Cs, M, K, Csp))) return e;
  if (Ct < 1) return QO_EARG;
  if ((e = check_codes(codes, (size_t)Ct * M, K))) return e;
  int failed = 0;
#pragma omp parallel for schedule(dynamic, 1)
  for (int n = 0; n < N; ++n) {
    double* lut = (double*)malloc((size_t)M * K * sizeof(double));
    double* alut = (double*)malloc((size_t)M * K * sizeof(double));
    if (!lut || !alut) { free(lut); free(alut); failed = 1; continue; }
    for (int m = 0; m < M; ++m)
      for (int k = 0; k < K; ++k) {
        double s = 0.0, a = 0.0;
        for (int j = 0; j < Csp; ++j) {
          double term = (double)D[((size_t)m * K + k) * Csp + j] *
                        (double)x[(size_t)n * Cs + (size_t)m * Csp + j];
          s += term;
          a += fabs(term);
        }
        lut[(size_t)m * K + k] = s;
        alut[(size_t)m * K + k] = a;
      }
    for (int t = 0; t < Ct; ++t) {
      double s = 0.0, a = 0.0;
      for (int m = 0; m < M; ++m) {
        int k = codes[(size_t)t * M + m];
        s += lut[(size_t)m * K + k];
        a += alut[(size_t)m * K + k];
      }
      if (bias) { s += (double)bias[t]; a += fabs((double)bias[t]); }
      if (relu && s < 0.0) s = 0.0;
      y[(size_t)n * Ct + t] = s;
      if (absb) absb[(size_t)n * Ct + t] = a;
    }
    free(lut);
    free(alut);
  }
  return failed ? QO_ENOMEM : 0;
}

/* Independent route, Eq. (5) first line with W^(m)_{c_t} replaced by its
 * sub-codeword (Eq. (4): D^(m) B^(m)): What[c_t][m C'_s + j] =
 * D[m][k_m(c_t)][j], then Eq. (2), T(c_t) = <What_{c_t}, S>.               */
int qo_fc_direct(const float* x, int N, int Cs,
                 const float* D, int M, int K, int Csp,
                 const uint8_t* codes, int Ct,
                 const float* bias, int relu, double* y) {
  int e;
  if (!x || !D || !codes || !y) return QO_EARG;
  if ((e = check_pq(N, Cs, M, K, Csp))) return e;
  if (Ct < 1) return QO_EARG;
  if ((e = check_codes(codes, (size_t)Ct * M, K))) return e;
  double* What = (double*)malloc((size_t)Ct * Cs * sizeof(double));
  if (!What) return QO_ENOMEM;
  for (int t = 0; t < Ct; ++t)
    for (int m = 0; m < M; ++m) {
      int k = codes[(size_t)t * M + m];
      for (int j = 0; j < Csp; ++j)
        What[(size_t)t * Cs + (size_t)m * Csp + j] = (double)D[((size_t)m * K + k) * Csp + j];
    }
#pragma omp parallel for schedule(static)
  for (int n = 0; n < N; ++n)
    for (int t = 0; t < Ct; ++t) {
      double s = 0.0;
      for (int c = 0; c < Cs; ++c) s += What[(size_t)t * Cs + c] * (double)x[(size_t)n * Cs + c];
      if (bias) s += (double)bias[t];
      if (relu && s < 0.0) s = 0.0;
      y[(size_t)n * Ct + t] = s;
    }
  free(What);
  return 0;
}

/* Single FC responses: pts is [P][2] = (n, c_t); each is Eq. (5) with the
 * selected entries evaluated from their definition on the spot.            */
int qo_fc_points(const float* x, int N, int Cs,
                 const float* D, int M, int K, int Csp,
                 const uint8_t* codes, int Ct,
                 const float* bias, int relu,
                 const int32_t* pts, int P, double* y, double* absb) {
  int e;
  if (!x || !D || !codes || !pts || !y || P < 0) return QO_EARG;
  if ((e = check_pq(N, Cs, M, K, Csp))) return e;
  if (Ct < 1) return QO_EARG;
  for (int i = 0; i < P; ++i)
    if (pts[2 * (size_t)i] < 0 || pts[2 * (size_t)i] >= N || pts[2 * (size_t)i + 1] < 0 ||
        pts[2 * (size_t)i + 1] >= Ct) return QO_EARG;
#pragma omp parallel for schedule(dynamic, 4)
  for (int i = 0; i < P; ++i) {
    const int n = pts[2 * (size_t)i], t = pts[2 * (size_t)i + 1];
    double s = 0.0, a = 0.0;
    for (int m = 0; m < M; ++m) {
      int k = codes[(size_t)t * M + m];
      for (int j = 0; j < Csp; ++j) {
        double term = (double)D[((size_t)m * K + k) * Csp + j] *
                      (double)x[(size_t)n * Cs + (size_t)m * Csp + j];
        s += term;
        a += fabs(term);
      }
    }
    if (bias) { s += (double)bias[t]; a += fabs((double)bias[t]); }
    if (relu && s < 0.0) s = 0.0;
    y[i] = s;
    if (absb) absb[i] = a;
  }
  return 0;
}

/* ------------------------------------------------------------------------ */
/* Network glue, not part of the paper's method: max pooling over k x k
 * windows with stride s and no padding (out = floor((in - k) / s) + 1).
 * x: [N][C][H][W] fp32, y: [N][C][Ho][Wo] (the max is exact).              */
int qo_maxpool(const float* x, int N, int C, int H, int W, int k, int s, double* y) {
  if (!x || !y || N < 1 || C < 1 || H < 1 || W < 1 || k < 1 || s < 1) return QO_EARG;
  const int Ho = out_size(H, k, s, 0), Wo = out_size(W, k, s, 0);
  if (Ho < 1 || Wo < 1) return QO_ESHAPE;
  for (int n = 0; n < N; ++n)
    for (int c = 0; c < C; ++c)
      for (int yo = 0; yo < Ho; ++yo)
        for (int xo = 0; xo < Wo; ++xo) {
          double best = -INFINITY;
          for (int dy = 0; dy < k; ++dy)
            for (int dx = 0; dx < k; ++dx) {
              double v = x[(((size_t)n * C + c) * H + yo * s + dy) * W + xo * s + dx];
              if (v > best) best = v;
            }
          y[(((size_t)n * C + c) * Ho + yo) * Wo + xo] = best;
        }
  return 0;
}

/* Threads the OpenMP runtime will use (1 when built without OpenMP). */
/* ------------------------------------------------------------------------ */
/* Parameter quantization: how the sub-codebooks and codes are learned.
 * Sec. 3.1, Eq. (4): for subspace m, minimise || D^(m) B^(m) - W^(m) ||_F^2
 * over D^(m) (K sub-codewords of C'_s entries) and B^(m) (one indicator
 * column per sub-vector); the paper solves it by k-means over the sub-vectors.
 * Sec. 3.2, Eq. (6): a conv layer shares D^(m) over every kernel position
 * p_k, so subspace m's k-means runs over the sub-vectors of all (c_t, p_k)
 * and its objective is the sum over p_k of Eq. (4)'s.
 *
 * Weights W: [C_t][C_s][d_k][d_k] (a fully-connected layer is d_k = 1, i.e.
 * W[c_t][c_s], the transpose of the paper's C_s x C_t matrix); the sub-vector
 * of (c_t, p_k = (ky, kx), m) is ( W[c_t][m C'_s + j][ky][kx] )_{j < C'_s}.
 * Codes [C_t][d_k][d_k][M] and codebooks [M][K][C'_s] as in the forward.
 *
 * Readings of what the paper leaves open (it names k-means only):
 *   Q1 the distance is the squared Euclidean one (the Frobenius objective
 *      taken column by column).
 *   Q2 assignment: the nearest sub-codeword of Eq. (4) / (6), distances
 *      taken in double from the fp32 values, ties going to the lowest index.
 *   Q3 update: a sub-codeword becomes the mean of the sub-vectors assigned to
 *      it, summed in double in sub-vector order (c_t, ky, kx) and rounded to
 *      fp32; a sub-codeword that no sub-vector chose keeps its value.
 *   Q4 the initial sub-codewords are an input (the caller draws them).
 *   Q5 an iteration is an assignment followed by an update; after the last
 *      one a final assignment makes the codes match the final sub-codewords.
 * The objective of an assignment is || D B - W ||^2 for the chosen codes, in
 * double (per subspace).                                                     */

/* Squared distance, in double, between sub-vector (t, p, m) of W and the
 * sub-codeword c (C'_s entries).                                            */
static double pq_dist(const float* W, int Cs, int dk, int t, int p, int m, int Csp, const float* c) {
  double d = 0.0;
  for (int j = 0; j < Csp; ++j) {
    double diff = (double)W[(((size_t)t * Cs + (size_t)m * Csp + j) * dk * dk) + p] - (double)c[j];
    d += diff * diff;
  }
  return d;
}

static int check_quant(int Ct, int Cs, int dk, int M, int K, int Csp) {
  if (Ct < 1 || Cs < 1 || dk < 1 || M < 1 || Csp < 1) return QO_EARG;
  if (K < 1 || K > 256) return QO_EK;
  if (Cs != M * Csp) return QO_ESHAPE;
  return 0;
}

/* Assignment step (Q1, Q2).  codes: [C_t][d_k][d_k][M]; obj: [M] or NULL. */
int qo_pq_assign(const float* W, int Ct, int Cs, int dk, const float* D, int M, int K, int Csp,
                 uint8_t* codes, double* obj) {
  int e;
  if (!W || !D || !codes) return QO_EARG;
  if ((e = check_quant(Ct, Cs, dk, M, K, Csp))) return e;
  const int P = dk * dk;
#pragma omp parallel for schedule(dynamic, 1)
  for (int m = 0; m < M; ++m) {
    const float* Dm = D + (size_t)m * K * Csp;
    double s = 0.0;
    for (int t = 0; t < Ct; ++t)
      for (int p = 0; p < P; ++p) {
        int best = 0;
        double bd = pq_dist(W, Cs, dk, t, p, m, Csp, Dm);
        for (int k = 1; k < K; ++k) {
          double d = pq_dist(W, Cs, dk, t, p, m, Csp, Dm + (size_t)k * Csp);
          if (d < bd) { bd = d; best = k; }
        }
        codes[((size_t)t * P + p) * M + m] = (uint8_t)best;
        s += bd;
      }
    if (obj) obj[m] = s;
  }
  return 0;
}

/* For checking an assignment made elsewhere: per sub-vector (in the codes'
 * order [C_t][d_k][d_k][M]), the double distance to the sub-codeword its
 * code names (dcode) and the smallest double distance over all K (dmin).   */
int qo_pq_distances(const float* W, int Ct, int Cs, int dk, const float* D, int M, int K, int Csp,
                    const uint8_t* codes, double* dcode, double* dmin) {
  int e;
  if (!W || !D || !codes || !dcode || !dmin) return QO_EARG;
  if ((e = check_quant(Ct, Cs, dk, M, K, Csp))) return e;
  if ((e = check_codes(codes, (size_t)Ct * dk * dk * M, K))) return e;
  const int P = dk * dk;
#pragma omp parallel for schedule(dynamic, 1)
  for (int m = 0; m < M; ++m) {
    const float* Dm = D + (size_t)m * K * Csp;
    for (int t = 0; t < Ct; ++t)
      for (int p = 0; p < P; ++p) {
        const size_t i = ((size_t)t * P + p) * M + m;
        double bd = pq_dist(W, Cs, dk, t, p, m, Csp, Dm);
        for (int k = 1; k < K; ++k) {
          double d = pq_dist(W, Cs, dk, t, p, m, Csp, Dm + (size_t)k * Csp);
          if (d < bd) bd = d;
        }
        dmin[i] = bd;
        dcode[i] = pq_dist(W, Cs, dk, t, p, m, Csp, Dm + (size_t)codes[i] * Csp);
      }
  }
  return 0;
}

/* Update step.  D_in, D_out: [M][K][C'_s] (may be the same array);
 * counts: [M][K] sub-vectors per sub-codeword, or NULL.                     */
int qo_pq_update(const float* W, int Ct, int Cs, int dk, const uint8_t* codes, int M, int K, int Csp,
                 const float* D_in, float* D_out, int* counts) {
  int e;
  if (!W || !codes || !D_in || !D_out) return QO_EARG;
  if ((e = check_quant(Ct, Cs, dk, M, K, Csp))) return e;
  if ((e = check_codes(codes, (size_t)Ct * dk * dk * M, K))) return e;
  const int P = dk * dk;
  int failed = 0;
#pragma omp parallel for schedule(dynamic, 1)
  for (int m = 0; m < M; ++m) {
    double* sum = (double*)calloc((size_t)K * Csp, sizeof(double));
    int* cnt = (int*)calloc((size_t)K, sizeof(int));
    if (!sum || !cnt) { free(sum); free(cnt); failed = 1; continue; }
    for (int t = 0; t < Ct; ++t)
      for (int p = 0; p < P; ++p) {
        int k = codes[((size_t)t * P + p) * M + m];
        cnt[k] += 1;
        for (int j = 0; j < Csp; ++j)
          sum[(size_t)k * Csp + j] += (double)W[(((size_t)t * Cs + (size_t)m * Csp + j) * P) + p];
      }
    for (int k = 0; k < K; ++k) {
      for (int j = 0; j < Csp; ++j) {
        size_t o = ((size_t)m * K + k) * Csp + j;
        D_out[o] = cnt[k] ? (float)(sum[(size_t)k * Csp + j] / (double)cnt[k]) : D_in[o];
      }
      if (counts) counts[(size_t)m * K + k] = cnt[k];
    }
    free(sum);
    free(cnt);
  }
  return failed ? QO_ENOMEM : 0;
}

/* k-means (Q5): iters x (assign, update), then a final assignment.
 * D: [M][K][C'_s] in: initial sub-codewords, out: learned ones.
 * obj: [iters + 1] totals over m of each assignment's objective.           */
int qo_pq_kmeans(const float* W, int Ct, int Cs, int dk, int M, int K, int Csp, int iters,
                 float* D, uint8_t* codes, double* obj) {
  int e;
  if (!W || !D || !codes || iters < 0) return QO_EARG;
  if ((e = check_quant(Ct, Cs, dk, M, K, Csp))) return e;
  double* om = (double*)malloc((size_t)M * sizeof(double));
  if (!om) return QO_ENOMEM;
  for (int it = 0; it <= iters && !e; ++it) {
    e = qo_pq_assign(W, Ct, Cs, dk, D, M, K, Csp, codes, om);
    if (e) break;
    double a = 0.0;
    for (int m = 0; m < M; ++m) a += om[m];
    if (obj) obj[it] = a;
    if (it < iters) e = qo_pq_update(W, Ct, Cs, dk, codes, M, K, Csp, D, D, NULL);
  }
  free(om);
  return e;
}

/* ---------------------------------------------------------- packed codes
 * Table 1 (Sec. 3.4) stores every quantization index in log2 K bits: the
 * code bytes of a layer are (1/8) d_k^2 M C_t log2 K (conv) or
 * (1/8) M C_t log2 K (FC).  The stream format is a reading (the paper fixes
 * only the width):
 *   R6b  b = the number of bits that hold 0 .. K-1 (b = 0 for K = 1, else the
 *        smallest b with 2^b >= K, i.e. log2 K for a power of two); code i of
 *        the array, in the array's own order, is bits i b .. i b + b - 1 of
 *        the stream, value bit j at stream bit i b + j; stream bit q is bit
 *        q % 8 of byte q / 8.  The stream is ceil(n b / 8) bytes.
 * Both functions go bit by bit, straight from that definition.
 */
int qo_code_bits(int K) {
  if (K < 1 || K > 256) return QO_EK;
  int b = 0;
  while ((1 << b) < K) ++b;
  return b;
}

int qo_pack_codes(const uint8_t* codes, long long n, int K, uint8_t* out) {
  const int b = qo_code_bits(K);
  if (b < 0) return b;
  if (n < 0 || (n > 0 && !codes) || (n * b > 0 && !out)) return QO_EARG;
  int e = check_codes(codes, (size_t)n, K);
  if (e) return e;
  const long long nbytes = (n * b + 7) / 8;
  for (long long q = 0; q < nbytes; ++q) out[q] = 0;
  for (long long i = 0; i < n; ++i)
    for (int j = 0; j < b; ++j) {
      const long long q = i * b + j;  /* stream bit of value bit j of code i */
      out[q / 8] |= (uint8_t)(((codes[i] >> j) & 1) << (q % 8));
    }
  return 0;
}

int qo_unpack_codes(const uint8_t* in, long long n, int K, uint8_t* codes) {
  const int b = qo_code_bits(K);
  if (b < 0) return b;
  if (n < 0 || (n > 0 && !codes) || (n * b > 0 && !in)) return QO_EARG;
  for (long long i = 0; i < n; ++i) {
    int v = 0;
    for (int j = 0; j < b; ++j) {
      const long long q = i * b + j;
      v |= ((in[q / 8] >> (q % 8)) & 1) << j;
    }
    codes[i] = (uint8_t)v;
  }
  return 0;
}

/* Thread count of the parallel loops (timing of the oracle only). */
#ifdef _OPENMP
#include <omp.h>
int qo_threads(void) { return omp_get_max_threads(); }
void qo_set_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }
#else
int qo_threads(void) { return 1; }
void qo_set_threads(int n) { (void)n; }
#endif
