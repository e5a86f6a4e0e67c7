/* Runs every function of the CPU oracle (oracle/qcnn_oracle.c) on small
 * shapes with exact-size heap buffers, for a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer (tests/test_sanitize.py): an out-of-bounds
 * access or undefined operation anywhere in the oracle aborts the run.
 * Prints "ok" when every call returned what it should. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int qo_lut(const float*, int, int, int, int, const float*, int, int, int, double*, double*);
int qo_conv_lut(const float*, int, int, int, int, const float*, int, int, int, const uint8_t*, int, int, int, int,
                const float*, int, double*, double*);
int qo_conv_direct(const float*, int, int, int, int, const float*, int, int, int, const uint8_t*, int, int, int, int,
                   const float*, int, double*);
int qo_conv_points(const float*, int, int, int, int, const float*, int, int, int, const uint8_t*, int, int, int, int,
                   const float*, int, const int32_t*, int, double*, double*);
int qo_fc_lut(const float*, int, int, const float*, int, int, int, const uint8_t*, int, const float*, int, double*,
              double*);
int qo_fc_direct(const float*, int, int, const float*, int, int, int, const uint8_t*, int, const float*, int, double*);
int qo_fc_points(const float*, int, int, const float*, int, int, int, const uint8_t*, int, const float*, int,
                 const int32_t*, int, double*, double*);
int qo_maxpool(const float*, int, int, int, int, int, int, double*);
int qo_pq_assign(const float*, int, int, int, const float*, int, int, int, uint8_t*, double*);
int qo_pq_distances(const float*, int, int, int, const float*, int, int, int, const uint8_t*, double*, double*);
int qo_pq_update(const float*, int, int, int, const uint8_t*, int, int, int, const float*, float*, int*);
int qo_pq_kmeans(const float*, int, int, int, int, int, int, int, float*, uint8_t*, double*);
int qo_code_bits(int);
int qo_pack_codes(const uint8_t*, long long, int, uint8_t*);
int qo_unpack_codes(const uint8_t*, long long, int, uint8_t*);

static int failures = 0;
#define EXPECT(cond)                                             \
  do {                                                           \
    if (!(cond)) {                                               \
      printf("FAILED line %d: %s\n", __LINE__, #cond);           \
      ++failures;                                                \
    }                                                            \
  } while (0)

static unsigned rng_state = 12345u;
static float frand(void) {
  rng_state = rng_state * 1664525u + 1013904223u;
  return (float)((rng_state >> 8) & 0xffff) / 65536.0f - 0.5f;
}
static float* fbuf(size_t n) {
  float* p = (float*)malloc((n ? n : 1) * sizeof(float));
  for (size_t i = 0; i < n; ++i) p[i] = frand();
  return p;
}
static uint8_t* cbuf(size_t n, int K) {
  uint8_t* p = (uint8_t*)malloc(n ? n : 1);
  for (size_t i = 0; i < n; ++i) {
    rng_state = rng_state * 1664525u + 1013904223u;
    p[i] = (uint8_t)((rng_state >> 16) % (unsigned)K);
  }
  return p;
}
static int outsz(int n, int k, int s, int p) { return n + 2 * p - k >= 0 ? (n + 2 * p - k) / s + 1 : 0; }

static void conv_case(int N, int Cs, int H, int W, int Ct, int dk, int s, int p, int Csp, int K) {
  const int M = Cs / Csp, Ho = outsz(H, dk, s, p), Wo = outsz(W, dk, s, p);
  float* x = fbuf((size_t)N * Cs * H * W);
  float* D = fbuf((size_t)M * K * Csp);
  float* b = fbuf((size_t)Ct);
  uint8_t* c = cbuf((size_t)Ct * dk * dk * M, K);
  double* y = (double*)malloc(sizeof(double) * N * Ct * Ho * Wo);
  double* a = (double*)malloc(sizeof(double) * N * Ct * Ho * Wo);
  double* lut = (double*)malloc(sizeof(double) * N * M * K * H * W);
  double* alut = (double*)malloc(sizeof(double) * N * M * K * H * W);
  EXPECT(qo_lut(x, N, Cs, H, W, D, M, K, Csp, lut, alut) == 0);
  EXPECT(qo_conv_lut(x, N, Cs, H, W, D, M, K, Csp, c, Ct, dk, s, p, b, 1, y, a) == 0);
  EXPECT(qo_conv_direct(x, N, Cs, H, W, D, M, K, Csp, c, Ct, dk, s, p, NULL, 0, y) == 0);
  int32_t pts[8] = {0, 0, 0, 0, N - 1, Ct - 1, Ho - 1, Wo - 1};
  double pv[2], pa[2];
  EXPECT(qo_conv_points(x, N, Cs, H, W, D, M, K, Csp, c, Ct, dk, s, p, b, 0, pts, 2, pv, pa) == 0);
  c[0] = (uint8_t)K;  /* a code out of range is refused */
  if (K < 256) EXPECT(qo_conv_lut(x, N, Cs, H, W, D, M, K, Csp, c, Ct, dk, s, p, NULL, 0, y, NULL) != 0);
  free(x); free(D); free(b); free(c); free(y); free(a); free(lut); free(alut);
}

static void fc_case(int N, int Cs, int Ct, int Csp, int K) {
  const int M = Cs / Csp;
  float* x = fbuf((size_t)N * Cs);
  float* D = fbuf((size_t)M * K * Csp);
  uint8_t* c = cbuf((size_t)Ct * M, K);
  double* y = (double*)malloc(sizeof(double) * N * Ct);
  double* a = (double*)malloc(sizeof(double) * N * Ct);
  EXPECT(qo_fc_lut(x, N, Cs, D, M, K, Csp, c, Ct, NULL, 1, y, a) == 0);
  EXPECT(qo_fc_direct(x, N, Cs, D, M, K, Csp, c, Ct, NULL, 0, y) == 0);
  int32_t pts[4] = {0, 0, N - 1, Ct - 1};
  double pv[2], pa[2];
  EXPECT(qo_fc_points(x, N, Cs, D, M, K, Csp, c, Ct, NULL, 0, pts, 2, pv, pa) == 0);
  free(x); free(D); free(c); free(y); free(a);
}

static void quant_case(int Ct, int Cs, int dk, int Csp, int K) {
  const int M = Cs / Csp;
  const size_t n = (size_t)Ct * dk * dk * M;
  float* W = fbuf((size_t)Ct * Cs * dk * dk);
  float* D = fbuf((size_t)M * K * Csp);
  float* D2 = (float*)malloc(sizeof(float) * M * K * Csp);
  uint8_t* c = (uint8_t*)malloc(n);
  double* obj = (double*)malloc(sizeof(double) * M);
  double* dc = (double*)malloc(sizeof(double) * n);
  double* dm = (double*)malloc(sizeof(double) * n);
  int* cnt = (int*)malloc(sizeof(int) * M * K);
  double* hist = (double*)malloc(sizeof(double) * 4);
  EXPECT(qo_pq_assign(W, Ct, Cs, dk, D, M, K, Csp, c, obj) == 0);
  EXPECT(qo_pq_distances(W, Ct, Cs, dk, D, M, K, Csp, c, dc, dm) == 0);
  EXPECT(qo_pq_update(W, Ct, Cs, dk, c, M, K, Csp, D, D2, cnt) == 0);
  EXPECT(qo_pq_kmeans(W, Ct, Cs, dk, M, K, Csp, 3, D, c, hist) == 0);
  free(W); free(D); free(D2); free(c); free(obj); free(dc); free(dm); free(cnt); free(hist);
}

static void pack_case(long long n, int K) {
  uint8_t* c = cbuf((size_t)n, K);
  const int b = qo_code_bits(K);
  const size_t bytes = (size_t)((n * b + 31) / 32 * 4);
  uint8_t* pk = (uint8_t*)malloc(bytes ? bytes : 1);
  uint8_t* back = (uint8_t*)malloc((size_t)(n ? n : 1));
  EXPECT(qo_pack_codes(c, n, K, pk) == 0);
  EXPECT(qo_unpack_codes(pk, n, K, back) == 0);
  for (long long i = 0; i < n; ++i) EXPECT(back[i] == c[i]);
  free(c); free(pk); free(back);
}

int main(void) {
  conv_case(2, 8, 7, 6, 5, 3, 1, 1, 4, 16);
  conv_case(1, 6, 9, 7, 3, 3, 2, 1, 3, 8);
  conv_case(1, 3, 15, 15, 2, 7, 4, 0, 3, 16);
  conv_case(1, 8, 6, 6, 3, 5, 1, 2, 4, 32);
  conv_case(2, 10, 8, 8, 7, 1, 1, 0, 5, 9);
  conv_case(1, 8, 1, 1, 4, 3, 1, 1, 4, 1);
  conv_case(1, 4, 5, 5, 2, 2, 3, 1, 1, 256);
  fc_case(3, 12, 7, 4, 8);
  fc_case(2, 9, 5, 3, 32);
  fc_case(1, 16, 3, 16, 256);
  float* xm = fbuf(2 * 3 * 7 * 9);
  double* ym = (double*)malloc(sizeof(double) * 2 * 3 * 3 * 4);
  EXPECT(qo_maxpool(xm, 2, 3, 7, 9, 3, 2, ym) == 0);
  free(xm); free(ym);
  quant_case(12, 24, 3, 4, 16);
  quant_case(16, 3, 11, 3, 64);
  quant_case(33, 6, 2, 1, 1);
  quant_case(40, 16, 1, 16, 7);
  for (int K = 1; K <= 256; K = K * 2 + 1) pack_case(37, K);
  pack_case(64, 256);
  pack_case(1, 2);
  EXPECT(qo_code_bits(0) < 0 && qo_code_bits(257) < 0);
  if (failures) return 1;
  printf("ok\n");
  return 0;
}
