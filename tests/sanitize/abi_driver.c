/* Host-side checks of the C ABI (include/qcnn.h) for a build of the library's
 * host code with AddressSanitizer and UndefinedBehaviorSanitizer
 * (tests/test_sanitize.py): argument validation of every entry point, the
 * status strings and helpers, and the conv planners over many layer shapes
 * (a layer too large for the allocation-free entry point's scratch is refused
 * after planning, before any HIP call).  Device pointers are fake: no call
 * here may reach a kernel.  The planner-only cases that get past validation
 * stop at the first HIP call, so they run only when no GPU is visible.
 * Prints "ok" when every call returned what it should. */
#include <stdint.h>
#include <stdio.h>

#include "qcnn.h"

int hipGetDeviceCount(int* count);  /* HIP runtime (C linkage) */

static int failures = 0;
#define EXPECT(cond)                                   \
  do {                                                 \
    if (!(cond)) {                                     \
      printf("FAILED line %d: %s\n", __LINE__, #cond); \
      ++failures;                                      \
    }                                                  \
  } while (0)

#define FP(a) ((const float*)(uintptr_t)(a))
#define FW(a) ((float*)(uintptr_t)(a))
#define CP(a) ((const uint8_t*)(uintptr_t)(a))
static const uintptr_t X = (uintptr_t)1 << 40, Dp = (uintptr_t)2 << 40, C = (uintptr_t)3 << 40,
                       Y = (uintptr_t)4 << 40, B = (uintptr_t)5 << 40;

static int conv(int N, int Cs, int H, int W, int M, int K, int Csp, int Ct, int dk, int s, int p, uintptr_t y,
                uintptr_t codes) {
  return qcnn_conv_forward(FP(X), N, Cs, H, W, FP(Dp), M, K, Csp, CP(codes), Ct, dk, s, p, NULL, 0, FW(y), NULL);
}

int main(void) {
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) != 0) ndev = 0;
  /* validation of the forwards */
  EXPECT(conv(2, 8, 5, 5, 2, 16, 4, 4, 3, 1, 1, 0, C) == QCNN_ERR_NULL);
  EXPECT(conv(0, 8, 5, 5, 2, 16, 4, 4, 3, 1, 1, Y, C) == QCNN_ERR_SHAPE);
  EXPECT(conv(2, 8, 5, 5, 3, 16, 4, 4, 3, 1, 1, Y, C) == QCNN_ERR_SHAPE);
  EXPECT(conv(2, 8, 5, 5, 2, 257, 4, 4, 3, 1, 1, Y, C) == QCNN_ERR_K_RANGE);
  EXPECT(conv(2, 8, 5, 5, 2, 16, 4, 4, 3, 1, 1, Y, C + 1) == QCNN_ERR_UNSUPPORTED);
  EXPECT(conv(2, 34, 5, 5, 2, 16, 17, 4, 3, 1, 1, Y, C) == QCNN_ERR_UNSUPPORTED);
  EXPECT(conv(2, 8, 5, 5, 2, 16, 4, 4, 3, 1, 1, X, C) == QCNN_ERR_ALIAS);
  EXPECT(conv(1, 8, 1, 1, 2, 16, 4, 4, 3, 1, 0, Y, C) == QCNN_ERR_SHAPE);
  EXPECT(conv(60000, 1 << 14, 1 << 12, 1 << 12, 1 << 12, 16, 4, 4, 3, 1, 0, Y, C) == QCNN_ERR_SHAPE);
  EXPECT(qcnn_fc_forward(FP(X), 2, 8, FP(Dp), 2, 16, 4, CP(C), 4, NULL, 0, NULL, NULL) == QCNN_ERR_NULL);
  EXPECT(qcnn_fc_forward(FP(X), 2, 8, FP(Dp), 3, 16, 4, CP(C), 4, NULL, 0, FW(Y), NULL) == QCNN_ERR_SHAPE);
  EXPECT(qcnn_fc_forward(FP(X), 2, 8, FP(Dp), 2, 300, 4, CP(C), 4, NULL, 0, FW(Y), NULL) == QCNN_ERR_K_RANGE);
  EXPECT(qcnn_fc_forward(FP(X), 2, 8, FP(Dp), 2, 16, 4, CP(C), 4, FP(Y + 4), 0, FW(Y), NULL) == QCNN_ERR_ALIAS);
  EXPECT(qcnn_lut_build(FP(X), 2, 8, 5, 5, FP(Dp), 2, 16, 4, NULL, NULL) == QCNN_ERR_NULL);
  EXPECT(qcnn_lut_build(FP(X), 2, 8, 5, 5, FP(Dp), 2, 16, 4, FW(X), NULL) == QCNN_ERR_ALIAS);
  EXPECT(qcnn_maxpool2d(FP(X), 1, 2, 5, 5, 3, 2, NULL, NULL) == QCNN_ERR_NULL);
  EXPECT(qcnn_maxpool2d(FP(X), 1, 2, 2, 2, 3, 2, FW(Y), NULL) == QCNN_ERR_SHAPE);
  EXPECT(qcnn_conv_forward_packed(FP(X), 2, 8, 5, 5, FP(Dp), 2, 0, 4, CP(C), 4, 3, 1, 1, NULL, 0, FW(Y), NULL) ==
         QCNN_ERR_K_RANGE);
  EXPECT(qcnn_fc_forward_packed(FP(X), 2, 8, FP(Dp), 2, 16, 4, NULL, 4, NULL, 0, FW(Y), NULL) == QCNN_ERR_NULL);
  EXPECT(qcnn_pack_codes(CP(C), 10, 0, (uint8_t*)Y, NULL) == QCNN_ERR_K_RANGE);
  EXPECT(qcnn_unpack_codes(NULL, 10, 16, (uint8_t*)Y, NULL) == QCNN_ERR_NULL);
  /* quantizer and error correction */
  EXPECT(qcnn_pq_assign(NULL, 4, 8, 3, FP(Dp), 2, 16, 4, (uint8_t*)C, NULL, NULL) == QCNN_ERR_NULL);
  EXPECT(qcnn_pq_assign(FP(X), 4, 8, 3, FP(Dp), 3, 16, 4, (uint8_t*)C, NULL, NULL) == QCNN_ERR_SHAPE);
  EXPECT(qcnn_pq_kmeans(FP(X), 4, 8, 3, 2, 16, 4, -1, FW(Dp), (uint8_t*)C, NULL, NULL) == QCNN_ERR_SHAPE);
  EXPECT(qcnn_pq_update(FP(X), 4, 8, 3, CP(C), 2, 300, 4, FW(Dp), NULL, NULL) == QCNN_ERR_K_RANGE);
  /* conv + max-pool: the conv's validation, then the pooling window */
  EXPECT(qcnn_conv_pool_forward(FP(X), 2, 8, 5, 5, FP(Dp), 2, 16, 4, CP(C), 4, 3, 1, 1, NULL, 0, 3, 2, NULL, NULL) ==
         QCNN_ERR_NULL);
  EXPECT(qcnn_conv_pool_forward(FP(X), 2, 8, 5, 5, FP(Dp), 2, 16, 4, CP(C), 4, 3, 1, 1, NULL, 0, 0, 2, FW(Y), NULL) ==
         QCNN_ERR_SHAPE);
  EXPECT(qcnn_conv_pool_forward(FP(X), 2, 8, 5, 5, FP(Dp), 2, 16, 4, CP(C), 4, 3, 1, 1, NULL, 0, 6, 1, FW(Y), NULL) ==
         QCNN_ERR_SHAPE);
  EXPECT(qcnn_conv_pool_forward(FP(X), 2, 8, 5, 5, FP(Dp), 3, 16, 4, CP(C), 4, 3, 1, 1, NULL, 0, 3, 2, FW(Y), NULL) ==
         QCNN_ERR_SHAPE);
  /* allocation-free conv: the same validation, then layers too large for its scratch */
  EXPECT(qcnn_conv_forward_noalloc(FP(X), 2, 8, 5, 5, FP(Dp), 2, 16, 4, CP(C), 4, 3, 1, 1, NULL, 0, NULL, NULL) ==
         QCNN_ERR_NULL);
  EXPECT(qcnn_conv_forward_noalloc(FP(X), 64, 256, 13, 13, FP(Dp), 64, 128, 4, CP(C), 384, 3, 1, 1, NULL, 0, FW(Y),
                                   NULL) == QCNN_ERR_WORKSPACE);
  EXPECT(qcnn_conv_forward_noalloc(FP(X), 64, 96, 27, 27, FP(Dp), 24, 128, 4, CP(C), 256, 5, 1, 2, NULL, 0, FW(Y),
                                   NULL) == QCNN_ERR_WORKSPACE);
  EXPECT(qcnn_conv_forward_noalloc(FP(X), 2, 4096, 13, 13, FP(Dp), 1024, 128, 4, CP(C), 4096, 3, 1, 1, NULL, 0,
                                   FW(Y), NULL) == QCNN_ERR_WORKSPACE);
  /* prepared layers: validation before any HIP call; *plan untouched on error */
  {
    qcnn_plan* plan = (qcnn_plan*)(uintptr_t)0xdead0;
    EXPECT(qcnn_conv_plan_create(2, 8, 5, 5, NULL, 2, 16, 4, CP(C), 0, 4, 3, 1, 1, NULL, 0, 0, 0, &plan, NULL) ==
           QCNN_ERR_NULL);
    EXPECT(qcnn_conv_plan_create(2, 8, 5, 5, FP(Dp), 2, 16, 4, CP(C), 0, 4, 3, 1, 1, NULL, 0, 0, 0, NULL, NULL) ==
           QCNN_ERR_NULL);
    EXPECT(qcnn_conv_plan_create(2, 8, 5, 5, FP(Dp), 3, 16, 4, CP(C), 0, 4, 3, 1, 1, NULL, 0, 0, 0, &plan, NULL) ==
           QCNN_ERR_SHAPE);
    EXPECT(qcnn_conv_plan_create(2, 8, 5, 5, FP(Dp), 2, 300, 4, CP(C), 1, 4, 3, 1, 1, NULL, 0, 0, 0, &plan, NULL) ==
           QCNN_ERR_K_RANGE);
    EXPECT(qcnn_conv_plan_create(2, 8, 5, 5, FP(Dp), 2, 16, 4, CP(C), 0, 4, 3, 1, 1, NULL, 0, 3, 0, &plan, NULL) ==
           QCNN_ERR_SHAPE);
    EXPECT(qcnn_conv_plan_create(2, 8, 5, 5, FP(Dp), 2, 16, 4, CP(C), 0, 4, 3, 1, 1, NULL, 0, 6, 1, &plan, NULL) ==
           QCNN_ERR_SHAPE);
    EXPECT(qcnn_conv_plan_create(2, 8, 5, 5, FP(Dp), 2, 16, 4, CP(C + 1), 0, 4, 3, 1, 1, NULL, 0, 0, 0, &plan,
                                 NULL) == QCNN_ERR_UNSUPPORTED);
    EXPECT(qcnn_fc_plan_create(2, 8, FP(Dp), 2, 16, 4, CP(C), 0, 4, NULL, 0, NULL, NULL) == QCNN_ERR_NULL);
    EXPECT(qcnn_fc_plan_create(2, 8, FP(Dp), 3, 16, 4, CP(C), 0, 4, NULL, 0, &plan, NULL) == QCNN_ERR_SHAPE);
    EXPECT(qcnn_fc_plan_create(2, 8, FP(Dp), 2, 0, 4, CP(C), 0, 4, NULL, 0, &plan, NULL) == QCNN_ERR_K_RANGE);
    EXPECT(qcnn_fc_plan_create(2, 8, FP(Dp), 2, 16, 4, CP(C + 1), 0, 4, NULL, 0, &plan, NULL) ==
           QCNN_ERR_UNSUPPORTED);
    EXPECT(plan == (qcnn_plan*)(uintptr_t)0xdead0);
    EXPECT(qcnn_plan_forward(NULL, FP(X), FW(Y), NULL) == QCNN_ERR_NULL);
    EXPECT(qcnn_plan_destroy(NULL) == QCNN_OK);
  }
  /* helpers */
  for (int s = 0; s <= 9; ++s) EXPECT(qcnn_status_string((qcnn_status)s) != NULL);
  EXPECT(qcnn_out_size(227, 11, 4, 0) == 55 && qcnn_out_size(2, 3, 1, 0) == 0);
  EXPECT(qcnn_code_bits(1) == 0 && qcnn_code_bits(256) == 8 && qcnn_code_bits(0) == -1);
  EXPECT(qcnn_packed_bytes(37, 16) == 20 && qcnn_packed_bytes(5, 0) == 0);
  EXPECT(qcnn_version() == 1);
  double ms = -1.0, each[4];
  long long n = -1;
  EXPECT(qcnn_timing_read(&ms, &n) == QCNN_OK && n == 0);
  EXPECT(qcnn_timing_read_each(each, 4, &n) == QCNN_OK && n == 0);
  double d;
  EXPECT(qcnn_probe_hbm(FP(X), FW(X + 512), 1024, &d, &d, &d, NULL) == QCNN_ERR_ALIAS);
  /* planners over many layer shapes: with no device the call stops at its
     first HIP call (after validation and planning) */
  if (ndev == 0) {
    static const int shapes[][10] = {
        /* N, Cs, H, W, Ct, dk, stride, pad, Csp, K */
        {32, 256, 13, 13, 384, 3, 1, 1, 4, 128}, {16, 256, 56, 56, 256, 3, 1, 1, 8, 128},
        {64, 3, 227, 227, 96, 11, 4, 0, 3, 64},  {64, 96, 27, 27, 256, 5, 1, 2, 4, 128},
        {1, 16, 14, 14, 32, 3, 1, 1, 4, 16},     {3, 12, 11, 9, 33, 3, 1, 1, 4, 32},
        {2, 24, 15, 15, 17, 5, 1, 2, 4, 128},    {1, 40, 9, 70, 5, 3, 1, 1, 8, 256},
        {2, 10, 8, 8, 7, 1, 1, 0, 5, 9},         {1, 32, 6, 6, 3, 3, 2, 3, 16, 8},
        {4, 2, 5, 5, 65, 2, 3, 1, 1, 2},         {1, 8, 1, 1, 4, 3, 1, 1, 4, 1},
        {2, 6, 30, 1, 3, 3, 2, 1, 2, 4},         {1, 64, 57, 57, 9, 3, 1, 1, 8, 128},
        {3, 12, 13, 13, 200, 3, 1, 1, 4, 9},     {2, 512, 6, 6, 16, 3, 1, 1, 2, 16},
        {1, 7, 3, 3, 5, 3, 1, 1, 1, 7},          {2, 16, 10, 90, 20, 3, 1, 1, 4, 128},
    };
    for (unsigned i = 0; i < sizeof(shapes) / sizeof(shapes[0]); ++i) {
      const int* q = shapes[i];
      const int st = conv(q[0], q[1], q[2], q[3], q[1] / q[8], q[9], q[8], q[4], q[5], q[6], q[7], Y, C);
      EXPECT(st == QCNN_ERR_HIP || st == QCNN_ERR_UNSUPPORTED);
    }
  }
  if (failures) return 1;
  printf("ok\n");
  return 0;
}
