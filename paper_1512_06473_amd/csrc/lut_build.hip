// Table of sub-codeword inner products, exported to device memory.
//
// Paper: Sec. 3.1, test phase (the paragraph after Eq. (5)): the input is
// split into M sub-vectors S^(m) and the inner products of S^(m) with every
// sub-codeword of D^(m) are stored in a look-up table; Sec. 3.2 (after
// Eq. (7)) pre-computes that table at every input position.  Table 1 counts
// its cost as d_s^2 C_s K multiply-adds.
//
//   lut[n][m][k][p] = sum_{j < C'_s} D[m][k][j] * x[n][m C'_s + j][p],  p in [0, H W)
//
// The kernel is bound by HBM writes: the table is K / C'_s times larger than
// the input it is built from.  A block is PX x KY threads: PX consecutive
// positions times KY codewords, so that for every k the stores of a wave are
// contiguous (PX >= 64) or, for tiny maps such as a fully-connected input
// (H = W = 1, PX = 1), contiguous along k.  Each thread loads its C'_s input
// values once and reuses them for all of its codewords; the block stages the
// subspace's K x C'_s sub-codewords in LDS first, so every codeword is read
// from HBM once per block and then served to the threads as LDS broadcasts.
#include "qcnn_internal.h"

namespace qcnn {
namespace {

template <int CSP>
__global__ __launch_bounds__(256) void lut_build_kernel(const float* __restrict__ x, const float* __restrict__ D,
                                                        float* __restrict__ lut, int Cs, int HW, int M, int K,
                                                        int csp_rt) {
  extern __shared__ float cb[];  // K x C'_s sub-codewords of subspace m
  const int csp = CSP > 0 ? CSP : csp_rt;
  const int m = blockIdx.y, n = blockIdx.z;
  const float* Dm = D + (size_t)m * K * csp;
  for (int i = threadIdx.y * blockDim.x + threadIdx.x; i < K * csp; i += blockDim.x * blockDim.y) cb[i] = Dm[i];
  __syncthreads();
  const int p = blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= HW) return;
  const float* xs = x + ((size_t)n * Cs + (size_t)m * csp) * HW + p;
  float* out = lut + ((size_t)n * M + m) * (size_t)K * HW + p;
  constexpr int XCAP = CSP > 0 ? CSP : 16;
  float xv[XCAP];
#pragma unroll
  for (int j = 0; j < XCAP; ++j) xv[j] = (j < csp) ? xs[(size_t)j * HW] : 0.f;
  for (int k = threadIdx.y; k < K; k += blockDim.y) {
    const float* d = cb + k * csp;
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < XCAP; ++j)
      if (j < csp) s = fmaf(d[j], xv[j], s);
    out[(size_t)k * HW] = s;
  }
}

}  // namespace

hipError_t launch_lut_build(const float* x, int N, int Cs, int H, int W, const float* D, int M, int K, int Csp,
                            float* lut, hipStream_t stream) {
  const int HW = H * W;
  int px = 256;
  while (px > 1 && px / 2 >= HW) px /= 2;  // smallest power of two >= HW, capped at 256
  const int ky = 256 / px;
  dim3 block(px, ky);
  dim3 grid(ceil_div(HW, px), M, N);
  const size_t lds = (size_t)K * Csp * sizeof(float);  // <= 256 x 16 x 4 = 16 KB
  LaunchTimer timer;
  switch (Csp) {
#define QCNN_LUT_CASE(C) \
  case C: return timed_launch(&timer, lut_build_kernel<C>, grid, block, (uint32_t)lds, stream, x, D, lut, Cs, HW, M, K, Csp);
    QCNN_LUT_CASE(1)
    QCNN_LUT_CASE(2)
    QCNN_LUT_CASE(3)
    QCNN_LUT_CASE(4)
    QCNN_LUT_CASE(6)
    QCNN_LUT_CASE(8)
#undef QCNN_LUT_CASE
    default:
      return timed_launch(&timer, lut_build_kernel<0>, grid, block, (uint32_t)lds, stream, x, D, lut, Cs, HW, M, K, Csp);
  }
}

}  // namespace qcnn
