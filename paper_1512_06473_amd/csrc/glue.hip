// Network glue that is not part of the paper's method, a debug check, and
// the packed code format.
//
// Max pooling joins the PQ layers of the AlexNet-shaped forward (k x k
// windows, stride s, no padding).  It moves 4 bytes per input element once
// and is bound by HBM; one thread computes one output.
//
// Packed codes: Table 1 (Sec. 3.4) stores every quantization index in
// log2 K bits.  pack_codes_kernel writes the stream of `bits` bits per code
// (code i at stream bits i bits .. i bits + bits - 1, least significant bit
// first), one thread per output dword: it ORs in the (at most 33 / bits + 1)
// codes whose bits fall in that dword.  unpack_codes_kernel writes one byte
// per code.  Both are bound by HBM (n bits / 8 bytes one way, n the other).
#include "qcnn_internal.h"

namespace qcnn {
namespace {

// One thread per output.  KW > 0: a KW x KW window, unrolled, so that all
// of a thread's loads are in flight together (with a run-time window size
// each load waited for the previous max: 36 us for AlexNet's pool1 at N = 64,
// 2.6 TB/s); KW = 0: any window size.
template <int KW>
__global__ __launch_bounds__(256) void maxpool_kernel(const float* __restrict__ x, int H, int W, int k, int s,
                                                      int Ho, int Wo, size_t total, float* __restrict__ y) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int xo = (int)(i % Wo);
  const int yo = (int)((i / Wo) % Ho);
  const size_t plane = i / ((size_t)Wo * Ho);
  const float* src = x + plane * H * W + (size_t)(yo * s) * W + xo * s;
  float best = src[0];
  if constexpr (KW > 0) {
    float v[KW * KW];
#pragma unroll
    for (int dy = 0; dy < KW; ++dy)
#pragma unroll
      for (int dx = 0; dx < KW; ++dx) v[dy * KW + dx] = src[dy * W + dx];
#pragma unroll
    for (int q = 0; q < KW * KW; ++q) best = fmaxf(best, v[q]);
  } else {
    for (int dy = 0; dy < k; ++dy)
      for (int dx = 0; dx < k; ++dx) best = fmaxf(best, src[dy * W + dx]);
  }
  y[i] = best;
}

__global__ void zero_int_kernel(int* __restrict__ v) { *v = 0; }

__global__ __launch_bounds__(256) void code_check_kernel(CodeStream codes, size_t n, int K,
                                                         int* __restrict__ bad) {
  int mine = 0;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    mine += code_at(codes, i) >= (uint32_t)K;
  if (mine) atomicAdd(bad, mine);
}

__global__ __launch_bounds__(256) void pack_codes_kernel(const uint8_t* __restrict__ codes, size_t n, int bits,
                                                         size_t nwords, uint32_t* __restrict__ packed) {
  const uint32_t mask = (1u << bits) - 1u;
  for (size_t w = (size_t)blockIdx.x * blockDim.x + threadIdx.x; w < nwords; w += (size_t)gridDim.x * blockDim.x) {
    const size_t b0 = w * 32;  // first stream bit of this dword
    uint32_t v = 0;
    for (size_t i = b0 / bits; i < n && i * bits < b0 + 32; ++i) {
      const long long off = (long long)(i * bits) - (long long)b0;  // in (-bits, 32)
      const uint32_t c = codes[i] & mask;
      v |= off >= 0 ? c << off : c >> (-off);
    }
    packed[w] = v;
  }
}

__global__ __launch_bounds__(256) void unpack_codes_kernel(CodeStream packed, size_t n,
                                                           uint8_t* __restrict__ codes) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    codes[i] = (uint8_t)code_at(packed, i);
}

}  // namespace

hipError_t launch_maxpool(const float* x, int N, int C, int H, int W, int k, int s, int Ho, int Wo, float* y,
                          hipStream_t stream) {
  const size_t total = (size_t)N * C * Ho * Wo;
  auto kern = k == 3 ? maxpool_kernel<3> : k == 2 ? maxpool_kernel<2> : maxpool_kernel<0>;
  hipLaunchKernelGGL(kern, dim3((unsigned)ceil_div_z(total, 256)), dim3(256), 0, stream, x, H, W, k, s, Ho, Wo,
                     total, y);
  return hipGetLastError();
}

hipError_t launch_pack_codes(const uint8_t* codes, size_t n, int bits, uint32_t* packed, hipStream_t stream) {
  const size_t nwords = ceil_div_z(n * (size_t)bits, 32);
  if (nwords == 0) return hipSuccess;
  const unsigned blocks = (unsigned)std::min<size_t>(4096, ceil_div_z(nwords, 256));
  hipLaunchKernelGGL(pack_codes_kernel, dim3(blocks), dim3(256), 0, stream, codes, n, bits, nwords, packed);
  return hipGetLastError();
}

hipError_t launch_unpack_codes(CodeStream packed, size_t n, uint8_t* codes, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  const unsigned blocks = (unsigned)std::min<size_t>(4096, ceil_div_z(n, 256));
  hipLaunchKernelGGL(unpack_codes_kernel, dim3(blocks), dim3(256), 0, stream, packed, n, codes);
  return hipGetLastError();
}

hipError_t launch_code_check(CodeStream codes, size_t n, int K, int* bad, hipStream_t stream) {
  const unsigned blocks = (unsigned)std::min<size_t>(1024, std::max<size_t>(1, ceil_div_z(n, 256)));
  hipLaunchKernelGGL(zero_int_kernel, dim3(1), dim3(1), 0, stream, bad);  // a kernel, not a memset node
  hipLaunchKernelGGL(code_check_kernel, dim3(blocks), dim3(256), 0, stream, codes, n, K, bad);
  return hipGetLastError();
}

}  // namespace qcnn
