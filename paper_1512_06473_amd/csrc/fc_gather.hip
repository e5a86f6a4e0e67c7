// PQ fully-connected layer: per-image table in LDS, gather over the codes.
//
// Paper: Sec. 3.1, Eq. (5) and the test-phase paragraph after it:
//     T(c_t) = sum_m < D^(m)_{k_m(c_t)}, S^(m) > = sum_m L[m][ k_m(c_t) ],
// with L[m][k] = < D^(m)_k, S^(m) > computed once per input.  Table 1: C_s K
// multiply-adds for the table plus C_t M additions for the responses.
//
// MI355X mapping:
//   * lanes own images (64 per wave), so a code k_m(c_t) -- which does not
//     depend on the image -- is wave-uniform: one scalar load, and the 64
//     lanes read 64 consecutive table entries [m][k][lane] (conflict-free);
//   * a workgroup (8 waves) owns 64 images, a block of 8 TW output channels
//     and a range of subspaces; it walks that range in chunks, each wave
//     building the table of one subspace in LDS, then all waves gather;
//   * the subspace range is split over `splits` workgroups so that the chip
//     fills; their partial sums land in a stream-ordered scratch buffer and a
//     second kernel adds them in a fixed order (deterministic), then applies
//     bias and ReLU.  With one split the first kernel writes y directly.
#include "qcnn_internal.h"

namespace qcnn {
namespace {

constexpr int kThreads = 512;
constexpr int kWaves = kThreads / kWave;
constexpr int kTW = 32;  // output channels per wave
constexpr size_t kLdsBudget = 64 * 1024;

struct FcParams {
  int N, Cs, M, K, Csp, Ct;
  int m_per_split, mchunk;
  int relu;
};

// partial: [splits][N][Ct], or null when the kernel writes y itself.
template <int CSP>
__global__ __launch_bounds__(kThreads) void fc_pq_kernel(const float* __restrict__ x, const float* __restrict__ D,
                                                         CodeStream codes, const float* __restrict__ bias,
                                                         float* __restrict__ y, float* __restrict__ partial,
                                                         FcParams p) {
  extern __shared__ float lut[];  // [mchunk][K][64]
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int n = blockIdx.y * kWave + lane;
  const bool nvalid = n < p.N;
  const int split = blockIdx.z;
  const int m0 = split * p.m_per_split;
  const int m1 = min(p.M, m0 + p.m_per_split);
  const int tbase = blockIdx.x * (kWaves * kTW) + wave * kTW;
  const int csp = CSP > 0 ? CSP : p.Csp;
  constexpr int XCAP = CSP > 0 ? CSP : 16;
  const uint32_t kmax = (uint32_t)(p.K - 1);

  float acc[kTW];
#pragma unroll
  for (int i = 0; i < kTW; ++i) acc[i] = 0.f;

  for (int mc = m0; mc < m1; mc += p.mchunk) {
    const int cnt = min(p.mchunk, m1 - mc);
    __syncthreads();
    // ---- table of subspaces mc .. mc+cnt-1 for this workgroup's images
    for (int w = wave; w < cnt; w += kWaves) {
      const int m = mc + w;
      float xv[XCAP];
#pragma unroll
      for (int j = 0; j < XCAP; ++j)
        xv[j] = (j < csp && nvalid) ? x[(size_t)n * p.Cs + (size_t)m * csp + j] : 0.f;
      const float* Dm = D + (size_t)m * p.K * csp;
      for (int k = 0; k < p.K; ++k) {
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < XCAP; ++j)
          if (j < csp) s = fmaf(Dm[(size_t)k * csp + j], xv[j], s);
        lut[(w * p.K + k) * kWave + lane] = s;
      }
    }
    __syncthreads();
    // ---- gather, Eq. (5)
    for (int w = 0; w < cnt; ++w) {
      const int m = mc + w;
      const float* row = lut + w * p.K * kWave + lane;
#pragma unroll
      for (int i = 0; i < kTW; ++i) {
        const int t = tbase + i;
        if (t < p.Ct) {
          uint32_t code = code_at(codes, (size_t)t * p.M + m);
          code = code < kmax ? code : kmax;
          acc[i] += row[code * kWave];
        }
      }
    }
  }

  if (!nvalid) return;
#pragma unroll
  for (int i = 0; i < kTW; ++i) {
    const int t = tbase + i;
    if (t >= p.Ct) continue;
    if (partial) {
      partial[((size_t)split * p.N + n) * p.Ct + t] = acc[i];
    } else {
      float v = acc[i] + (bias ? bias[t] : 0.f);
      if (p.relu) v = fmaxf(v, 0.f);
      y[(size_t)n * p.Ct + t] = v;
    }
  }
}

// y = sum over splits (in split order) + bias, then ReLU.
__global__ __launch_bounds__(256) void fc_reduce_kernel(const float* __restrict__ partial, int splits, int N, int Ct,
                                                        const float* __restrict__ bias, int relu,
                                                        float* __restrict__ y) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t total = (size_t)N * Ct;
  if (i >= total) return;
  float s = partial[i];
  for (int k = 1; k < splits; ++k) s += partial[(size_t)k * total + i];
  if (bias) s += bias[i % Ct];
  if (relu) s = fmaxf(s, 0.f);
  y[i] = s;
}

}  // namespace

hipError_t launch_fc_forward(int N, int Cs, int M, int K, int Csp, int Ct, const float* x, const float* D,
                             CodeStream codes, const float* bias, int relu, float* y, hipStream_t stream) {
  if (fc_tiled_supported(N, Cs, M, K, Csp, Ct))
    return launch_fc_tiled(N, Cs, M, K, Csp, Ct, x, D, codes, bias, relu, y, stream);
  FcParams p;
  float* partial = nullptr;
  p.N = N;
  p.Cs = Cs;
  p.M = M;
  p.K = K;
  p.Csp = Csp;
  p.Ct = Ct;
  p.relu = relu;
  const size_t per_m = (size_t)K * kWave * sizeof(float);
  p.mchunk = (int)std::max<size_t>(1, std::min<size_t>(kWaves, kLdsBudget / per_m));
  const int tblocks = ceil_div(Ct, kWaves * kTW);
  const int nblocks = ceil_div(N, kWave);
  // Enough workgroups to cover the chip about twice, each with at least a
  // few chunks of subspaces.
  int splits = ceil_div(512, tblocks * nblocks);
  splits = std::max(1, std::min(splits, ceil_div(M, 4 * p.mchunk)));
  p.m_per_split = ceil_div(M, splits);
  splits = ceil_div(M, p.m_per_split);
  const size_t lds = (size_t)p.mchunk * per_m;

  hipError_t e;
  Scratch scratch;
  if (splits > 1) {
    e = scratch.acquire(stream, (size_t)splits * N * Ct * sizeof(float));
    if (e != hipSuccess) return e;
    partial = reinterpret_cast<float*>(scratch.get());
  }
  dim3 grid(tblocks, nblocks, splits);
  void (*kern)(const float*, const float*, CodeStream, const float*, float*, float*, FcParams);
  switch (Csp) {
    case 1: kern = fc_pq_kernel<1>; break;
    case 2: kern = fc_pq_kernel<2>; break;
    case 3: kern = fc_pq_kernel<3>; break;
    case 4: kern = fc_pq_kernel<4>; break;
    case 8: kern = fc_pq_kernel<8>; break;
    default: kern = fc_pq_kernel<0>; break;
  }
  e = allow_max_lds((const void*)kern);
  if (e == hipSuccess) {
    LaunchTimer timer;
    e = timed_launch(&timer, kern, grid, dim3(kThreads), (uint32_t)lds, stream, x, D, codes, bias, y, partial, p);
  }
  if (e == hipSuccess && splits > 1) {
    const size_t total = (size_t)N * Ct;
    hipLaunchKernelGGL(fc_reduce_kernel, dim3((unsigned)ceil_div_z(total, 256)), dim3(256), 0, stream,
                       partial, splits, N, Ct, bias, relu, y);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace qcnn
