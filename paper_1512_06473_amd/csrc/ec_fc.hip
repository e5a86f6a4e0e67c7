// Error-corrected quantization of a fully-connected layer.
//
// Paper: Sec. 3.3.1.  With the layer inputs S_n and desired responses T_n of
// N images, the sub-codebooks D^(m) and assignments B^(m) minimise the
// response error of Eq. (8) by block coordinate descent over the subspaces:
// for subspace m, the residual of the others R^(m) (Eq. (9)) is fitted by
// alternating the sub-codebook update of Eq. (11) (a least-squares problem
// per sub-codeword over the output channels assigned to it) and the
// assignment update of Eq. (12) (the best sub-codeword per output channel).
// With G = S^(m)T S^(m) and P = S^(m)T R^(m), Eq. (11) is
// |L_k| G D_k = sum_{c in L_k} P_c and Eq. (12) minimises
// D_k^T G D_k - 2 D_k^T P_c, so only P touches the large arrays.
//
// State, all float64: E = T - Y, the residual of the whole quantized layer
// [N][C_t]; the sub-codebooks D64; the Gram blocks G[m].  Per subspace m:
//   ec_pass_kernel   one pass over E: adds back the change of the subspace
//                    updated just before (E += S^(m') (W_old - W_new)), sums
//                    E^2 (the objective after that step, Eq. (8)) and the
//                    partial products S^(m)T E over chunks of images;
//   ec_reduce_kernel P = sum of the partials (fixed order) + G W^(m), so that
//                    P = S^(m)T R^(m) with R^(m) = E + S^(m) W^(m);
//   ec_fit_kernel    one workgroup: Eq. (11) for every sub-codeword;
//   ec_assign_kernel one thread per output channel: Eq. (12);
//                    the last two `inner` times.
// Readings (shared with the oracle): the descent starts from the given
// sub-codebooks and codes; a sweep visits m in order; a sub-codeword no
// channel uses keeps its value; the normal equations are solved by
// elimination in channel order without row exchanges, a pivot <= 1e-12 x
// the largest diagonal entry of G dropping that coordinate (set to 0);
// assignment ties go to the lowest index.
//
// Bound: HBM.  A subspace step reads and writes E once (16 N C_t bytes) and
// reads S^(m) (4 N C'_s bytes); the fit kernel is latency-bound on one CU.
#include "qcnn_internal.h"

namespace qcnn {
namespace {

constexpr int kEcThreads = 256;      // pass / reduce kernels
constexpr int kEcChunk = 16;         // images per pass workgroup
constexpr int kUpdThreads = 256;     // update kernel (one workgroup; up to 512 registers per lane)
constexpr int kMaxCsp = 16;

struct EcParams {
  int N, Cs, Ct, M, K, Csp, inner;
  int nchunks;
};

__device__ __forceinline__ uint32_t ec_code(const uint8_t* codes, int c, int M, int m, int K) {
  const uint32_t k = codes[(size_t)c * M + m];
  return k < (uint32_t)K ? k : (uint32_t)(K - 1);
}

// E = T, D64 = codebooks, G[m][i][j] = sum_n S[n][m C's + i] S[n][m C's + j].
__global__ __launch_bounds__(kEcThreads) void ec_init_kernel(const float* __restrict__ S, const float* __restrict__ T,
                                                           const float* __restrict__ D, EcParams p,
                                                           double* __restrict__ E, double* __restrict__ D64,
                                                           double* __restrict__ G) {
  const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x, stride = (size_t)gridDim.x * blockDim.x;
  const size_t ne = (size_t)p.N * p.Ct, nd = (size_t)p.M * p.K * p.Csp, ng = (size_t)p.M * p.Csp * p.Csp;
  for (size_t i = tid; i < ne; i += stride) E[i] = (double)T[i];
  for (size_t i = tid; i < nd; i += stride) D64[i] = (double)D[i];
  for (size_t i = tid; i < ng; i += stride) {
    const int m = (int)(i / ((size_t)p.Csp * p.Csp));
    const int r = (int)(i % ((size_t)p.Csp * p.Csp));
    const int a = m * p.Csp + r / p.Csp, b = m * p.Csp + r % p.Csp;
    double s = 0.0;
    for (int n = 0; n < p.N; ++n) s += (double)S[(size_t)n * p.Cs + a] * (double)S[(size_t)n * p.Cs + b];
    G[i] = s;
  }
}

// One pass over E for a chunk of kEcChunk images and 256 columns.
//   apply (ma >= 0): E[n][c] -= sum_j S[n][ma C's + j] (Dnew[knew(c)][j] - Dold[kold(c)][j]);
//                    Dold == nullptr for the starting residual (W_old = 0);
//   collect (mp >= 0): part[chunk][j][c] = sum_n S[n][mp C's + j] E[n][c];
//   obj: opart[block] = sum of E[n][c]^2 over the block (after the apply).
template <int CSP>
__global__ __launch_bounds__(kEcThreads) void ec_pass_kernel(const float* __restrict__ S, EcParams p,
                                                           double* __restrict__ E, int ma,
                                                           const double* __restrict__ Dnew,
                                                           const uint8_t* __restrict__ codes,
                                                           const double* __restrict__ Dold,
                                                           const uint8_t* __restrict__ codes_old, int mp,
                                                           double* __restrict__ part, double* __restrict__ opart) {
  __shared__ double red[kEcThreads / kWave];
  const int c = blockIdx.x * kEcThreads + threadIdx.x;
  const int chunk = blockIdx.y;
  const int n0 = chunk * kEcChunk, n1 = min(p.N, n0 + kEcChunk);
  const bool col = c < p.Ct;
  double dw[CSP];
#pragma unroll
  for (int j = 0; j < CSP; ++j) dw[j] = 0.0;
  if (ma >= 0 && col) {
    const uint32_t kn = ec_code(codes, c, p.M, ma, p.K);
    const double* dn = Dnew + ((size_t)ma * p.K + kn) * CSP;
#pragma unroll
    for (int j = 0; j < CSP; ++j) dw[j] = dn[j];
    if (Dold) {
      const uint32_t ko = codes_old[c] < (uint32_t)p.K ? codes_old[c] : (uint32_t)(p.K - 1);
#pragma unroll
      for (int j = 0; j < CSP; ++j) dw[j] -= Dold[(size_t)ko * CSP + j];
    }
  }
  double acc[CSP];
#pragma unroll
  for (int j = 0; j < CSP; ++j) acc[j] = 0.0;
  double sq = 0.0;
  for (int n = n0; n < n1; ++n) {
    double e = col ? E[(size_t)n * p.Ct + c] : 0.0;
    if (ma >= 0) {
      const float* srow = S + (size_t)n * p.Cs + (size_t)ma * CSP;
      double d = 0.0;
#pragma unroll
      for (int j = 0; j < CSP; ++j) d += (double)srow[j] * dw[j];
      e -= d;
      if (col) E[(size_t)n * p.Ct + c] = e;
    }
    sq += e * e;
    if (mp >= 0) {
      const float* srow = S + (size_t)n * p.Cs + (size_t)mp * CSP;
#pragma unroll
      for (int j = 0; j < CSP; ++j) acc[j] += (double)srow[j] * e;
    }
  }
  if (mp >= 0 && col)
#pragma unroll
    for (int j = 0; j < CSP; ++j) part[((size_t)chunk * CSP + j) * p.Ct + c] = acc[j];
  if (opart) {
    // fixed-order block sum: wave shuffles, then the waves in order
    for (int off = kWave / 2; off > 0; off >>= 1) sq += __shfl_down(sq, off, kWave);
    if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = sq;
    __syncthreads();
    if (threadIdx.x == 0) {
      double s = 0.0;
      for (int w = 0; w < kEcThreads / kWave; ++w) s += red[w];
      opart[(size_t)blockIdx.y * gridDim.x + blockIdx.x] = s;
    }
  }
}

// P[j][c] = sum over chunks (in order) of part[chunk][j][c] + sum_i G[m][j][i] W^(m)[i][c].
__global__ __launch_bounds__(kEcThreads) void ec_reduce_kernel(const double* __restrict__ part, EcParams p, int m,
                                                             const double* __restrict__ G,
                                                             const double* __restrict__ D64,
                                                             const uint8_t* __restrict__ codes,
                                                             double* __restrict__ P) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (size_t)p.Csp * p.Ct) return;
  const int j = (int)(i / p.Ct), c = (int)(i % p.Ct);
  double s = 0.0;
  for (int ch = 0; ch < p.nchunks; ++ch) s += part[((size_t)ch * p.Csp + j) * p.Ct + c];
  const double* g = G + ((size_t)m * p.Csp + j) * p.Csp;
  const double* w = D64 + ((size_t)m * p.K + ec_code(codes, c, p.M, m, p.K)) * p.Csp;
  for (int q = 0; q < p.Csp; ++q) s += g[q] * w[q];
  P[i] = s;
}

// x with G x = b by elimination in channel order without row exchanges; a
// pivot <= 1e-12 x max diag(G) (or <= 0) drops that coordinate (x = 0).
__device__ __forceinline__ void solve_normal(const double* __restrict__ Gm, const double* __restrict__ bin, int n, double* x) {
  double A[kMaxCsp][kMaxCsp], y[kMaxCsp];
  bool live[kMaxCsp];
  double scale = 0.0;
  for (int i = 0; i < n; ++i) {
    for (int j = 0; j < n; ++j) A[i][j] = Gm[i * n + j];
    y[i] = bin[i];
    scale = fmax(scale, Gm[i * n + i]);
  }
  for (int j = 0; j < n; ++j) {
    live[j] = A[j][j] > 1e-12 * scale && A[j][j] > 0.0;
    if (!live[j]) continue;
    for (int i = j + 1; i < n; ++i) {
      const double f = A[i][j] / A[j][j];
      for (int q = j; q < n; ++q) A[i][q] -= f * A[j][q];
      y[i] -= f * y[j];
    }
  }
  for (int j = n - 1; j >= 0; --j) {
    x[j] = 0.0;
    if (!live[j]) continue;
    double s = y[j];
    for (int i = j + 1; i < n; ++i)
      if (live[i]) s -= A[j][i] * x[i];
    x[j] = s / A[j][j];
  }
}

// Eq. (11), one workgroup.  On the first round of a subspace (`first`) it
// also records the objective after the previous step (from the pass
// kernel's block sums) and keeps the subspace's old sub-codebook and codes
// for the next pass.  Then each sub-codeword used by some channel becomes
// the least-squares fit, and qv[k] = D_k^T G D_k for the assignment.
template <int CSP>
__global__ __launch_bounds__(kUpdThreads) void ec_fit_kernel(const double* __restrict__ P, EcParams p, int m,
                                                           const double* __restrict__ G, double* __restrict__ D64,
                                                           const uint8_t* __restrict__ codes, int first,
                                                           double* __restrict__ Dold,
                                                           uint8_t* __restrict__ codes_old,
                                                           const double* __restrict__ opart, int nopart,
                                                           double* __restrict__ objective, double* __restrict__ qv) {
  // All LDS is dynamic (the kernel may take up to the whole 160 KB, so it
  // cannot also have static LDS).
  extern __shared__ double sh[];
  double* Gs = sh;                               // [C's][C's]
  double* Ds = Gs + kMaxCsp * kMaxCsp;           // [K][C's]
  double* red = Ds + 256 * kMaxCsp;              // [threads] objective tree
  // this subspace's codes, read from the [C_t][M] array (stride M) once
  uint8_t* cs = reinterpret_cast<uint8_t*>(red + kUpdThreads);
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  constexpr int Csp = CSP;
  const int K = p.K;
  if (first && objective) {
    // the pass kernel's block sums: thread strides, then a fixed tree
    double s = 0.0;
    for (int i = tid; i < nopart; i += kUpdThreads) s += opart[i];
    red[tid] = s;
    __syncthreads();
    for (int h = kUpdThreads / 2; h > 0; h >>= 1) {
      if (tid < h) red[tid] += red[tid + h];
      __syncthreads();
    }
    if (tid == 0) *objective = red[0];
  }
  for (int i = tid; i < Csp * Csp; i += kUpdThreads) Gs[i] = G[(size_t)m * Csp * Csp + i];
  for (int i = tid; i < K * Csp; i += kUpdThreads) {
    Ds[i] = D64[(size_t)m * K * Csp + i];
    if (first) Dold[i] = Ds[i];
  }
  // the codes (stride M bytes apart): eight loads in flight per thread
  for (int c0 = tid; c0 < p.Ct; c0 += 8 * kUpdThreads) {
    uint8_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int c = c0 + u * kUpdThreads;
      v[u] = c < p.Ct ? (uint8_t)ec_code(codes, c, p.M, m, K) : 0;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int c = c0 + u * kUpdThreads;
      if (c < p.Ct) {
        if (first) codes_old[c] = v[u];
        cs[c] = v[u];
      }
    }
  }
  __syncthreads();
  // Wave w fits sub-codewords in groups of KC (k = KC w .. KC w + KC - 1,
  // then KC (w + 4) ...; KC C'_s <= 32 bins per lane): its lanes read the
  // channels c = lane, lane + 64, ... in
  // order, each channel's P_c once and unconditionally (coalesced, several
  // loads in flight), adding it to the bin of its code; the wave then adds
  // the lanes' bins in a fixed tree.
  constexpr int KC = CSP <= 4 ? 8 : (CSP <= 8 ? 4 : 2);
  for (int kbase = wave * KC; kbase < K; kbase += (kUpdThreads / kWave) * KC) {
    double b[KC][CSP];
    int cnt[KC];
#pragma unroll
    for (int u = 0; u < KC; ++u) {
      cnt[u] = 0;
#pragma unroll
      for (int j = 0; j < CSP; ++j) b[u][j] = 0.0;
    }
    for (int c = lane; c < p.Ct; c += kWave) {
      const int kc = (int)cs[c] - kbase;
      double pc[CSP];
#pragma unroll
      for (int j = 0; j < CSP; ++j) pc[j] = P[(size_t)j * p.Ct + c];
#pragma unroll
      for (int u = 0; u < KC; ++u) {
        const bool hit = kc == u;
        cnt[u] += hit ? 1 : 0;
#pragma unroll
        for (int j = 0; j < CSP; ++j) b[u][j] += hit ? pc[j] : 0.0;
      }
    }
#pragma unroll
    for (int u = 0; u < KC; ++u)
      for (int off = kWave / 2; off > 0; off >>= 1) {
        cnt[u] += __shfl_down(cnt[u], off, kWave);
#pragma unroll
        for (int j = 0; j < CSP; ++j) b[u][j] += __shfl_down(b[u][j], off, kWave);
      }
    if (lane == 0) {
#pragma unroll
      for (int u = 0; u < KC; ++u) {
        const int k = kbase + u;
        if (k < K && cnt[u] > 0) {
          double x[kMaxCsp];
          solve_normal(Gs, b[u], Csp, x);
          for (int j = 0; j < Csp; ++j) Ds[k * Csp + j] = x[j] / cnt[u];
        }
      }
    }
  }
  __syncthreads();
  for (int k = tid; k < K; k += kUpdThreads) {  // D_k^T G D_k
    double s = 0.0;
    for (int i = 0; i < Csp; ++i) {
      double g = 0.0;
      for (int j = 0; j < Csp; ++j) g += Gs[i * Csp + j] * Ds[k * Csp + j];
      s += Ds[k * Csp + i] * g;
    }
    qv[k] = s;
  }
  for (int i = tid; i < K * Csp; i += kUpdThreads) D64[(size_t)m * K * Csp + i] = Ds[i];
}

// Eq. (12), one thread per output channel: the first k minimising
// D_k^T G D_k - 2 D_k^T P_c.
template <int CSP>
__global__ __launch_bounds__(kEcThreads) void ec_assign_kernel(const double* __restrict__ P, EcParams p, int m,
                                                             const double* __restrict__ D64,
                                                             const double* __restrict__ qv,
                                                             uint8_t* __restrict__ codes) {
  extern __shared__ double sd[];  // [K][C's], then [K]
  double* q = sd + (size_t)p.K * CSP;
  for (int i = threadIdx.x; i < p.K * CSP; i += kEcThreads) sd[i] = D64[(size_t)m * p.K * CSP + i];
  for (int i = threadIdx.x; i < p.K; i += kEcThreads) q[i] = qv[i];
  __syncthreads();
  const int c = blockIdx.x * kEcThreads + threadIdx.x;
  if (c >= p.Ct) return;
  double pc[CSP];
#pragma unroll
  for (int j = 0; j < CSP; ++j) pc[j] = P[(size_t)j * p.Ct + c];
  int best = 0;
  double bv = 0.0;
  for (int k = 0; k < p.K; ++k) {
    double d = 0.0;
#pragma unroll
    for (int j = 0; j < CSP; ++j) d += sd[k * CSP + j] * pc[j];
    const double v = q[k] - 2.0 * d;
    if (k == 0 || v < bv) {
      bv = v;
      best = k;
    }
  }
  codes[(size_t)c * p.M + m] = (uint8_t)best;
}

__global__ __launch_bounds__(kEcThreads) void ec_finish_kernel(const double* __restrict__ D64, size_t nd,
                                                             float* __restrict__ D, const double* __restrict__ opart,
                                                             int nopart, double* __restrict__ objective) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nd) D[i] = (float)D64[i];
  if (i == 0 && objective) {  // once per call: a serial sum is fine here
    double s = 0.0;
    for (int b = 0; b < nopart; ++b) s += opart[b];
    *objective = s;
  }
}

}  // namespace

size_t ec_fc_workspace(int N, int Ct, int M, int K, int Csp) {
  const int nchunks = ceil_div(N, kEcChunk);
  const size_t cblocks = (size_t)ceil_div(Ct, kEcThreads);
  size_t b = 0;
  b += (size_t)N * Ct * 8;                       // E
  b += (size_t)nchunks * Csp * Ct * 8;           // partial P
  b += (size_t)Csp * Ct * 8;                     // P
  b += (size_t)M * Csp * Csp * 8;                // G
  b += (size_t)M * K * Csp * 8;                  // D64
  b += (size_t)K * Csp * 8;                      // Dold
  b += (size_t)K * 8;                            // q
  b += cblocks * nchunks * 8;                    // objective partials
  b += (size_t)Ct + 64;                          // codes_old
  return b + 16 * 256;                           // each slice is rounded up to 256 bytes
}

template <int CSP>
hipError_t launch_ec_csp(int N, int Cs, int Ct, int M, int K, const float* S, const float* T, float* D,
                         uint8_t* codes, int sweeps, int inner, double* objective, hipStream_t stream) {
  constexpr int Csp = CSP;
  EcParams p{N, Cs, Ct, M, K, Csp, inner, ceil_div(N, kEcChunk)};
  const size_t cblocks = (size_t)ceil_div(Ct, kEcThreads);
  const int nopart = (int)(cblocks * p.nchunks);
  Scratch scratch;
  hipError_t e = scratch.acquire(stream, ec_fc_workspace(N, Ct, M, K, Csp));
  auto pass = ec_pass_kernel<CSP>;
  auto fit = ec_fit_kernel<CSP>;
  auto assign = ec_assign_kernel<CSP>;
  if (e != hipSuccess) return e;
  char* w = scratch.get();
  auto take = [&](size_t bytes) {
    char* r = w;
    w += (bytes + 255) & ~(size_t)255;
    return r;
  };
  double* E = reinterpret_cast<double*>(take((size_t)N * Ct * 8));
  double* part = reinterpret_cast<double*>(take((size_t)p.nchunks * Csp * Ct * 8));
  double* P = reinterpret_cast<double*>(take((size_t)Csp * Ct * 8));
  double* G = reinterpret_cast<double*>(take((size_t)M * Csp * Csp * 8));
  double* D64 = reinterpret_cast<double*>(take((size_t)M * K * Csp * 8));
  double* Dold = reinterpret_cast<double*>(take((size_t)K * Csp * 8));
  double* qv = reinterpret_cast<double*>(take((size_t)K * 8));
  double* opart = reinterpret_cast<double*>(take((size_t)nopart * 8));
  uint8_t* codes_old = reinterpret_cast<uint8_t*>(take((size_t)Ct));

  const size_t ninit = std::max<size_t>({(size_t)N * Ct, (size_t)M * K * Csp, (size_t)M * Csp * Csp});
  hipLaunchKernelGGL(ec_init_kernel, dim3((unsigned)std::min<size_t>(8192, ceil_div_z(ninit, kEcThreads))),
                     dim3(kEcThreads), 0, stream, S, T, D, p, E, D64, G);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const dim3 pgrid((unsigned)cblocks, (unsigned)p.nchunks);
  // Starting residual E = T - sum_m S^(m) W^(m); the last pass also sums E^2.
  for (int m = 0; m < M; ++m) {
    hipLaunchKernelGGL(pass, pgrid, dim3(kEcThreads), 0, stream, S, p, E, m, D64,
                       (const uint8_t*)codes, (const double*)nullptr, (const uint8_t*)nullptr, -1, part,
                       m == M - 1 ? opart : nullptr);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const size_t fit_lds = (kMaxCsp * kMaxCsp + 256 * kMaxCsp + kUpdThreads) * sizeof(double) + (size_t)Ct;
  const size_t asg_lds = (size_t)K * (Csp + 1) * sizeof(double);
  if (fit_lds > kLdsBytes) return hipErrorInvalidValue;
  if ((e = allow_max_lds((const void*)fit)) != hipSuccess) return e;
  int step = 0;
  int ma = -1;  // subspace updated by the previous step, whose change the next pass applies
  for (int s = 0; s < sweeps; ++s) {
    for (int m = 0; m < M; ++m, ++step) {
      hipLaunchKernelGGL(pass, pgrid, dim3(kEcThreads), 0, stream, S, p, E, ma, D64,
                         (const uint8_t*)codes, ma >= 0 ? (const double*)Dold : nullptr,
                         (const uint8_t*)codes_old, m, part, ma >= 0 ? opart : nullptr);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      hipLaunchKernelGGL(ec_reduce_kernel, dim3((unsigned)ceil_div_z((size_t)Csp * Ct, kEcThreads)),
                         dim3(kEcThreads), 0, stream, part, p, m, G, D64, (const uint8_t*)codes, P);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      for (int it = 0; it < inner; ++it) {
        // objective[step] is the value before this step (after the previous one)
        hipLaunchKernelGGL(fit, dim3(1), dim3(kUpdThreads), fit_lds, stream, P, p, m, G, D64,
                           (const uint8_t*)codes, it == 0 ? 1 : 0, Dold, codes_old, opart, nopart,
                           objective ? objective + step : nullptr, qv);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(assign, dim3((unsigned)cblocks), dim3(kEcThreads), asg_lds, stream, P, p, m,
                           (const double*)D64, (const double*)qv, codes);
        if ((e = hipGetLastError()) != hipSuccess) return e;
      }
      ma = m;
    }
  }
  if (ma >= 0) {  // apply the last step and sum the final objective
    hipLaunchKernelGGL(pass, pgrid, dim3(kEcThreads), 0, stream, S, p, E, ma, D64,
                       (const uint8_t*)codes, (const double*)Dold, (const uint8_t*)codes_old, -1, part, opart);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const size_t nd = (size_t)M * K * Csp;
  hipLaunchKernelGGL(ec_finish_kernel, dim3((unsigned)ceil_div_z(nd, kEcThreads)), dim3(kEcThreads), 0, stream, D64,
                     nd, D, opart, nopart, objective ? objective + step : nullptr);
  return hipGetLastError();
}

hipError_t launch_ec_fc(int N, int Cs, int Ct, int M, int K, int Csp, const float* S, const float* T, float* D,
                        uint8_t* codes, int sweeps, int inner, double* objective, hipStream_t stream) {
#define QCNN_EC_CASE(c) \
  case c: return launch_ec_csp<c>(N, Cs, Ct, M, K, S, T, D, codes, sweeps, inner, objective, stream);
  switch (Csp) {
    QCNN_EC_CASE(1) QCNN_EC_CASE(2) QCNN_EC_CASE(3) QCNN_EC_CASE(4) QCNN_EC_CASE(5) QCNN_EC_CASE(6)
    QCNN_EC_CASE(7) QCNN_EC_CASE(8) QCNN_EC_CASE(9) QCNN_EC_CASE(10) QCNN_EC_CASE(11) QCNN_EC_CASE(12)
    QCNN_EC_CASE(13) QCNN_EC_CASE(14) QCNN_EC_CASE(15) QCNN_EC_CASE(16)
    default: return hipErrorInvalidValue;
  }
#undef QCNN_EC_CASE
}

}  // namespace qcnn
