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
// State, all float64 but the codes: E = T - Y, the residual of the whole
// quantized layer [N][C_t]; the sub-codebooks D64; the Gram blocks G[m]; the
// codes transposed to [M][C_t] (one subspace's codes contiguous), written
// back to [C_t][M] at the end.  ec_start_kernel forms the starting E in one
// pass over the subspaces.  Per subspace m:
//   ec_step_kernel   one pass over E: finishes the subspace m' fitted just
//                    before (its assignment, Eq. (12), then
//                    E -= S^(m') (W_new - W_old)), sums E^2 (the objective
//                    after that step, Eq. (8)) and the partial products
//                    S^(m)T E over chunks of images;
//   ec_reduce_kernel P = sum of the partials (fixed order) + G W^(m), so that
//                    P = S^(m)T R^(m) with R^(m) = E + S^(m) W^(m); then, per
//                    block of channels, the sums of P_c over the channels
//                    assigned to each sub-codeword;
//   ec_fit_kernel    one workgroup: adds the blocks' sums and solves Eq. (11)
//                    for every sub-codeword.
// With `inner` > 1 the reduce kernel's second form (assignment from P, then
// the sums) and the fit kernel repeat before the next step kernel.
// Readings (shared with the oracle): the descent starts from the given
// sub-codebooks and codes; a sweep visits m in order; a sub-codeword no
// channel uses keeps its value; the normal equations are solved by
// elimination in channel order without row exchanges, a pivot <= 1e-12 x
// the largest diagonal entry of G dropping that coordinate (set to 0);
// assignment ties go to the lowest index.
//
// Bound: HBM.  A subspace step reads and writes E once (16 N C_t bytes) and
// reads S^(m) (4 N C'_s bytes); the fit kernel is latency-bound on one CU.
// The starting residual is fp64 arithmetic, 2 N C_t C_s flops once.
#include "qcnn_internal.h"

namespace qcnn {
namespace {

constexpr int kEcThreads = 256;      // pass / reduce kernels
constexpr int kEcChunk = 16;         // images per pass workgroup
constexpr int kUpdThreads = 256;     // update kernel (one workgroup; up to 512 registers per lane)

struct EcParams {
  int N, Cs, Ct, M, K, Csp, inner;
  int nchunks;
};

// D64 = codebooks, ct[m][c] = codes[c][m] (codes >= K read as K - 1),
// G[m][i][j] = sum_n S[n][m C's + i] S[n][m C's + j].
__global__ __launch_bounds__(kEcThreads) void ec_init_kernel(const float* __restrict__ S, const float* __restrict__ D,
                                                           const uint8_t* __restrict__ codes, EcParams p,
                                                           double* __restrict__ D64, uint8_t* __restrict__ ct,
                                                           double* __restrict__ G) {
  const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x, stride = (size_t)gridDim.x * blockDim.x;
  const size_t nc = (size_t)p.M * p.Ct, nd = (size_t)p.M * p.K * p.Csp, ng = (size_t)p.M * p.Csp * p.Csp;
  for (size_t i = tid; i < nc; i += stride) {
    const size_t m = i / p.Ct, c = i % p.Ct;
    const uint8_t k = codes[c * p.M + m];
    ct[i] = k < p.K ? k : (uint8_t)(p.K - 1);
  }
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

// Fixed-order sum of one value per thread over the workgroup (wave
// shuffles, then the waves in order) into opart[block].
__device__ __forceinline__ void ec_block_sum(double v, double* red, double* __restrict__ opart) {
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_down(v, off, kWave);
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int w = 0; w < kEcThreads / kWave; ++w) s += red[w];
    opart[(size_t)blockIdx.y * gridDim.x + blockIdx.x] = s;
  }
}

// The starting residual E = T - sum_m S^(m) W^(m) for a chunk of kEcChunk
// images and 256 columns (one column per thread, the chunk's E in
// registers, the subspaces in order), and its block sums of E^2.
template <int CSP>
__global__ __launch_bounds__(kEcThreads) void ec_start_kernel(const float* __restrict__ S,
                                                            const float* __restrict__ T, EcParams p,
                                                            const double* __restrict__ D64,
                                                            const uint8_t* __restrict__ ct,
                                                            double* __restrict__ E, double* __restrict__ opart) {
  __shared__ double red[kEcThreads / kWave];
  const int c = blockIdx.x * kEcThreads + threadIdx.x;
  const int n0 = blockIdx.y * kEcChunk, nn = min(p.N - n0, kEcChunk);
  const bool col = c < p.Ct;
  double e[kEcChunk];
#pragma unroll
  for (int i = 0; i < kEcChunk; ++i) e[i] = col && i < nn ? (double)T[(size_t)(n0 + i) * p.Ct + c] : 0.0;
  if (col) {
    for (int m = 0; m < p.M; ++m) {
      const double* w = D64 + ((size_t)m * p.K + ct[(size_t)m * p.Ct + c]) * CSP;
      double dw[CSP];
#pragma unroll
      for (int j = 0; j < CSP; ++j) dw[j] = w[j];
#pragma unroll
      for (int i = 0; i < kEcChunk; ++i) {
        if (i < nn) {
          const float* srow = S + (size_t)(n0 + i) * p.Cs + (size_t)m * CSP;
          double d = 0.0;
#pragma unroll
          for (int j = 0; j < CSP; ++j) d += (double)srow[j] * dw[j];
          e[i] -= d;
        }
      }
    }
  }
  double sq = 0.0;
#pragma unroll
  for (int i = 0; i < kEcChunk; ++i) {
    if (col && i < nn) E[(size_t)(n0 + i) * p.Ct + c] = e[i];
    sq += e[i] * e[i];
  }
  ec_block_sum(sq, red, opart);
}

// Eq. (12) for one output channel: the first k minimising
// D_k^T G D_k - 2 D_k^T P_c, with sd = D^(m) [K][C's] and q[k] = D_k^T G D_k.
template <int CSP>
__device__ __forceinline__ int ec_best(const double* sd, const double* q, int K, const double (&pc)[CSP]) {
  int best = 0;
  double bv = 0.0;
  for (int k = 0; k < K; ++k) {
    double d = 0.0;
#pragma unroll
    for (int j = 0; j < CSP; ++j) d += sd[k * CSP + j] * pc[j];
    const double v = q[k] - 2.0 * d;
    if (k == 0 || v < bv) {
      bv = v;
      best = k;
    }
  }
  return best;
}

// One pass over E for a chunk of kEcChunk images and 256 columns, after the
// fit of subspace ma (ma >= 0) and before that of mp (mp >= 0):
//   assign:  knew(c) by Eq. (12) from P (still that of ma), D^(ma) and q;
//            the chunk-0 workgroup stores it in ct[ma];
//   apply:   E[n][c] -= sum_j S[n][ma C's + j] (D^(ma)[knew(c)][j] - Dold[kold(c)][j]);
//   collect: part[chunk][j][c] = sum_n S[n][mp C's + j] E[n][c];
//   obj:     opart[block] = sum of E[n][c]^2 over the block (after the apply).
// The chunk's E is loaded into registers before any of it is written, so
// the loads are all in flight together.
template <int CSP>
__global__ __launch_bounds__(kEcThreads) void ec_step_kernel(const float* __restrict__ S, EcParams p,
                                                           double* __restrict__ E, int ma,
                                                           const double* __restrict__ P,
                                                           const double* __restrict__ D64,
                                                           const double* __restrict__ qv, uint8_t* __restrict__ ct,
                                                           const double* __restrict__ Dold,
                                                           const uint8_t* __restrict__ codes_old, int mp,
                                                           double* __restrict__ part, double* __restrict__ opart) {
  extern __shared__ double sd[];  // D^(ma) [K][C's], q [K], block-sum scratch [4]
  double* q = sd + (size_t)p.K * CSP;
  double* red = q + p.K;
  const int c = blockIdx.x * kEcThreads + threadIdx.x;
  const int chunk = blockIdx.y;
  const int n0 = chunk * kEcChunk, nn = min(p.N - n0, kEcChunk);
  const bool col = c < p.Ct;
  double e[kEcChunk];
#pragma unroll
  for (int i = 0; i < kEcChunk; ++i) e[i] = col && i < nn ? E[(size_t)(n0 + i) * p.Ct + c] : 0.0;
  if (ma >= 0) {
    // this channel's P_c and old sub-codeword are fetched before the LDS fill
    double pc[CSP], dd[CSP];
#pragma unroll
    for (int j = 0; j < CSP; ++j) pc[j] = col ? P[(size_t)j * p.Ct + c] : 0.0;
    const double* ddp = Dold + (size_t)(col ? codes_old[c] : 0) * CSP;
#pragma unroll
    for (int j = 0; j < CSP; ++j) dd[j] = ddp[j];
    for (int i = threadIdx.x; i < p.K * CSP; i += kEcThreads) sd[i] = D64[(size_t)ma * p.K * CSP + i];
    for (int i = threadIdx.x; i < p.K; i += kEcThreads) q[i] = qv[i];
    __syncthreads();
    if (col) {
      const int kn = ec_best<CSP>(sd, q, p.K, pc);
      if (chunk == 0) ct[(size_t)ma * p.Ct + c] = (uint8_t)kn;
      double dw[CSP];
#pragma unroll
      for (int j = 0; j < CSP; ++j) dw[j] = sd[kn * CSP + j] - dd[j];
#pragma unroll
      for (int i = 0; i < kEcChunk; ++i) {
        if (i < nn) {
          const float* srow = S + (size_t)(n0 + i) * p.Cs + (size_t)ma * CSP;
          double d = 0.0;
#pragma unroll
          for (int j = 0; j < CSP; ++j) d += (double)srow[j] * dw[j];
          e[i] -= d;
          E[(size_t)(n0 + i) * p.Ct + c] = e[i];
        }
      }
    }
  }
  if (mp >= 0 && col) {
    double acc[CSP];
#pragma unroll
    for (int j = 0; j < CSP; ++j) acc[j] = 0.0;
#pragma unroll
    for (int i = 0; i < kEcChunk; ++i) {
      if (i < nn) {
        const float* srow = S + (size_t)(n0 + i) * p.Cs + (size_t)mp * CSP;
#pragma unroll
        for (int j = 0; j < CSP; ++j) acc[j] += (double)srow[j] * e[i];
      }
    }
#pragma unroll
    for (int j = 0; j < CSP; ++j) part[((size_t)chunk * CSP + j) * p.Ct + c] = acc[j];
  }
  double sq = 0.0;
#pragma unroll
  for (int i = 0; i < kEcChunk; ++i) sq += e[i] * e[i];
  ec_block_sum(sq, red, opart);
}

// Doubles of the reduce kernel's LDS after its P block: D^(m) and q, later
// reused for the quarter sums of one group of 64 sub-codewords.
__host__ __device__ constexpr size_t red_area(int K, int Csp) {
  return (size_t)K * (Csp + 1) > (size_t)(kEcThreads / kWave) * kWave * (Csp + 1)
             ? (size_t)K * (Csp + 1)
             : (size_t)(kEcThreads / kWave) * kWave * (Csp + 1);
}

// Per block of 256 output channels, for subspace m:
//   assign == 0: P[j][c] = sum over chunks (in order) of part[chunk][j][c]
//                + sum_i G[m][j][i] W^(m)[i][c], so that P = S^(m)T R^(m);
//                codes_old[c] = ct[m][c];
//   assign == 1: ct[m][c] by Eq. (12) from P, D^(m) and q (a later round);
// then, in channel order, the block's sums over the channels assigned to
// each sub-codeword: bins[block][k][j] = sum of P[j][c], nbin[block][k] the
// number of those channels.
template <int CSP>
__global__ __launch_bounds__(kEcThreads) void ec_reduce_kernel(const double* __restrict__ part, EcParams p, int m,
                                                             const double* __restrict__ G,
                                                             const double* __restrict__ D64,
                                                             const double* __restrict__ qv, int assign,
                                                             uint8_t* __restrict__ ct, double* __restrict__ P,
                                                             uint8_t* __restrict__ codes_old,
                                                             double* __restrict__ bins, int* __restrict__ nbin) {
  extern __shared__ double sr[];
  double* Pl = sr;                             // [C's][256] this block's P
  double* sd = Pl + CSP * kEcThreads;          // [K][C's] D^(m) (assign == 1)
  double* q = sd + (size_t)p.K * CSP;          // [K]
  // [256] codes, after the larger of that and the quarter sums below
  uint8_t* ks = reinterpret_cast<uint8_t*>(sd + red_area(p.K, CSP));
  const int tid = threadIdx.x, c = blockIdx.x * kEcThreads + tid;
  const bool col = c < p.Ct;
  double pc[CSP];
  int k = 0;
  if (assign) {
    for (int i = tid; i < p.K * CSP; i += kEcThreads) sd[i] = D64[(size_t)m * p.K * CSP + i];
    for (int i = tid; i < p.K; i += kEcThreads) q[i] = qv[i];
    __syncthreads();
    if (col) {
#pragma unroll
      for (int j = 0; j < CSP; ++j) pc[j] = P[(size_t)j * p.Ct + c];
      k = ec_best<CSP>(sd, q, p.K, pc);
      ct[(size_t)m * p.Ct + c] = (uint8_t)k;
    }
  } else if (col) {
    k = ct[(size_t)m * p.Ct + c];
#pragma unroll
    for (int j = 0; j < CSP; ++j) pc[j] = 0.0;
    // the chunks in order, eight chunks' loads in flight at a time
    for (int ch0 = 0; ch0 < p.nchunks; ch0 += 8) {
      double v[8][CSP];
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int j = 0; j < CSP; ++j)
          v[u][j] = ch0 + u < p.nchunks ? part[((size_t)(ch0 + u) * CSP + j) * p.Ct + c] : 0.0;
#pragma unroll
      for (int u = 0; u < 8; ++u)
#pragma unroll
        for (int j = 0; j < CSP; ++j)
          if (ch0 + u < p.nchunks) pc[j] += v[u][j];
    }
    const double* g = G + (size_t)m * CSP * CSP;
    const double* w = D64 + ((size_t)m * p.K + k) * CSP;
#pragma unroll
    for (int j = 0; j < CSP; ++j) {
#pragma unroll
      for (int i = 0; i < CSP; ++i) pc[j] += g[j * CSP + i] * w[i];
      P[(size_t)j * p.Ct + c] = pc[j];
    }
    codes_old[c] = (uint8_t)k;
  }
#pragma unroll
  for (int j = 0; j < CSP; ++j) Pl[j * kEcThreads + tid] = col ? pc[j] : 0.0;
  ks[tid] = (uint8_t)k;
  __syncthreads();
  // For k in groups of 64, wave w sums the channels of its quarter (in
  // order) for k = group + lane: branch-free, every lane reads the same P_c
  // (a broadcast).  The quarters' sums are then added in order.
  constexpr int kQ = kEcThreads / kWave;
  double* qs = sd;  // [4][64][C's] quarter sums (sd is free again)
  int* qn = reinterpret_cast<int*>(qs + kQ * kWave * CSP);  // [4][64]
  const int lane = tid & (kWave - 1), wave = tid / kWave;
  const int i0 = wave * kWave;
  const int i1 = min(i0 + kWave, p.Ct - (int)blockIdx.x * kEcThreads);
  for (int k0 = 0; k0 < p.K; k0 += kWave) {
    __syncthreads();  // sd / qs may still be read
    const int kk = k0 + lane;
    double b[CSP];
#pragma unroll
    for (int j = 0; j < CSP; ++j) b[j] = 0.0;
    int n = 0;
#pragma unroll 4
    for (int i = i0; i < i1; ++i) {
      const bool hit = ks[i] == kk;
      n += hit ? 1 : 0;
#pragma unroll
      for (int j = 0; j < CSP; ++j) b[j] += hit ? Pl[j * kEcThreads + i] : 0.0;
    }
#pragma unroll
    for (int j = 0; j < CSP; ++j) qs[(wave * kWave + lane) * CSP + j] = b[j];
    qn[wave * kWave + lane] = n;
    __syncthreads();
    const int nk = min(kWave, p.K - k0);
    for (int i = tid; i < nk * CSP; i += kEcThreads) {
      double v = 0.0;
      for (int w = 0; w < kQ; ++w) v += qs[w * kWave * CSP + i];
      bins[((size_t)blockIdx.x * p.K + k0) * CSP + i] = v;
    }
    for (int i = tid; i < nk; i += kEcThreads) {
      int v = 0;
      for (int w = 0; w < kQ; ++w) v += qn[w * kWave + i];
      nbin[(size_t)blockIdx.x * p.K + k0 + i] = v;
    }
  }
}

// Threads of the fit kernel that solve at once, and the LDS each takes for
// its elimination (registers up to C'_s = 8).
template <int CSP> constexpr int fit_solvers() { return CSP <= 8 ? kUpdThreads : 16; }
template <int CSP> constexpr int fit_solve_lds() {
  return CSP <= 8 ? 0 : fit_solvers<CSP>() * CSP * CSP * (int)sizeof(double);
}
template <int CSP> size_t fit_lds_bytes(int K) {
  return (size_t)(CSP * CSP + 2 * K * CSP + kUpdThreads) * sizeof(double) + fit_solve_lds<CSP>() +
         (size_t)K * sizeof(int);
}

// Eq. (11), one workgroup.  On the first round of a subspace (`first`) it
// also records the objective after the previous step (from the step
// kernel's block sums) and keeps the subspace's old sub-codebook for the
// next step kernel.  b_k and |L_k| are the sums over the channel blocks (in
// order) of the reduce kernel's bins; each sub-codeword used by some channel
// becomes G^-1 b_k / |L_k|, and qv[k] = D_k^T G D_k for the assignment.
template <int CSP>
__global__ __launch_bounds__(kUpdThreads) void ec_fit_kernel(const double* __restrict__ bins,
                                                           const int* __restrict__ nbin, int nblk, EcParams p,
                                                           int m, const double* __restrict__ G,
                                                           double* __restrict__ D64, int first,
                                                           double* __restrict__ Dold,
                                                           const double* __restrict__ opart, int nopart,
                                                           double* __restrict__ objective, double* __restrict__ qv) {
  // All LDS is dynamic (the kernel may take up to the whole 160 KB, so it
  // cannot also have static LDS).
  extern __shared__ double sh[];
  const int K = p.K;
  double* Gs = sh;                               // [C's][C's]
  double* Ds = Gs + CSP * CSP;                   // [K][C's]
  double* bs = Ds + K * CSP;                     // [K][C's] b_k
  double* red = bs + K * CSP;                    // [threads] objective tree
  double* Aw = red + kUpdThreads;                // elimination storage (C'_s > 8)
  int* ns = reinterpret_cast<int*>(Aw + fit_solve_lds<CSP>() / sizeof(double));  // [K] |L_k|
  const int tid = threadIdx.x;
  const bool obj = first && objective;
  // the step kernel's block sums: thread strides, then a fixed tree (below)
  double os = 0.0;
  if (obj)
    for (int i0 = tid; i0 < nopart; i0 += 4 * kUpdThreads) {
      double v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = i0 + u * kUpdThreads < nopart ? opart[i0 + u * kUpdThreads] : 0.0;
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (i0 + u * kUpdThreads < nopart) os += v[u];
    }
  for (int i = tid; i < CSP * CSP; i += kUpdThreads) Gs[i] = G[(size_t)m * CSP * CSP + i];
  for (int i = tid; i < K * CSP; i += kUpdThreads) {
    Ds[i] = D64[(size_t)m * K * CSP + i];
    if (first) Dold[i] = Ds[i];
    double s = 0.0;
    for (int b0 = 0; b0 < nblk; b0 += 8) {  // blocks in order, 8 loads in flight
      double v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = b0 + u < nblk ? bins[(size_t)(b0 + u) * K * CSP + i] : 0.0;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (b0 + u < nblk) s += v[u];
    }
    bs[i] = s;
  }
  for (int k = tid; k < K; k += kUpdThreads) {
    int n = 0;
    for (int b0 = 0; b0 < nblk; b0 += 8) {
      int v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = b0 + u < nblk ? nbin[(size_t)(b0 + u) * K + k] : 0;
#pragma unroll
      for (int u = 0; u < 8; ++u) n += v[u];
    }
    ns[k] = n;
  }
  if (obj) red[tid] = os;
  __syncthreads();
  if (obj) {
    for (int h = kUpdThreads / 2; h > 0; h >>= 1) {
      if (tid < h) red[tid] += red[tid + h];
      __syncthreads();
    }
    if (tid == 0) *objective = red[0];
  }
  constexpr int SOLVERS = fit_solvers<CSP>();
  for (int k0 = 0; k0 < K; k0 += SOLVERS) {
    const int k = k0 + tid;
    if (tid < SOLVERS && k < K && ns[k] > 0) {
      double bk[CSP], x[CSP];
#pragma unroll
      for (int j = 0; j < CSP; ++j) bk[j] = bs[k * CSP + j];
      if constexpr (fit_solve_lds<CSP>() > 0) {
        solve_normal<CSP>(Gs, bk, Aw + (size_t)tid * CSP * CSP, x);
      } else {
        double A[CSP * CSP];
        solve_normal<CSP>(Gs, bk, A, x);
      }
#pragma unroll
      for (int j = 0; j < CSP; ++j) Ds[k * CSP + j] = x[j] / ns[k];
    }
  }
  __syncthreads();
  for (int k = tid; k < K; k += kUpdThreads) {  // D_k^T G D_k
    double s = 0.0;
#pragma unroll
    for (int i = 0; i < CSP; ++i) {
      double g = 0.0;
#pragma unroll
      for (int j = 0; j < CSP; ++j) g += Gs[i * CSP + j] * Ds[k * CSP + j];
      s += Ds[k * CSP + i] * g;
    }
    qv[k] = s;
  }
  for (int i = tid; i < K * CSP; i += kUpdThreads) D64[(size_t)m * K * CSP + i] = Ds[i];
}

// codebooks = fp32(D64), codes[c][m] = ct[m][c], and the final objective.
__global__ __launch_bounds__(kEcThreads) void ec_finish_kernel(const double* __restrict__ D64, EcParams p,
                                                             const uint8_t* __restrict__ ct,
                                                             float* __restrict__ D, uint8_t* __restrict__ codes,
                                                             const double* __restrict__ opart, int nopart,
                                                             double* __restrict__ objective) {
  const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x, stride = (size_t)gridDim.x * blockDim.x;
  const size_t nd = (size_t)p.M * p.K * p.Csp, nc = (size_t)p.M * p.Ct;
  for (size_t i = tid; i < nd; i += stride) D[i] = (float)D64[i];
  for (size_t i = tid; i < nc; i += stride) codes[i] = ct[(i % p.M) * p.Ct + i / p.M];
  if (tid == 0 && objective) {  // once per call: a serial sum is fine here
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
  b += cblocks * K * Csp * 8;                    // bins
  b += cblocks * K * 4;                          // nbin
  b += (size_t)Ct;                               // codes_old
  b += (size_t)M * Ct;                           // codes, [M][C_t]
  return b + 16 * 256;                           // each slice is rounded up to 256 bytes
}

template <int CSP>
hipError_t launch_ec_csp(int N, int Cs, int Ct, int M, int K, const float* S, const float* T, float* D,
                         uint8_t* codes, int sweeps, int inner, double* objective, hipStream_t stream) {
  constexpr int Csp = CSP;
  EcParams p{N, Cs, Ct, M, K, Csp, inner, ceil_div(N, kEcChunk)};
  const int cblocks = ceil_div(Ct, kEcThreads);
  const int nopart = cblocks * p.nchunks;
  Scratch scratch;
  hipError_t e = scratch.acquire(stream, ec_fc_workspace(N, Ct, M, K, Csp));
  if (e != hipSuccess) return e;
  auto step = ec_step_kernel<CSP>;
  auto reduce = ec_reduce_kernel<CSP>;
  auto fit = ec_fit_kernel<CSP>;
  const size_t step_lds = ((size_t)K * (Csp + 1) + kEcThreads / kWave) * sizeof(double);
  const size_t red_lds = ((size_t)Csp * kEcThreads + red_area(K, Csp)) * sizeof(double) + kEcThreads;
  const size_t fit_lds = fit_lds_bytes<CSP>(K);
  if (step_lds > kLdsBytes || red_lds > kLdsBytes || fit_lds > kLdsBytes) return hipErrorInvalidValue;
  if ((e = allow_max_lds((const void*)step)) != hipSuccess) return e;
  if ((e = allow_max_lds((const void*)reduce)) != hipSuccess) return e;
  if ((e = allow_max_lds((const void*)fit)) != hipSuccess) return e;
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
  double* bins = reinterpret_cast<double*>(take((size_t)cblocks * K * Csp * 8));
  int* nbin = reinterpret_cast<int*>(take((size_t)cblocks * K * 4));
  uint8_t* codes_old = reinterpret_cast<uint8_t*>(take((size_t)Ct));
  uint8_t* ct = reinterpret_cast<uint8_t*>(take((size_t)M * Ct));

  const size_t ninit = std::max<size_t>({(size_t)M * Ct, (size_t)M * K * Csp, (size_t)M * Csp * Csp});
  const unsigned iblocks = (unsigned)std::min<size_t>(8192, ceil_div_z(ninit, kEcThreads));
  hipLaunchKernelGGL(ec_init_kernel, dim3(iblocks), dim3(kEcThreads), 0, stream, S, D, (const uint8_t*)codes, p,
                     D64, ct, G);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const dim3 pgrid((unsigned)cblocks, (unsigned)p.nchunks);
  hipLaunchKernelGGL(ec_start_kernel<CSP>, pgrid, dim3(kEcThreads), 0, stream, S, T, p, (const double*)D64,
                     (const uint8_t*)ct, E, opart);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  int nstep = 0;
  int ma = -1;  // subspace fitted by the previous step, which the next step kernel finishes
  for (int s = 0; s < sweeps; ++s) {
    for (int m = 0; m < M; ++m, ++nstep) {
      hipLaunchKernelGGL(step, pgrid, dim3(kEcThreads), step_lds, stream, S, p, E, ma, (const double*)P,
                         (const double*)D64, (const double*)qv, ct, (const double*)Dold,
                         (const uint8_t*)codes_old, m, part, opart);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      for (int it = 0; it < inner; ++it) {
        hipLaunchKernelGGL(reduce, dim3((unsigned)cblocks), dim3(kEcThreads), red_lds, stream, (const double*)part,
                           p, m, (const double*)G, (const double*)D64, (const double*)qv, it == 0 ? 0 : 1, ct,
                           P, codes_old, bins, nbin);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        // objective[nstep] is the value before this step (after the previous one)
        hipLaunchKernelGGL(fit, dim3(1), dim3(kUpdThreads), fit_lds, stream, (const double*)bins,
                           (const int*)nbin, cblocks, p, m, (const double*)G, D64, it == 0 ? 1 : 0, Dold,
                           (const double*)opart, nopart, objective ? objective + nstep : nullptr, qv);
        if ((e = hipGetLastError()) != hipSuccess) return e;
      }
      ma = m;
    }
  }
  if (ma >= 0) {  // finish the last step and sum the final objective
    hipLaunchKernelGGL(step, pgrid, dim3(kEcThreads), step_lds, stream, S, p, E, ma, (const double*)P,
                       (const double*)D64, (const double*)qv, ct, (const double*)Dold, (const uint8_t*)codes_old,
                       -1, part, opart);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  hipLaunchKernelGGL(ec_finish_kernel, dim3(iblocks), dim3(kEcThreads), 0, stream, (const double*)D64, p,
                     (const uint8_t*)ct, D, codes, (const double*)opart, nopart,
                     objective ? objective + nstep : nullptr);
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
