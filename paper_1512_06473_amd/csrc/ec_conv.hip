// Error-corrected quantization of a convolutional layer.
//
// Paper: Sec. 3.3.2 (Eq. (13)) and App. B (Eq. (14)-(21)).  With the input
// maps S_n and desired responses T_n of N images, the sub-codebooks D^(m)
// (shared by every kernel position p) and the assignments k(c, p) minimise
// the response error by block coordinate descent over the subspaces; for
// subspace m, with R the residual of the other subspaces (Eq. (15)):
//   * sub-codewords k = 0 .. K-1 in order (Eq. (17)-(19)): D_k becomes the
//     least-squares fit, over images, output positions and channels, of the
//     residual without the other sub-codewords' terms;
//   * kernel positions p = 0 .. d_k^2 - 1 in order (Eq. (20)-(21)): each
//     channel takes the sub-codeword of least error for the residual without
//     the other positions' terms, tried exhaustively.
// Readings: Q_k of Eq. (18) takes out, per channel, the positions whose
// sub-codeword is not k, and Eq. (19) sums over the channels with a position
// on k; P of Eq. (20) takes out every other position p' (paired with its own
// input position); p_s = p_t s - pad + p (no flip), S = 0 outside the input;
// normal equations with the pivot rule of the FC case; ties to the lowest k.
//
// Both updates see the large arrays only through two small summaries of
// subspace m, with s_p(n, o) the input sub-vector that position p meets at
// output o of image n:
//   G[p][p'] = sum_{n,o} s_p s_p'^T          ([d_k^2][d_k^2][C'_s][C'_s], once)
//   H[c][p]  = sum_{n,o} s_p R(c)             ([C_t][d_k^2][C'_s], per step)
// Eq. (19) for k is then sum_{(c,p) on k} (sum_{p' on k} G[p][p']) D_k =
// sum_{(c,p) on k} (H[c][p] - sum_{p' not on k} G[p][p'] D_{k(c,p')}), and the
// error of Eq. (21) for (c, p) and candidate k is, up to a constant,
// D_k^T G[p][p] D_k - 2 D_k^T (H[c][p] - sum_{p' != p} G[p][p'] D_{k(c,p')}).
//
// State, float64: the residual of the whole layer E = T - Y [N][C_t][O]
// (O = H_o W_o), D64, G, and the codes as [M][C_t][d_k^2].  Per subspace:
//   ecc_apply_kernel  E -= the change of the subspace fitted before (from
//                     its delta[c][p] = D_new[k_new] - D_old[k_old]); block
//                     sums of E^2 (the objective after that step);
//   ecc_corr_kernel   partial sum_{n,o} s_p E(c) per chunk of images;
//   ecc_reduce_kernel H = the partials in chunk order + sum_p' G[p][p'] W(c, p')
//                     (so H is taken against R = E + this subspace's terms);
//   ecc_dupdate_kernel one workgroup: Eq. (17)-(19), the sub-codewords in
//                     order;
//   ecc_bupdate_kernel one wave per channel: Eq. (20)-(21), the positions in
//                     order; after the last of `inner` rounds, delta for the
//                     next apply.
#include "qcnn_internal.h"

namespace qcnn {
namespace {

constexpr int kCThreads = 256;

struct EccParams {
  int N, Cs, H, W, Ct, Ho, Wo, dk, stride, pad, M, K, Csp, P, O;
  int chunk, nchunks;  // images per correlation chunk, number of chunks
};

// Fixed-order sum of one value per thread into opart[block].
__device__ __forceinline__ void ecc_block_sum(double v, double* red, double* __restrict__ opart) {
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_down(v, off, kWave);
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int w = 0; w < kCThreads / kWave; ++w) s += red[w];
    opart[blockIdx.x] = s;
  }
}

// D64 = codebooks; ct[m][c][p] = codes[c][p][m] (codes >= K read as K - 1).
__global__ __launch_bounds__(kCThreads) void ecc_init_kernel(const float* __restrict__ D,
                                                           const uint8_t* __restrict__ codes, EccParams q,
                                                           double* __restrict__ D64, uint8_t* __restrict__ ct) {
  const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x, stride = (size_t)gridDim.x * blockDim.x;
  const size_t nd = (size_t)q.M * q.K * q.Csp, nc = (size_t)q.M * q.Ct * q.P;
  for (size_t i = tid; i < nd; i += stride) D64[i] = (double)D[i];
  for (size_t i = tid; i < nc; i += stride) {
    const size_t m = i / ((size_t)q.Ct * q.P), cp = i % ((size_t)q.Ct * q.P);
    const uint8_t k = codes[cp * q.M + m];
    ct[i] = k < q.K ? k : (uint8_t)(q.K - 1);
  }
}

// G[m][p][p'][i][j] = sum over n, o (in order) of s_p[i] s_p'[j].
__global__ __launch_bounds__(kCThreads) void ecc_gram_kernel(const float* __restrict__ S, EccParams q,
                                                           double* __restrict__ G) {
  const size_t i0 = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t per_m = (size_t)q.P * q.P * q.Csp * q.Csp;
  if (i0 >= (size_t)q.M * per_m) return;
  const int m = (int)(i0 / per_m);
  size_t r = i0 % per_m;
  const int j = (int)(r % q.Csp);
  r /= q.Csp;
  const int i = (int)(r % q.Csp);
  r /= q.Csp;
  const int p2 = (int)(r % q.P), p = (int)(r / q.P);
  // output positions whose two input positions both lie inside the input
  // (the others add exact zeros)
  const int ky = p / q.dk, kx = p - ky * q.dk, ky2 = p2 / q.dk, kx2 = p2 - ky2 * q.dk;
  const size_t HW = (size_t)q.H * q.W;
  double s = 0.0;
  for (int n = 0; n < q.N; ++n) {
    const float* si = S + ((size_t)n * q.Cs + (size_t)m * q.Csp + i) * HW;
    const float* sj = S + ((size_t)n * q.Cs + (size_t)m * q.Csp + j) * HW;
    for (int yo = 0; yo < q.Ho; ++yo) {
      const int y = yo * q.stride - q.pad + ky, y2 = yo * q.stride - q.pad + ky2;
      if ((unsigned)y >= (unsigned)q.H || (unsigned)y2 >= (unsigned)q.H) continue;
      for (int xo0 = 0; xo0 < q.Wo; xo0 += 8) {  // eight positions' loads in flight, added in order
        float a[8], b[8];
        bool ok[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int xo = xo0 + u;
          const int x = xo * q.stride - q.pad + kx, x2 = xo * q.stride - q.pad + kx2;
          ok[u] = xo < q.Wo && (unsigned)x < (unsigned)q.W && (unsigned)x2 < (unsigned)q.W;
          const float va = si[ok[u] ? y * q.W + x : 0], vb = sj[ok[u] ? y2 * q.W + x2 : 0];
          a[u] = va;
          b[u] = vb;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (ok[u]) s += (double)a[u] * (double)b[u];
      }
    }
  }
  G[i0] = s;
}

// E = T - sum_m sum_p D^(m)[k(c, p)]^T s_p as a float64 implicit GEMM on
// MFMA (v_mfma_f64_16x16x4_f64): rows are the output channels, columns the
// output positions of all images (g = n O + o), and the reduction runs over
// (kernel position p, input channel cs), p outer, so that a stage of
// kStartKB reduction indices mostly shares one p.  A workgroup of 4 waves
// owns 64 channels x 64 columns, wave w the channels 16 w .. 16 w + 15 as
// four 16 x 16 tiles.  Each thread loads its share of a stage (the decoded
// weights D^(m)[k(c, p)][a], cs = m C's + a: code, then sub-codeword entry;
// the input values, 0 outside the map) one stage ahead into registers,
// stores them into one of two LDS buffers, and every wave runs the stage's
// MFMAs from LDS.  Register i of lane l of a 16 x 16 f64 result holds row
// 4 i + l / 16, column l % 16.  Block sums of E^2 into
// opart[blockIdx.y gridDim.x + blockIdx.x].
constexpr int kStartTile = 64;          // channels and columns per workgroup
constexpr int kStartKB = 32;            // reduction indices per stage
constexpr int kStartLd = kStartKB + 1;  // LDS row stride in doubles (odd: spreads the rows over the banks)
typedef double d4v __attribute__((ext_vector_type(4)));

template <int CSP>
__global__ __launch_bounds__(kCThreads) void ecc_start_kernel(const float* __restrict__ S,
                                                            const float* __restrict__ T, EccParams q,
                                                            const double* __restrict__ D64,
                                                            const uint8_t* __restrict__ ct, double* __restrict__ E,
                                                            double* __restrict__ opart) {
  static_assert(kCThreads == 256, "four waves, 8 values per thread and operand");
  __shared__ double As[2][kStartTile * kStartLd];  // [channel][index]
  __shared__ double Bs[2][kStartTile * kStartLd];  // [column][index]
  __shared__ double red[kCThreads / kWave];
  constexpr int PER = kStartTile * kStartKB / kCThreads;  // 8
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int c0 = blockIdx.x * kStartTile, g0 = blockIdx.y * kStartTile;
  const int ncol = q.N * q.O, KD = q.Cs * q.P;
  // this thread's share of a stage: row r (channel c0 + r of the weights,
  // column g0 + r of the inputs), reduction indices q0 .. q0 + PER - 1
  const int r = tid / (kStartKB / PER), q0 = (tid % (kStartKB / PER)) * PER;
  const int cw = c0 + r, gb = g0 + r;
  const bool rowa = cw < q.Ct, rowb = gb < ncol;
  const int nb = rowb ? gb / q.O : 0, ob = rowb ? gb - (gb / q.O) * q.O : 0;
  const int yb = (ob / q.Wo) * q.stride - q.pad, xb = (ob - (ob / q.Wo) * q.Wo) * q.stride - q.pad;
  const size_t HW = (size_t)q.H * q.W;
  const float* sb = S + (size_t)nb * q.Cs * HW;
  const int nst = (KD + kStartKB - 1) / kStartKB;
  float sv[PER];
  double wv[PER];
  auto load_stage = [&](int st) {
    const int k0 = st * kStartKB + q0;
    int p = k0 / q.Cs, cs = k0 - p * q.Cs;
    int code[PER], ma[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const bool okk = p < q.P;
      const int pp = okk ? p : 0, cc = okk ? cs : 0;
      const int ky = pp / q.dk, kx = pp - ky * q.dk;
      const int y = yb + ky, x = xb + kx;
      const bool oks = rowb && okk && (unsigned)y < (unsigned)q.H && (unsigned)x < (unsigned)q.W;
      const float v = sb[oks ? cc * HW + (size_t)y * q.W + x : 0];
      sv[i] = oks ? v : 0.f;
      const int m = cc / CSP;
      const bool okw = rowa && okk;
      const int cd = ct[okw ? ((size_t)m * q.Ct + cw) * q.P + pp : 0];
      code[i] = cd;
      ma[i] = okw ? (m * q.K) * CSP + (cc - m * CSP) : -1;
      if (++cs == q.Cs) {
        cs = 0;
        ++p;
      }
    }
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const double w = D64[ma[i] >= 0 ? ma[i] + (size_t)code[i] * CSP : 0];
      wv[i] = ma[i] >= 0 ? w : 0.0;
    }
  };
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      As[buf][r * kStartLd + q0 + i] = wv[i];
      Bs[buf][r * kStartLd + q0 + i] = (double)sv[i];
    }
  };
  d4v acc[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) acc[t] = d4v{0.0, 0.0, 0.0, 0.0};
  const int arow = 16 * wave + (lane & 15), kq = lane >> 4;
  load_stage(0);
  for (int st = 0; st < nst; ++st) {
    const int buf = st & 1;
    store_stage(buf);
    __syncthreads();  // the stage is in LDS; the other buffer's readers (stage st - 1) are done
    if (st + 1 < nst) load_stage(st + 1);
#pragma unroll
    for (int kk = 0; kk < kStartKB / 4; ++kk) {
      const double av = As[buf][arow * kStartLd + 4 * kk + kq];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const double bv = Bs[buf][(16 * t + (lane & 15)) * kStartLd + 4 * kk + kq];
        acc[t] = __builtin_amdgcn_mfma_f64_16x16x4f64(av, bv, acc[t], 0, 0, 0);
      }
    }
  }
  // acc[t][i]: channel c0 + 16 wave + 4 i + lane / 16, column g0 + 16 t + lane % 16
  double sq = 0.0;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int g = g0 + 16 * t + (lane & 15);
    const int n = g / q.O, o = g - (g / q.O) * q.O;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = c0 + 16 * wave + 4 * i + kq;
      if (g < ncol && c < q.Ct) {
        const size_t at = ((size_t)n * q.Ct + c) * q.O + o;
        const double e = (double)T[at] - acc[t][i];
        E[at] = e;
        sq += e * e;
      }
    }
  }
  for (int off = kWave / 2; off > 0; off >>= 1) sq += __shfl_down(sq, off, kWave);
  if (lane == 0) red[wave] = sq;
  __syncthreads();
  if (tid == 0) {
    double s2 = 0.0;
    for (int w = 0; w < kCThreads / kWave; ++w) s2 += red[w];
    opart[(size_t)blockIdx.y * gridDim.x + blockIdx.x] = s2;
  }
}

// E -= sum_p delta[c][p]^T s_p for subspace ma; block sums of E^2.
template <int CSP>
__global__ __launch_bounds__(kCThreads) void ecc_apply_kernel(const float* __restrict__ S, EccParams q, int ma,
                                                            const double* __restrict__ delta,
                                                            double* __restrict__ E, double* __restrict__ opart) {
  __shared__ double red[kCThreads / kWave];
  const size_t i = (size_t)blockIdx.x * kCThreads + threadIdx.x;
  const size_t total = (size_t)q.N * q.Ct * q.O;
  double e = 0.0;
  if (i < total) {
    const int o = (int)(i % q.O);
    const int c = (int)((i / q.O) % q.Ct);
    const int n = (int)(i / ((size_t)q.O * q.Ct));
    e = E[i];
    const int yo = o / q.Wo, xo = o - yo * q.Wo;
    const size_t HW = (size_t)q.H * q.W;
    const float* sn = S + ((size_t)n * q.Cs + (size_t)ma * CSP) * HW;
    const double* dl = delta + (size_t)c * q.P * CSP;
    double d = 0.0;  // positions outside the input add exact zeros: skipped
    for (int ky = 0; ky < q.dk; ++ky) {
      const int y = yo * q.stride - q.pad + ky;
      if ((unsigned)y >= (unsigned)q.H) continue;
      for (int kx = 0; kx < q.dk; ++kx) {
        const int x = xo * q.stride - q.pad + kx;
        if ((unsigned)x >= (unsigned)q.W) continue;
        const double* dp = dl + (ky * q.dk + kx) * CSP;
#pragma unroll
        for (int j = 0; j < CSP; ++j) d += (double)sn[j * HW + (size_t)y * q.W + x] * dp[j];
      }
    }
    e -= d;
    E[i] = e;
  }
  ecc_block_sum(e * e, red, opart);
}

// part[chunk][c][p][j] = sum over the chunk's images and all o (in order) of
// s_p[j] E(c), for subspace m; one (c, p) per thread.
template <int CSP>
__global__ __launch_bounds__(kCThreads) void ecc_corr_kernel(const float* __restrict__ S, EccParams q, int m,
                                                           const double* __restrict__ E,
                                                           double* __restrict__ part) {
  const int i = blockIdx.x * kCThreads + threadIdx.x;
  if (i >= q.Ct * q.P) return;
  const int c = i / q.P, p = i - c * q.P;
  const int n0 = blockIdx.y * q.chunk, n1 = min(q.N, n0 + q.chunk);
  double acc[CSP];
#pragma unroll
  for (int j = 0; j < CSP; ++j) acc[j] = 0.0;
  const int ky = p / q.dk, kx = p - ky * q.dk;
  const size_t HW = (size_t)q.H * q.W;
  for (int n = n0; n < n1; ++n) {
    const double* er = E + ((size_t)n * q.Ct + c) * q.O;
    const float* sn = S + ((size_t)n * q.Cs + (size_t)m * CSP) * HW;
    for (int yo = 0; yo < q.Ho; ++yo) {
      const int y = yo * q.stride - q.pad + ky;
      if ((unsigned)y >= (unsigned)q.H) continue;  // exact zeros: skipped
      const double* erow = er + (size_t)yo * q.Wo;
      const float* srow = sn + (size_t)y * q.W;
#pragma unroll 4
      for (int xo = 0; xo < q.Wo; ++xo) {
        const int x = xo * q.stride - q.pad + kx;
        if ((unsigned)x >= (unsigned)q.W) continue;
        const double e = erow[xo];
#pragma unroll
        for (int j = 0; j < CSP; ++j) acc[j] += (double)srow[j * HW + x] * e;
      }
    }
  }
  double* dst = part + (((size_t)blockIdx.y * q.Ct + c) * q.P + p) * CSP;
#pragma unroll
  for (int j = 0; j < CSP; ++j) dst[j] = acc[j];
}

// H[c][p][j] = sum over chunks (in order) of part + sum_p' sum_i G[p][p'][j][i] W(c, p')[i].
template <int CSP>
__global__ __launch_bounds__(kCThreads) void ecc_reduce_kernel(const double* __restrict__ part, EccParams q, int m,
                                                             const double* __restrict__ G,
                                                             const double* __restrict__ D64,
                                                             const uint8_t* __restrict__ ct,
                                                             double* __restrict__ H) {
  const int i = blockIdx.x * kCThreads + threadIdx.x;
  if (i >= q.Ct * q.P) return;
  const int c = i / q.P, p = i - c * q.P;
  double h[CSP];
#pragma unroll
  for (int j = 0; j < CSP; ++j) h[j] = 0.0;
  for (int ch = 0; ch < q.nchunks; ++ch) {
    const double* src = part + ((size_t)ch * q.Ct * q.P + i) * CSP;
#pragma unroll
    for (int j = 0; j < CSP; ++j) h[j] += src[j];
  }
  const double* Gp = G + ((size_t)m * q.P + p) * q.P * CSP * CSP;
  const uint8_t* km = ct + ((size_t)m * q.Ct + c) * q.P;
  for (int p2 = 0; p2 < q.P; ++p2) {
    const double* w = D64 + ((size_t)m * q.K + km[p2]) * CSP;
    const double* g = Gp + (size_t)p2 * CSP * CSP;
#pragma unroll
    for (int j = 0; j < CSP; ++j)
#pragma unroll
      for (int i2 = 0; i2 < CSP; ++i2) h[j] += g[j * CSP + i2] * w[i2];
  }
#pragma unroll
  for (int j = 0; j < CSP; ++j) H[(size_t)i * CSP + j] = h[j];
}

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  __builtin_amdgcn_wave_barrier();
}

// x with A x = b for the normal matrix A of Eq. (19): elimination in channel
// order without row exchanges, one reciprocal per pivot; a pivot <= 1e-12 x
// the largest diagonal entry (or <= 0) drops that coordinate (x = 0).  A is
// read only; W is N x N working storage of the calling lane.
template <int N>
__device__ __forceinline__ void solve_rcp(const double* __restrict__ A, const double (&bin)[N], double* W,
                                          double (&x)[N]) {
  double y[N], inv[N];
  bool live[N];
  double scale = 0.0;
#pragma unroll
  for (int i = 0; i < N; ++i) {
#pragma unroll
    for (int j = 0; j < N; ++j) W[i * N + j] = A[i * N + j];
    y[i] = bin[i];
    scale = fmax(scale, A[i * N + i]);
  }
#pragma unroll
  for (int j = 0; j < N; ++j) {
    live[j] = W[j * N + j] > 1e-12 * scale && W[j * N + j] > 0.0;
    inv[j] = live[j] ? 1.0 / W[j * N + j] : 0.0;
    if (live[j]) {
#pragma unroll
      for (int i = j + 1; i < N; ++i) {
        const double f = W[i * N + j] * inv[j];
#pragma unroll
        for (int c = j; c < N; ++c) W[i * N + c] -= f * W[j * N + c];
        y[i] -= f * y[j];
      }
    }
  }
#pragma unroll
  for (int j = N - 1; j >= 0; --j) {
    double s = y[j];
#pragma unroll
    for (int i = j + 1; i < N; ++i)
      if (live[i]) s -= W[j * N + i] * x[i];
    x[j] = live[j] ? s * inv[j] : 0.0;
  }
}

// Bytes of the D-update kernel's LDS, with (gl) or without the Gram blocks.
template <int CSP> size_t solve_lds_bytes(int K, int npairs, int P, bool gl) {
  constexpr int QS = kWave / CSP;
  const size_t dbl = (size_t)2 * K * CSP + kCThreads + (size_t)(kCThreads / kWave) * QS * CSP * (CSP + 1) +
                     (size_t)(kCThreads / kWave) * CSP * (CSP + 1) + (gl ? (size_t)P * P * CSP * CSP : 0);
  const size_t ints = 3 * 256 + (kCThreads / kWave) * 256;
  return dbl * 8 + ints * 4 + (size_t)npairs * 2 + (size_t)npairs;
}

// Eq. (17)-(19), one workgroup: the sub-codewords in order.  On the first
// round of a step (`first`) it also records the objective before the step
// (from the apply kernel's block sums) and keeps the subspace's sub-codebook
// and codes as they were (Dold, cold) for delta.  At the end it stores
// qkg[p][k] = D_k^T G[p][p] D_k for the assignment kernel.  GL: the
// subspace's Gram blocks are staged in LDS.
template <int CSP, bool GL>
__global__ __launch_bounds__(kCThreads) void ecc_dupdate_kernel(const double* __restrict__ H, EccParams q, int m,
                                                              const double* __restrict__ G, double* __restrict__ D64,
                                                              const uint8_t* __restrict__ ct, int first,
                                                              double* __restrict__ Dold, uint8_t* __restrict__ cold,
                                                              double* __restrict__ qkg,
                                                              const double* __restrict__ opart, int nopart,
                                                              double* __restrict__ objective) {
  extern __shared__ double sh[];
  constexpr int NW = kCThreads / kWave;
  constexpr int QS = kWave / CSP;               // pair slots per wave
  constexpr int NE = CSP * (CSP + 1);           // entries of [rhs | normal matrix]
  const int K = q.K, P = q.P, Ct = q.Ct, npairs = Ct * P;
  double* Ds = sh;                              // [K][C's] current sub-codewords
  double* hs = Ds + K * CSP;                    // [K][C's] sums of H over each sub-codeword's pairs
  double* red = hs + K * CSP;                   // [256]
  double* wred = red + kCThreads;               // [4][QS][C's][C's + 1] slot partials
  double* wpart = wred + NW * QS * NE;          // [4][C's][C's + 1] wave partials
  double* Gl = wpart + NW * NE;                 // [P][P][C's][C's] (GL)
  int* cnt = reinterpret_cast<int*>(Gl + (GL ? (size_t)P * P * CSP * CSP : 0));  // [256]
  int* start = cnt + 256;                       // [256]
  int* run = start + 256;                       // [256]
  int* wcnt = run + 256;                        // [4][256]
  uint16_t* list = reinterpret_cast<uint16_t*>(wcnt + NW * 256);  // pairs by code
  uint8_t* cs = reinterpret_cast<uint8_t*>(list + npairs);        // [C_t][P] codes
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const double* Gg = G + (size_t)m * P * P * CSP * CSP;
  const double* Gm = GL ? Gl : Gg;

  const bool obj = first && objective;
  double os = 0.0;
  if (obj)
    for (int i = tid; i < nopart; i += kCThreads) os += opart[i];
  for (int i = tid; i < K * CSP; i += kCThreads) {
    Ds[i] = D64[(size_t)m * K * CSP + i];
    if (first) Dold[i] = Ds[i];
  }
  for (int i = tid; i < npairs; i += kCThreads) {
    cs[i] = ct[(size_t)m * npairs + i];
    if (first) cold[i] = cs[i];
  }
  if (GL)
    for (int i = tid; i < P * P * CSP * CSP; i += kCThreads) Gl[i] = Gg[i];
  if (obj) {
    red[tid] = os;
    __syncthreads();
    for (int h = kCThreads / 2; h > 0; h >>= 1) {
      if (tid < h) red[tid] += red[tid + h];
      __syncthreads();
    }
    if (tid == 0) *objective = red[0];
  }
  __syncthreads();

  {
    // ---- the (c, p) pairs sorted stably by code: list[start[k] ..]
    for (int k = tid; k < 256; k += kCThreads) cnt[k] = run[k] = 0;
    for (int k = tid; k < NW * 256; k += kCThreads) wcnt[k] = 0;
    __syncthreads();
    for (int i = tid; i < npairs; i += kCThreads) atomicAdd(&cnt[cs[i]], 1);  // counts: order-free
    __syncthreads();
    if (tid == 0) {
      int s = 0;
      for (int k = 0; k < 256; ++k) {
        start[k] = s;
        s += cnt[k];
      }
    }
    __syncthreads();
    for (int r0 = 0; r0 < npairs; r0 += kCThreads) {
      const int i = r0 + tid;
      const bool valid = i < npairs;
      const uint32_t c = valid ? cs[i] : 0u;
      uint64_t same = __ballot(valid);
#pragma unroll
      for (int b = 0; b < 8; ++b) {
        const uint64_t ones = __ballot(valid && ((c >> b) & 1u));
        same &= ((c >> b) & 1u) ? ones : ~ones;
      }
      const int below = __popcll(same & ((1ull << lane) - 1ull));
      if (valid && below == 0) wcnt[wave * 256 + c] = __popcll(same);
      __syncthreads();
      if (valid) {
        int off = start[c] + run[c] + below;
        for (int w = 0; w < wave; ++w) off += wcnt[w * 256 + c];
        list[off] = (uint16_t)i;
      }
      __syncthreads();
      for (int k = tid; k < 256; k += kCThreads) {
        int add = 0;
        for (int w = 0; w < NW; ++w) {
          add += wcnt[w * 256 + k];
          wcnt[w * 256 + k] = 0;
        }
        run[k] += add;
      }
      __syncthreads();
    }

    // the H part of each sub-codeword's right-hand side (it does not depend
    // on the sub-codewords), its pairs in list order
    for (int e = tid; e < K * CSP; e += kCThreads) {
      const int k = e / CSP, j = e - k * CSP;
      const int s0 = start[k], n_k = cnt[k];
      double v = 0.0;
      for (int r0 = 0; r0 < n_k; r0 += 4) {
        double h[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) h[u] = r0 + u < n_k ? H[(size_t)list[s0 + r0 + u] * CSP + j] : 0.0;
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (r0 + u < n_k) v += h[u];
      }
      hs[e] = v;
    }
    __syncthreads();

    // ---- Eq. (17)-(19): sub-codewords in order.  Pair slot g = wave QS +
    // lane / C's takes pairs g, g + 4 QS, ... of the sub-codeword's list;
    // lane % C's is its row j of [rhs | normal matrix].  Slot sums are added
    // within each wave (a fixed shuffle tree, or in slot order when C's does
    // not divide 64), then the waves in order.
    {
      const int slot = lane / CSP, j = lane - slot * CSP;
      const bool act = slot < QS;
      const int g0 = wave * QS + slot;
      for (int k = 0; k < K; ++k) {
        const int n_k = cnt[k];  // uniform
        if (n_k == 0) continue;  // unused: keeps its value
        double rhs = 0.0, mat[CSP];
#pragma unroll
        for (int i = 0; i < CSP; ++i) mat[i] = 0.0;
        if (act) {
          for (int r = g0; r < n_k; r += NW * QS) {
            const int pr = list[start[k] + r];
            const int c = pr / P, p = pr - c * P;
            const uint8_t* kc = cs + c * P;
            const double* grow = Gm + ((size_t)p * P * CSP + j) * CSP;  // G[p][p2][j][.] at p2 * C's^2
            constexpr int PB = CSP <= 4 ? 9 : 5;  // positions whose loads are in flight together
            for (int p0 = 0; p0 < P; p0 += PB) {
              int k2[PB];
#pragma unroll
              for (int u = 0; u < PB; ++u) k2[u] = p0 + u < P ? kc[p0 + u] : 0;
              double gv[PB][CSP], dv[PB][CSP];
#pragma unroll
              for (int u = 0; u < PB; ++u)
#pragma unroll
                for (int i = 0; i < CSP; ++i) {
                  gv[u][i] = p0 + u < P ? grow[(size_t)(p0 + u) * CSP * CSP + i] : 0.0;
                  dv[u][i] = Ds[k2[u] * CSP + i];
                }
#pragma unroll
              for (int u = 0; u < PB; ++u) {
                if (p0 + u < P) {
                  const bool on = k2[u] == k;
                  double t = 0.0;
#pragma unroll
                  for (int i = 0; i < CSP; ++i) {
                    t += gv[u][i] * dv[u][i];
                    mat[i] += on ? gv[u][i] : 0.0;
                  }
                  rhs -= on ? 0.0 : t;
                }
              }
            }
          }
          if constexpr (QS * CSP != kWave) {
            double* w = wred + ((size_t)(wave * QS + slot) * CSP + j) * (CSP + 1);
            w[0] = rhs;
#pragma unroll
            for (int i = 0; i < CSP; ++i) w[1 + i] = mat[i];
          }
        }
        if constexpr (QS * CSP == kWave) {
          // C's divides 64: the slots' sums by a fixed shuffle tree over the
          // lanes of one row (stride C's); slot 0 then holds the wave's sums
          double vals[CSP + 1];
          vals[0] = rhs;
#pragma unroll
          for (int i = 0; i < CSP; ++i) vals[1 + i] = mat[i];
#pragma unroll
          for (int off = kWave / 2; off >= CSP; off >>= 1)
#pragma unroll
            for (int e = 0; e <= CSP; ++e) vals[e] += __shfl_down(vals[e], off, kWave);
          if (slot == 0)
#pragma unroll
            for (int e = 0; e <= CSP; ++e) wpart[wave * NE + j * (CSP + 1) + e] = vals[e];
        } else {
          wave_sync_lds();
          // this wave's slots, in order
          const int used = max(0, min(QS, n_k - wave * QS));
          for (int e = lane; e < NE; e += kWave) {
            double v = 0.0;
            for (int s0 = 0; s0 < used; s0 += 4) {
              double w4[4];
#pragma unroll
              for (int u = 0; u < 4; ++u) w4[u] = s0 + u < used ? wred[(size_t)(wave * QS + s0 + u) * NE + e] : 0.0;
#pragma unroll
              for (int u = 0; u < 4; ++u)
                if (s0 + u < used) v += w4[u];
            }
            wpart[wave * NE + e] = v;
          }
        }
        __syncthreads();
        if (wave == 0) {
          double* rb = red;        // [C's] rhs
          double* rA = red + CSP;  // [C's][C's] normal matrix
          for (int e = lane; e < NE; e += kWave) {
            double v = 0.0;
#pragma unroll
            for (int w = 0; w < NW; ++w) v += wpart[w * NE + e];
            const int jr = e / (CSP + 1), col = e - jr * (CSP + 1);
            if (col == 0)
              rb[jr] = v;
            else
              rA[jr * CSP + col - 1] = v;
          }
          wave_sync_lds();
          if (lane == 0) {
            double b[CSP], x[CSP], Aw[CSP * CSP];
#pragma unroll
            for (int r = 0; r < CSP; ++r) b[r] = hs[k * CSP + r] + rb[r];
            solve_rcp<CSP>(rA, b, Aw, x);
#pragma unroll
            for (int r = 0; r < CSP; ++r) Ds[k * CSP + r] = x[r];
          }
        }
        __syncthreads();
      }
    }

  }

  for (int i = tid; i < K * CSP; i += kCThreads) D64[(size_t)m * K * CSP + i] = Ds[i];
  for (int e = tid; e < P * K; e += kCThreads) {  // D_k^T G[p][p] D_k
    const int p = e / K, k = e - p * K;
    const double* Gpp = Gm + ((size_t)p * P + p) * CSP * CSP;
    double s2 = 0.0;
#pragma unroll
    for (int r = 0; r < CSP; ++r) {
      double g = 0.0;
#pragma unroll
      for (int i = 0; i < CSP; ++i) g += Gpp[r * CSP + i] * Ds[k * CSP + i];
      s2 += Ds[k * CSP + r] * g;
    }
    qkg[e] = s2;
  }
}

// Eq. (20)-(21): one wave per output channel c, the kernel positions in
// order.  For position p, b = H[c][p] - sum_{p' != p} G[p][p'] D_{k(c,p')}
// (lanes take (p', row) terms; the rows are added over p' in a fixed order),
// then lane l tries candidates l, l + 64, ... and the wave keeps the first
// minimum of qkg[p][k] - 2 D_k^T b (ties to the lowest k).  On the last round
// it also writes delta[c][p] = D_{k_new} - Dold_{k_old}.
template <int CSP>
__global__ __launch_bounds__(kCThreads) void ecc_bupdate_kernel(const double* __restrict__ H, EccParams q, int m,
                                                              const double* __restrict__ G,
                                                              const double* __restrict__ D64,
                                                              const double* __restrict__ qkg,
                                                              uint8_t* __restrict__ ct,
                                                              const double* __restrict__ Dold,
                                                              const uint8_t* __restrict__ cold,
                                                              double* __restrict__ delta, int last) {
  extern __shared__ double sb[];
  constexpr int NW = kCThreads / kWave;
  constexpr int QS = kWave / CSP;
  const int K = q.K, P = q.P;
  double* Ds = sb;                                   // [K][C's]
  double* part = Ds + K * CSP;                       // [4][QS][C's] row partials per wave
  double* bb = part + NW * QS * CSP;                 // [4][C's]
  uint8_t* kc = reinterpret_cast<uint8_t*>(bb + NW * CSP);  // [4][P] this wave's codes
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  for (int i = tid; i < K * CSP; i += kCThreads) Ds[i] = D64[(size_t)m * K * CSP + i];
  const int c = blockIdx.x * NW + wave;
  const bool col = c < q.Ct;
  uint8_t* kw = kc + wave * P;
  if (col)
    for (int p = lane; p < P; p += kWave) kw[p] = ct[((size_t)m * q.Ct + c) * P + p];
  __syncthreads();
  if (!col) return;  // no barriers below
  const double* Gg = G + (size_t)m * P * P * CSP * CSP;
  const int g = lane / CSP, j = lane - g * CSP;
  for (int p = 0; p < P; ++p) {
    // row j of sum_{p' != p} G[p][p'] D_{k(c,p')}: group g takes p' = g, g + QS, ...
    double t = 0.0;
    if (g < QS) {
      for (int p2 = g; p2 < P; p2 += QS) {
        if (p2 == p) continue;
        const double* gr = Gg + (((size_t)p * P + p2) * CSP + j) * CSP;
        const double* dk = Ds + kw[p2] * CSP;
#pragma unroll
        for (int i = 0; i < CSP; ++i) t += gr[i] * dk[i];
      }
      part[(wave * QS + g) * CSP + j] = t;
    }
    wave_sync_lds();
    if (lane < CSP) {
      double v = H[(((size_t)c * P + p) * CSP) + lane];
      double sub = 0.0;
      for (int g2 = 0; g2 < QS; ++g2) sub += part[(wave * QS + g2) * CSP + lane];
      bb[wave * CSP + lane] = v - sub;
    }
    wave_sync_lds();
    double b[CSP];
#pragma unroll
    for (int r = 0; r < CSP; ++r) b[r] = bb[wave * CSP + r];
    // this lane's candidates, then the wave's first minimum
    int best = -1;
    double bv = 0.0;
    const double* qp = qkg + (size_t)p * K;
    for (int k = lane; k < K; k += kWave) {
      double d = 0.0;
#pragma unroll
      for (int r = 0; r < CSP; ++r) d += Ds[k * CSP + r] * b[r];
      const double v = qp[k] - 2.0 * d;
      if (best < 0 || v < bv) {
        bv = v;
        best = k;
      }
    }
    for (int off = kWave / 2; off > 0; off >>= 1) {
      const double ov = __shfl_down(bv, off, kWave);
      const int ok = __shfl_down(best, off, kWave);
      if (ok >= 0 && (best < 0 || ov < bv || (ov == bv && ok < best))) {
        bv = ov;
        best = ok;
      }
    }
    best = __shfl(best, 0, kWave);
    if (lane == 0) kw[p] = (uint8_t)best;
    wave_sync_lds();
  }
  for (int p = lane; p < P; p += kWave) {
    const size_t i = (size_t)c * P + p;
    ct[(size_t)m * q.Ct * P + i] = kw[p];
    if (last)
#pragma unroll
      for (int r = 0; r < CSP; ++r) delta[i * CSP + r] = Ds[kw[p] * CSP + r] - Dold[cold[i] * CSP + r];
  }
}

// codebooks = fp32(D64), codes[c][p][m] = ct[m][c][p], and the final objective.
__global__ __launch_bounds__(kCThreads) void ecc_finish_kernel(const double* __restrict__ D64, EccParams q,
                                                             const uint8_t* __restrict__ ct,
                                                             float* __restrict__ D, uint8_t* __restrict__ codes,
                                                             const double* __restrict__ opart, int nopart,
                                                             double* __restrict__ objective) {
  const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x, stride = (size_t)gridDim.x * blockDim.x;
  const size_t nd = (size_t)q.M * q.K * q.Csp, nc = (size_t)q.M * q.Ct * q.P;
  for (size_t i = tid; i < nd; i += stride) D[i] = (float)D64[i];
  for (size_t i = tid; i < nc; i += stride) {  // i = (c P + p) M + m
    const size_t m = i % q.M, cp = i / q.M;
    codes[i] = ct[m * q.Ct * q.P + cp];
  }
  if (objective && blockIdx.x == 0) {  // the block sums in a fixed order: strided per thread, then a tree
    __shared__ double red[kCThreads];
    double s = 0.0;
    for (int b = threadIdx.x; b < nopart; b += kCThreads) s += opart[b];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int h = kCThreads / 2; h > 0; h >>= 1) {
      if ((int)threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
      __syncthreads();
    }
    if (threadIdx.x == 0) *objective = red[0];
  }
}

EccParams make_params(int N, int Cs, int H, int W, int Ct, int dk, int stride, int pad, int M, int K, int Csp) {
  EccParams q{};
  q.N = N, q.Cs = Cs, q.H = H, q.W = W, q.Ct = Ct, q.dk = dk, q.stride = stride, q.pad = pad;
  q.Ho = (H + 2 * pad - dk) / stride + 1;
  q.Wo = (W + 2 * pad - dk) / stride + 1;
  q.M = M, q.K = K, q.Csp = Csp, q.P = dk * dk, q.O = q.Ho * q.Wo;
  // about 256 Ki correlation threads: (c, p) pairs times image chunks
  const int pairs = Ct * q.P;
  const int want = std::max(1, std::min(N, 262144 / std::max(1, pairs)));
  q.chunk = ceil_div(N, want);
  q.nchunks = ceil_div(N, q.chunk);
  return q;
}

}  // namespace

template <int CSP>
hipError_t launch_ecc_csp(const EccParams& q, const float* S, const float* T, float* D, uint8_t* codes, int sweeps,
                          int inner, double* objective, hipStream_t stream) {
  const size_t total = (size_t)q.N * q.Ct * q.O;
  const int npairs = q.Ct * q.P;
  const int eblocks = (int)ceil_div_z(total, kCThreads);
  const unsigned sbx = (unsigned)ceil_div(q.Ct, kStartTile), sby = (unsigned)ceil_div_z((size_t)q.N * q.O, kStartTile);
  const int sblocks = (int)(sbx * sby);  // the starting residual's block sums
  const int pblocks = ceil_div(npairs, kCThreads);
  // the Gram blocks go to LDS when they fit beside the rest
  const bool gl = solve_lds_bytes<CSP>(q.K, npairs, q.P, true) <= kLdsBytes;
  const size_t slds = solve_lds_bytes<CSP>(q.K, npairs, q.P, gl);
  constexpr int NW = kCThreads / kWave;
  const size_t blds = ((size_t)q.K * CSP + NW * (kWave / CSP) * CSP + NW * CSP) * 8 + (size_t)NW * q.P;
  if (slds > kLdsBytes || blds > kLdsBytes) return hipErrorInvalidValue;
  auto dupdate = gl ? ecc_dupdate_kernel<CSP, true> : ecc_dupdate_kernel<CSP, false>;
  auto bupdate = ecc_bupdate_kernel<CSP>;
  hipError_t e = allow_max_lds((const void*)dupdate);
  if (e != hipSuccess) return e;
  if ((e = allow_max_lds((const void*)bupdate)) != hipSuccess) return e;
  Scratch scratch;
  size_t bytes = 0;
  const size_t szE = total * 8, szPart = (size_t)q.nchunks * npairs * CSP * 8, szH = (size_t)npairs * CSP * 8;
  const size_t szG = (size_t)q.M * q.P * q.P * CSP * CSP * 8, szD = (size_t)q.M * q.K * CSP * 8;
  const size_t szDelta = (size_t)npairs * CSP * 8, szOp = (size_t)std::max(eblocks, sblocks) * 8, szCt = (size_t)q.M * npairs;
  const size_t szDold = (size_t)q.K * CSP * 8, szCold = (size_t)npairs, szQk = (size_t)q.P * q.K * 8;
  for (size_t b : {szE, szPart, szH, szG, szD, szDelta, szOp, szCt, szDold, szCold, szQk})
    bytes += (b + 255) & ~(size_t)255;
  if ((e = scratch.acquire(stream, bytes)) != hipSuccess) return e;
  char* w = scratch.get();
  auto take = [&](size_t b) {
    char* r = w;
    w += (b + 255) & ~(size_t)255;
    return r;
  };
  double* E = reinterpret_cast<double*>(take(szE));
  double* part = reinterpret_cast<double*>(take(szPart));
  double* Hs = reinterpret_cast<double*>(take(szH));
  double* G = reinterpret_cast<double*>(take(szG));
  double* D64 = reinterpret_cast<double*>(take(szD));
  double* delta = reinterpret_cast<double*>(take(szDelta));
  double* opart = reinterpret_cast<double*>(take(szOp));
  uint8_t* ct = reinterpret_cast<uint8_t*>(take(szCt));
  double* Dold = reinterpret_cast<double*>(take(szDold));
  uint8_t* cold = reinterpret_cast<uint8_t*>(take(szCold));
  double* qkg = reinterpret_cast<double*>(take(szQk));

  const size_t ninit = std::max((size_t)q.M * q.K * CSP, (size_t)q.M * npairs);
  const unsigned iblocks = (unsigned)std::min<size_t>(8192, std::max<size_t>(1, ceil_div_z(ninit, kCThreads)));
  hipLaunchKernelGGL(ecc_init_kernel, dim3(iblocks), dim3(kCThreads), 0, stream, D, (const uint8_t*)codes, q, D64,
                     ct);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const size_t ng = (size_t)q.M * q.P * q.P * CSP * CSP;
  hipLaunchKernelGGL(ecc_gram_kernel, dim3((unsigned)ceil_div_z(ng, kCThreads)), dim3(kCThreads), 0, stream, S, q,
                     G);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(ecc_start_kernel<CSP>, dim3(sbx, sby), dim3(kCThreads), 0, stream, S, T, q,
                     (const double*)D64, (const uint8_t*)ct, E, opart);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  int nstep = 0;
  int ma = -1;
  for (int s = 0; s < sweeps; ++s) {
    for (int m = 0; m < q.M; ++m, ++nstep) {
      if (ma >= 0) {
        hipLaunchKernelGGL(ecc_apply_kernel<CSP>, dim3((unsigned)eblocks), dim3(kCThreads), 0, stream, S, q, ma,
                           (const double*)delta, E, opart);
        if ((e = hipGetLastError()) != hipSuccess) return e;
      }
      hipLaunchKernelGGL(ecc_corr_kernel<CSP>, dim3((unsigned)pblocks, (unsigned)q.nchunks), dim3(kCThreads), 0,
                         stream, S, q, m, (const double*)E, part);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      hipLaunchKernelGGL(ecc_reduce_kernel<CSP>, dim3((unsigned)pblocks), dim3(kCThreads), 0, stream,
                         (const double*)part, q, m, (const double*)G, (const double*)D64, (const uint8_t*)ct, Hs);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      for (int it = 0; it < inner; ++it) {
        hipLaunchKernelGGL(dupdate, dim3(1), dim3(kCThreads), slds, stream, (const double*)Hs, q, m,
                           (const double*)G, D64, (const uint8_t*)ct, it == 0 ? 1 : 0, Dold, cold, qkg,
                           (const double*)opart, nstep == 0 ? sblocks : eblocks,
                           objective ? objective + nstep : nullptr);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        hipLaunchKernelGGL(bupdate, dim3((unsigned)ceil_div(q.Ct, NW)), dim3(kCThreads), blds, stream,
                           (const double*)Hs, q, m, (const double*)G, (const double*)D64, (const double*)qkg, ct,
                           (const double*)Dold, (const uint8_t*)cold, delta, it == inner - 1 ? 1 : 0);
        if ((e = hipGetLastError()) != hipSuccess) return e;
      }
      ma = m;
    }
  }
  if (ma >= 0) {
    hipLaunchKernelGGL(ecc_apply_kernel<CSP>, dim3((unsigned)eblocks), dim3(kCThreads), 0, stream, S, q, ma,
                       (const double*)delta, E, opart);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  hipLaunchKernelGGL(ecc_finish_kernel, dim3(iblocks), dim3(kCThreads), 0, stream, (const double*)D64, q,
                     (const uint8_t*)ct, D, codes, (const double*)opart, ma >= 0 ? eblocks : sblocks,
                     objective ? objective + nstep : nullptr);
  return hipGetLastError();
}

hipError_t launch_ec_conv(int N, int Cs, int H, int W, int Ct, int dk, int stride, int pad, int M, int K, int Csp,
                          const float* S, const float* T, float* D, uint8_t* codes, int sweeps, int inner,
                          double* objective, hipStream_t stream) {
  const EccParams q = make_params(N, Cs, H, W, Ct, dk, stride, pad, M, K, Csp);
#define QCNN_ECC_CASE(c) \
  case c: return launch_ecc_csp<c>(q, S, T, D, codes, sweeps, inner, objective, stream);
  switch (Csp) {
    QCNN_ECC_CASE(1) QCNN_ECC_CASE(2) QCNN_ECC_CASE(3) QCNN_ECC_CASE(4)
    QCNN_ECC_CASE(5) QCNN_ECC_CASE(6) QCNN_ECC_CASE(7) QCNN_ECC_CASE(8)
    default: return hipErrorInvalidValue;
  }
#undef QCNN_ECC_CASE
}

}  // namespace qcnn
