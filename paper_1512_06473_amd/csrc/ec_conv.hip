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
//   ecc_solve_kernel  one workgroup: `inner` rounds of the two updates, then
//                     delta for the next apply.
#include "qcnn_internal.h"

namespace qcnn {
namespace {

constexpr int kCThreads = 256;

struct EccParams {
  int N, Cs, H, W, Ct, Ho, Wo, dk, stride, pad, M, K, Csp, P, O;
  int chunk, nchunks;  // images per correlation chunk, number of chunks
};

// Coordinate j of the input sub-vector of subspace m that kernel position p
// meets at output o of image n (0 outside the input).
__device__ __forceinline__ float ecc_s(const float* __restrict__ S, const EccParams& q, int n, int m, int j, int o,
                                       int p) {
  const int yo = o / q.Wo, xo = o - yo * q.Wo;
  const int ky = p / q.dk, kx = p - ky * q.dk;
  const int y = yo * q.stride - q.pad + ky, x = xo * q.stride - q.pad + kx;
  if ((unsigned)y >= (unsigned)q.H || (unsigned)x >= (unsigned)q.W) return 0.f;
  return S[(((size_t)n * q.Cs + (size_t)m * q.Csp + j) * q.H + y) * q.W + x];
}

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
  double s = 0.0;
  for (int n = 0; n < q.N; ++n)
    for (int o = 0; o < q.O; ++o)
      s += (double)ecc_s(S, q, n, m, i, o, p) * (double)ecc_s(S, q, n, m, j, o, p2);
  G[i0] = s;
}

// E = T - sum_m sum_p D^(m)[k(c, p)]^T s_p, one element per thread (o
// fastest), subspaces and positions in order; block sums of E^2.
template <int CSP>
__global__ __launch_bounds__(kCThreads) void ecc_start_kernel(const float* __restrict__ S,
                                                            const float* __restrict__ T, EccParams q,
                                                            const double* __restrict__ D64,
                                                            const uint8_t* __restrict__ ct, double* __restrict__ E,
                                                            double* __restrict__ opart) {
  __shared__ double red[kCThreads / kWave];
  const size_t i = (size_t)blockIdx.x * kCThreads + threadIdx.x;
  const size_t total = (size_t)q.N * q.Ct * q.O;
  double e = 0.0;
  if (i < total) {
    const int o = (int)(i % q.O);
    const int c = (int)((i / q.O) % q.Ct);
    const int n = (int)(i / ((size_t)q.O * q.Ct));
    e = (double)T[i];
    for (int m = 0; m < q.M; ++m) {
      const uint8_t* km = ct + ((size_t)m * q.Ct + c) * q.P;
      double d = 0.0;
      for (int p = 0; p < q.P; ++p) {
        const double* w = D64 + ((size_t)m * q.K + km[p]) * CSP;
#pragma unroll
        for (int j = 0; j < CSP; ++j) d += (double)ecc_s(S, q, n, m, j, o, p) * w[j];
      }
      e -= d;
    }
    E[i] = e;
  }
  ecc_block_sum(e * e, red, opart);
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
    const double* dl = delta + (size_t)c * q.P * CSP;
    double d = 0.0;
    for (int p = 0; p < q.P; ++p)
#pragma unroll
      for (int j = 0; j < CSP; ++j) d += (double)ecc_s(S, q, n, ma, j, o, p) * dl[p * CSP + j];
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
  for (int n = n0; n < n1; ++n) {
    const double* er = E + ((size_t)n * q.Ct + c) * q.O;
    for (int o = 0; o < q.O; ++o) {
      const double e = er[o];
#pragma unroll
      for (int j = 0; j < CSP; ++j) acc[j] += (double)ecc_s(S, q, n, m, j, o, p) * e;
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

// Doubles and bytes of the solve kernel's LDS.
template <int CSP> size_t solve_lds_bytes(int K, int npairs) {
  const size_t dbl = (size_t)2 * K * CSP + K + kCThreads + (size_t)kWave * (CSP + 1);
  const size_t ints = 3 * 256 + (kCThreads / kWave) * 256;
  return dbl * 8 + ints * 4 + (size_t)npairs * 2 + (size_t)npairs * 2;
}

// One workgroup per subspace step: the objective before the step (from the
// apply kernel's block sums), `inner` rounds of Eq. (17)-(19) then Eq.
// (20)-(21), and delta for the next apply.
template <int CSP>
__global__ __launch_bounds__(kCThreads) void ecc_solve_kernel(const double* __restrict__ H, EccParams q, int m,
                                                            const double* __restrict__ G, double* __restrict__ D64,
                                                            uint8_t* __restrict__ ct, double* __restrict__ delta,
                                                            const double* __restrict__ opart, int nopart,
                                                            double* __restrict__ objective, int inner) {
  extern __shared__ double sh[];
  const int K = q.K, P = q.P, Ct = q.Ct, npairs = Ct * P;
  double* Ds = sh;                              // [K][C's] current sub-codewords
  double* Do = Ds + K * CSP;                    // [K][C's] at the start of the step
  double* qk = Do + K * CSP;                    // [K]
  double* red = qk + K;                         // [256]
  double* wred = red + kCThreads;               // [64][C's + 1] slot partials
  int* cnt = reinterpret_cast<int*>(wred + kWave * (CSP + 1));  // [256]
  int* start = cnt + 256;                       // [256]
  int* run = start + 256;                       // [256]
  int* wcnt = run + 256;                        // [4][256]
  uint16_t* list = reinterpret_cast<uint16_t*>(wcnt + (kCThreads / kWave) * 256);  // pairs by code
  uint8_t* cs = reinterpret_cast<uint8_t*>(list + npairs);  // [C_t][P] codes
  uint8_t* cso = cs + npairs;                               // [C_t][P] at the start of the step
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const double* Gm = G + (size_t)m * P * P * CSP * CSP;

  double os = 0.0;
  if (objective)
    for (int i = tid; i < nopart; i += kCThreads) os += opart[i];
  for (int i = tid; i < K * CSP; i += kCThreads) Ds[i] = Do[i] = D64[(size_t)m * K * CSP + i];
  for (int i = tid; i < npairs; i += kCThreads) cs[i] = cso[i] = ct[(size_t)m * npairs + i];
  if (objective) {
    red[tid] = os;
    __syncthreads();
    for (int h = kCThreads / 2; h > 0; h >>= 1) {
      if (tid < h) red[tid] += red[tid + h];
      __syncthreads();
    }
    if (tid == 0) *objective = red[0];
  }
  __syncthreads();

  for (int it = 0; it < inner; ++it) {
    // ---- the (c, p) pairs sorted stably by code: list[start[k] ..]
    for (int k = tid; k < 256; k += kCThreads) cnt[k] = run[k] = 0;
    for (int k = tid; k < (kCThreads / kWave) * 256; k += kCThreads) wcnt[k] = 0;
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
        for (int w = 0; w < kCThreads / kWave; ++w) {
          add += wcnt[w * 256 + k];
          wcnt[w * 256 + k] = 0;
        }
        run[k] += add;
      }
      __syncthreads();
    }

    // ---- Eq. (17)-(19): sub-codewords in order, on wave 0.  Lane l works
    // on row j = l % C's of the pairs slot, slot + QS, ... (slot = l / C's);
    // the slots' sums are then added in order.
    if (wave == 0) {
      constexpr int QS = kWave / CSP;
      const int slot = lane / CSP, j = lane - slot * CSP;
      const bool act = slot < QS;
      for (int k = 0; k < K; ++k) {
        const int n_k = cnt[k];
        if (n_k == 0) continue;  // unused: keeps its value
        double rhs = 0.0, mat[CSP];
#pragma unroll
        for (int i = 0; i < CSP; ++i) mat[i] = 0.0;
        if (act) {
          for (int r = slot; r < n_k; r += QS) {
            const int pr = list[start[k] + r];
            const int c = pr / P, p = pr - c * P;
            rhs += H[(size_t)pr * CSP + j];
            for (int p2 = 0; p2 < P; ++p2) {
              const int k2 = cs[c * P + p2];
              const double* g = Gm + (((size_t)p * P + p2) * CSP + j) * CSP;  // G[p][p2][j][.]
              if (k2 == k) {
#pragma unroll
                for (int i = 0; i < CSP; ++i) mat[i] += g[i];
              } else {
                double t = 0.0;
#pragma unroll
                for (int i = 0; i < CSP; ++i) t += g[i] * Ds[k2 * CSP + i];
                rhs -= t;
              }
            }
          }
          double* w = wred + (size_t)(slot * CSP + j) * (CSP + 1);
          w[0] = rhs;
#pragma unroll
          for (int i = 0; i < CSP; ++i) w[1 + i] = mat[i];
        }
        wave_sync_lds();
        // entry e = (row j, column col) of [rhs | matrix]: the used slots in order
        const int used = min(QS, n_k);
        double* rb = red;        // [C's] rhs
        double* rA = red + CSP;  // [C's][C's] normal matrix
        for (int e = lane; e < CSP * (CSP + 1); e += kWave) {
          double v = 0.0;
          for (int s = 0; s < used; ++s) v += wred[(size_t)s * CSP * (CSP + 1) + e];
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
          for (int r = 0; r < CSP; ++r) b[r] = rb[r];
          solve_normal<CSP>(rA, b, Aw, x);
#pragma unroll
          for (int r = 0; r < CSP; ++r) Ds[k * CSP + r] = x[r];
        }
        wave_sync_lds();
      }
    }
    __syncthreads();

    // ---- Eq. (20)-(21): kernel positions in order, one channel per thread
    for (int p = 0; p < P; ++p) {
      const double* Gpp = Gm + ((size_t)p * P + p) * CSP * CSP;
      for (int k = tid; k < K; k += kCThreads) {
        double s = 0.0;
#pragma unroll
        for (int r = 0; r < CSP; ++r) {
          double g = 0.0;
#pragma unroll
          for (int i = 0; i < CSP; ++i) g += Gpp[r * CSP + i] * Ds[k * CSP + i];
          s += Ds[k * CSP + r] * g;
        }
        qk[k] = s;
      }
      __syncthreads();
      for (int c = tid; c < Ct; c += kCThreads) {
        double b[CSP];
        const double* hc = H + ((size_t)c * P + p) * CSP;
#pragma unroll
        for (int r = 0; r < CSP; ++r) b[r] = hc[r];
        for (int p2 = 0; p2 < P; ++p2) {
          if (p2 == p) continue;
          const int k2 = cs[c * P + p2];
          const double* g = Gm + ((size_t)p * P + p2) * CSP * CSP;
#pragma unroll
          for (int r = 0; r < CSP; ++r) {
            double t = 0.0;
#pragma unroll
            for (int i = 0; i < CSP; ++i) t += g[r * CSP + i] * Ds[k2 * CSP + i];
            b[r] -= t;
          }
        }
        int best = 0;
        double bv = 0.0;
        for (int k = 0; k < K; ++k) {
          double d = 0.0;
#pragma unroll
          for (int r = 0; r < CSP; ++r) d += Ds[k * CSP + r] * b[r];
          const double v = qk[k] - 2.0 * d;
          if (k == 0 || v < bv) {
            bv = v;
            best = k;
          }
        }
        cs[c * P + p] = (uint8_t)best;
      }
      __syncthreads();
    }
  }

  for (int i = tid; i < K * CSP; i += kCThreads) D64[(size_t)m * K * CSP + i] = Ds[i];
  for (int i = tid; i < npairs; i += kCThreads) {
    ct[(size_t)m * npairs + i] = cs[i];
#pragma unroll
    for (int r = 0; r < CSP; ++r) delta[(size_t)i * CSP + r] = Ds[cs[i] * CSP + r] - Do[cso[i] * CSP + r];
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
  if (tid == 0 && objective) {  // once per call: a serial sum is fine here
    double s = 0.0;
    for (int b = 0; b < nopart; ++b) s += opart[b];
    *objective = s;
  }
}

EccParams make_params(int N, int Cs, int H, int W, int Ct, int dk, int stride, int pad, int M, int K, int Csp) {
  EccParams q{};
  q.N = N, q.Cs = Cs, q.H = H, q.W = W, q.Ct = Ct, q.dk = dk, q.stride = stride, q.pad = pad;
  q.Ho = (H + 2 * pad - dk) / stride + 1;
  q.Wo = (W + 2 * pad - dk) / stride + 1;
  q.M = M, q.K = K, q.Csp = Csp, q.P = dk * dk, q.O = q.Ho * q.Wo;
  // about 64 Ki correlation threads: (c, p) pairs times image chunks
  const int pairs = Ct * q.P;
  const int want = std::max(1, std::min(N, 65536 / std::max(1, pairs)));
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
  const int pblocks = ceil_div(npairs, kCThreads);
  const size_t slds = solve_lds_bytes<CSP>(q.K, npairs);
  if (slds > kLdsBytes) return hipErrorInvalidValue;
  auto solve = ecc_solve_kernel<CSP>;
  hipError_t e = allow_max_lds((const void*)solve);
  if (e != hipSuccess) return e;
  Scratch scratch;
  size_t bytes = 0;
  const size_t szE = total * 8, szPart = (size_t)q.nchunks * npairs * CSP * 8, szH = (size_t)npairs * CSP * 8;
  const size_t szG = (size_t)q.M * q.P * q.P * CSP * CSP * 8, szD = (size_t)q.M * q.K * CSP * 8;
  const size_t szDelta = (size_t)npairs * CSP * 8, szOp = (size_t)eblocks * 8, szCt = (size_t)q.M * npairs;
  for (size_t b : {szE, szPart, szH, szG, szD, szDelta, szOp, szCt}) bytes += (b + 255) & ~(size_t)255;
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

  const size_t ninit = std::max((size_t)q.M * q.K * CSP, (size_t)q.M * npairs);
  const unsigned iblocks = (unsigned)std::min<size_t>(8192, std::max<size_t>(1, ceil_div_z(ninit, kCThreads)));
  hipLaunchKernelGGL(ecc_init_kernel, dim3(iblocks), dim3(kCThreads), 0, stream, D, (const uint8_t*)codes, q, D64,
                     ct);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const size_t ng = (size_t)q.M * q.P * q.P * CSP * CSP;
  hipLaunchKernelGGL(ecc_gram_kernel, dim3((unsigned)ceil_div_z(ng, kCThreads)), dim3(kCThreads), 0, stream, S, q,
                     G);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(ecc_start_kernel<CSP>, dim3((unsigned)eblocks), dim3(kCThreads), 0, stream, S, T, q,
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
      hipLaunchKernelGGL(solve, dim3(1), dim3(kCThreads), slds, stream, (const double*)Hs, q, m, (const double*)G,
                         D64, ct, delta, (const double*)opart, eblocks, objective ? objective + nstep : nullptr,
                         inner);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      ma = m;
    }
  }
  if (ma >= 0) {
    hipLaunchKernelGGL(ecc_apply_kernel<CSP>, dim3((unsigned)eblocks), dim3(kCThreads), 0, stream, S, q, ma,
                       (const double*)delta, E, opart);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  hipLaunchKernelGGL(ecc_finish_kernel, dim3(iblocks), dim3(kCThreads), 0, stream, (const double*)D64, q,
                     (const uint8_t*)ct, D, codes, (const double*)opart, eblocks,
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
