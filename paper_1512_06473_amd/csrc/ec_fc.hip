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
// quantized layer [N][C_t]; the sub-codebooks D64; the Gram blocks
// Gc[m][d] = S^(m)T S^(m-d) for d < B (d = 0: G of Eq. (11)); the codes
// transposed to [M][C_t] (one subspace's codes contiguous), written back to
// [C_t][M] at the end.  ec_start_kernel forms the starting E in one pass
// over the subspaces.
//
// Batches.  The subspaces are taken B = 32 / C'_s (at most 16) at a time.
// One pass over E per batch (ec_pass_kernel) applies the updates of the
// previous batch's steps in order, E -= S^(m) (W_new - W_old), summing E^2
// after each (the objective after that step, Eq. (8)), and forms
// X^(j) = S^(m_j)T E for every subspace m_j of the next batch.  The step of
// m_j then needs P = S^(m_j)T R^(m_j) with R^(m_j) = E_j + S^(m_j) W^(m_j),
// E_j the residual after the batch's earlier steps i < j, so
//   P = X^(j) - sum_{i<j} Gc[m_j][j-i] (W_new - W_old)^(m_i) + G W^(m_j)
// (the same quantity as a pass over E_j would give, up to rounding), which
// ec_prep_kernel forms per channel without touching E.  Per subspace:
//   ec_prep_kernel  the fit (Eq. (11)) the step waits for, which every
//                   workgroup solves from the blocks' sums of the step
//                   before; the assignment (Eq. (12)) of the subspace fitted
//                   just before (when it lies in the same batch), P as
//                   above, then per block of channels the sums of P_c over
//                   the channels assigned to each sub-codeword, in channel
//                   order (a counting sort in LDS).
// With `inner` > 1 the prep kernel's second form (fit, assignment from P,
// then the sums) repeats.  The last subspace of a batch is fitted and
// assigned by the next pass.
// Readings (shared with the oracle): the descent starts from the given
// sub-codebooks and codes; a sweep visits m in order; a sub-codeword no
// channel uses keeps its value; the normal equations are solved by
// elimination in channel order without row exchanges, a pivot <= 1e-12 x
// the largest diagonal entry of G dropping that coordinate (set to 0);
// assignment ties go to the lowest index.
//
// Bound: HBM for the passes, latency for the per-subspace kernels.  A pass
// reads and writes E once (16 N C_t bytes) per batch of B subspaces; the
// prep and fit kernels move O(C'_s C_t) values each.  The starting residual
// is fp64 arithmetic, 2 N C_t C_s flops once.
#include <stdlib.h>
#include <string.h>

#include "qcnn_internal.h"

namespace qcnn {
namespace {

constexpr int kEcThreads = 256;      // start / prep kernels
constexpr int kPassThreads = 512;    // pass kernel
constexpr int kPassChunk = 8;        // images per thread in the pass kernel
constexpr int kPassCh = 16;          // channels per pass workgroup (32 image chunks each)
constexpr int kUpdThreads = 256;     // fit / objective kernels (one workgroup)

// Subspaces per batch: the pass keeps B x C'_s accumulators per thread.
template <int CSP> constexpr int ec_batch() { return 32 / CSP < 1 ? 1 : (32 / CSP > 16 ? 16 : 32 / CSP); }

struct EcParams {
  int N, Cs, Ct, M, K, Csp, inner;
  int B;        // subspaces per batch
};

// D64 = codebooks, ct[m][c] = codes[c][m] (codes >= K read as K - 1),
// Gc[m][d][i][j] = sum_n S[n][m C's + i] S[n][(m - d) C's + j] (0 for m < d),
// and the grid barriers' failure flag cleared.
__global__ __launch_bounds__(kEcThreads) void ec_init_kernel(const float* __restrict__ S, const float* __restrict__ D,
                                                           const uint8_t* __restrict__ codes, EcParams p,
                                                           double* __restrict__ D64, uint8_t* __restrict__ ct,
                                                           double* __restrict__ Gc, int* __restrict__ fail) {
  const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x, stride = (size_t)gridDim.x * blockDim.x;
  if (tid == 0) *fail = 0;
  const size_t nc = (size_t)p.M * p.Ct, nd = (size_t)p.M * p.K * p.Csp;
  const size_t cc = (size_t)p.Csp * p.Csp, ng = (size_t)p.M * p.B * cc;
  for (size_t i = tid; i < nc; i += stride) {
    const size_t m = i / p.Ct, c = i % p.Ct;
    const uint8_t k = codes[c * p.M + m];
    ct[i] = k < p.K ? k : (uint8_t)(p.K - 1);
  }
  for (size_t i = tid; i < nd; i += stride) D64[i] = (double)D[i];
  for (size_t i = tid; i < ng; i += stride) {
    const int m = (int)(i / (p.B * cc));
    const int d = (int)((i / cc) % p.B);
    const int r = (int)(i % cc);
    double s = 0.0;
    if (m >= d) {
      const int a = m * p.Csp + r / p.Csp, b = (m - d) * p.Csp + r % p.Csp;
      for (int n = 0; n < p.N; ++n) s += (double)S[(size_t)n * p.Cs + a] * (double)S[(size_t)n * p.Cs + b];
    }
    Gc[i] = s;
  }
}

// Fixed-order sum of one value per thread over the workgroup (wave
// shuffles, then the waves in order) into *out.  Every thread must call it.
__device__ __forceinline__ void ec_block_sum(double v, double* red, double* __restrict__ out) {
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_down(v, off, kWave);
  __syncthreads();  // red may still be read by a previous call
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = v;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int w = 0; w < (int)blockDim.x / kWave; ++w) s += red[w];
    *out = s;
  }
}

// The starting residual E = T - S W^T, W[c][m C's + a] = D^(m)[k_m(c)][a]
// (the quantized layer's weights, decoded from the codes), as a float64 GEMM
// on MFMA (v_mfma_f64_16x16x4_f64), and its block sums of E^2.  A workgroup
// of 4 waves owns 64 images x 64 channels; wave w the images 16 w .. 16 w +
// 15 as four 16 x 16 tiles.  The input dimensions go in stages of kStartKB:
// each thread loads its share of the stage's S values (fp32, widened) and
// decoded weights (code, then sub-codeword entry) one stage ahead into
// registers, stores them into one of two LDS buffers, and every wave runs
// the stage's MFMAs from LDS.  Rows and columns past N, C_t or C_s are 0.
constexpr int kStartTile = 64;  // images and channels per workgroup
constexpr int kStartKB = 32;    // input dimensions per stage
constexpr int kStartLd = kStartKB + 1;  // LDS row stride in doubles (odd: spreads the rows over the banks)
typedef double d4v __attribute__((ext_vector_type(4)));

template <int CSP>
__global__ __launch_bounds__(kEcThreads) void ec_start_kernel(const float* __restrict__ S,
                                                            const float* __restrict__ T, EcParams p,
                                                            const double* __restrict__ D64,
                                                            const uint8_t* __restrict__ ct,
                                                            double* __restrict__ E, double* __restrict__ opart) {
  __shared__ double As[2][kStartTile * kStartLd];  // [image][dim]
  __shared__ double Bs[2][kStartTile * kStartLd];  // [channel][dim]
  __shared__ double red[kEcThreads / kWave];
  constexpr int PER = kStartTile * kStartKB / kEcThreads;  // values of each operand per thread and stage (8)
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int c0 = blockIdx.x * kStartTile, n0 = blockIdx.y * kStartTile;
  // this thread's share of a stage: row r (an image of A, a channel of B),
  // dimensions q0 .. q0 + PER - 1 of the stage
  const int r = tid / (kStartKB / PER), q0 = (tid % (kStartKB / PER)) * PER;
  const int na = n0 + r, cb = c0 + r;
  const bool rowa = na < p.N, rowb = cb < p.Ct;
  const int nst = (p.Cs + kStartKB - 1) / kStartKB;
  float sv[PER];
  double wv[PER];
  auto load_stage = [&](int st) {
    int code[PER];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int k = st * kStartKB + q0 + i;
      const bool okk = k < p.Cs;
      const float x = S[rowa && okk ? (size_t)na * p.Cs + k : 0];
      sv[i] = rowa && okk ? x : 0.f;
      const int m = okk ? k / CSP : 0;
      const int cd = ct[rowb && okk ? (size_t)m * p.Ct + cb : 0];
      code[i] = cd;
    }
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int k = st * kStartKB + q0 + i;
      const bool ok = rowb && k < p.Cs;
      const int m = ok ? k / CSP : 0, a = ok ? k % CSP : 0;
      const double w = D64[((size_t)m * p.K + code[i]) * CSP + a];
      wv[i] = ok ? w : 0.0;
    }
  };
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      As[buf][r * kStartLd + q0 + i] = (double)sv[i];
      Bs[buf][r * kStartLd + q0 + i] = wv[i];
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
  // acc[t][i]: image n0 + 16 wave + 4 i + lane / 16, channel c0 + 16 t + lane % 16
  // (the f64 instruction's output layout: register i of lane l holds row
  // 4 i + l / 16, column l % 16)
  double sq = 0.0;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int c = c0 + 16 * t + (lane & 15);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int n = n0 + 16 * wave + 4 * i + kq;
      if (n < p.N && c < p.Ct) {
        const double e = (double)T[(size_t)n * p.Ct + c] - acc[t][i];
        E[(size_t)n * p.Ct + c] = e;
        sq += e * e;
      }
    }
  }
  ec_block_sum(sq, red, opart + (size_t)blockIdx.y * gridDim.x + blockIdx.x);
}

// Eq. (12) for one output channel: the first k minimising
// D_k^T G D_k - 2 D_k^T P_c, with sd = D^(m) [K][C's] and q[k] = D_k^T G D_k.
template <int CSP>
__device__ __forceinline__ int ec_best(const double* sd, const double* q, int K, const double (&pc)[CSP]) {
  int best = 0;
  double bv = 0.0;
#pragma unroll 8
  for (int k = 0; k < K; ++k) {  // unrolled: the table reads of 8 sub-codewords in flight
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

// Threads of a fit that solve at once, and the LDS each takes for its
// elimination (registers up to C'_s = 8).
template <int CSP> __host__ __device__ constexpr int fit_solvers() { return CSP <= 8 ? kUpdThreads : 16; }
template <int CSP> __host__ __device__ constexpr int fit_solve_lds() {
  return CSP <= 8 ? 0 : fit_solvers<CSP>() * CSP * CSP * (int)sizeof(double);
}
// LDS of one fit: G, D, b_k, q (doubles), the elimination storage, |L_k|.
template <int CSP> __host__ __device__ size_t fit_lds_bytes(int K) {
  return (size_t)(CSP * CSP + 2 * K * CSP + K) * sizeof(double) + fit_solve_lds<CSP>() + (size_t)K * sizeof(int);
}

struct FitLds {
  double *Gs, *Ds, *bs, *qs, *Aw;
  int* ns;
};

template <int CSP>
__device__ __forceinline__ FitLds fit_lds(double* base, int K) {
  FitLds f;
  f.Gs = base;                        // [C's][C's]
  f.Ds = f.Gs + CSP * CSP;            // [K][C's]
  f.bs = f.Ds + K * CSP;              // [K][C's] b_k
  f.qs = f.bs + K * CSP;              // [K] D_k^T G D_k
  f.Aw = f.qs + K;                    // elimination storage (C'_s > 8)
  f.ns = reinterpret_cast<int*>(f.Aw + fit_solve_lds<CSP>() / sizeof(double));  // [K] |L_k|
  return f;
}

// Eq. (11) by one workgroup of kUpdThreads threads (vt: the thread's index
// in that role, threadIdx.x if negative; threads of a larger workgroup take
// part with an index >= kUpdThreads and only pass its barriers), for
// subspace mf: b_k and
// |L_k| are the sums over the channel blocks (in order) of the prep
// kernel's bins; each sub-codeword used by some channel becomes
// G^-1 b_k / |L_k|, the others keep their value in Din.  Leaves D in f.Ds
// and q_k = D_k^T G D_k in f.qs (LDS, after a barrier).  Every workgroup
// that runs it on the same inputs gets the same values.
// Inputs of a fit that one thread loads when K C'_s <= kUpdThreads and the
// blocks number at most 16 (the usual case): issued together, straight-line,
// so that a kernel can put them in flight with its own loads.
struct FitRegs {
  double b[16];
  int n[16];
  double din, g;
  bool on;
};

template <int CSP>
__device__ __forceinline__ void ec_fit_issue(const double* __restrict__ bins, const int* __restrict__ nbin, int nblk,
                                             const EcParams& p, int mf, const double* __restrict__ Gc,
                                             const double* __restrict__ Din, FitRegs& r, int vt = -1) {
  const int K = p.K, tid = vt >= 0 ? vt : (int)threadIdx.x;
  r.on = K * CSP <= kUpdThreads && nblk <= 16;
  if (!r.on) return;  // uniform
  const bool bi = tid < K * CSP, ki = tid < K;
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const bool okb = bi && u < nblk, okn = ki && u < nblk;
    const double vb = bins[okb ? (size_t)u * K * CSP + tid : 0];
    const int vn = nbin[okn ? (size_t)u * K + tid : 0];
    r.b[u] = okb ? vb : 0.0;
    r.n[u] = okn ? vn : 0;
  }
  const double vd = Din[bi ? tid : 0];
  const double vg = Gc[(size_t)mf * p.B * CSP * CSP + (tid < CSP * CSP ? tid : 0)];
  r.din = vd;
  r.g = vg;
}

template <int CSP>
__device__ void ec_fit_wg(const double* __restrict__ bins, const int* __restrict__ nbin, int nblk,
                          const EcParams& p, int mf, const double* __restrict__ Gc, const double* __restrict__ Din,
                          const FitLds& f, const FitRegs* pre = nullptr, int vt = -1) {
  const int K = p.K, tid = vt >= 0 ? vt : (int)threadIdx.x;
  if (pre && pre->on) {  // the loads were issued by ec_fit_issue; the sums in block order
    if (tid < CSP * CSP) f.Gs[tid] = pre->g;
    if (tid < K * CSP) {
      f.Ds[tid] = pre->din;
      double s = 0.0;
#pragma unroll
      for (int u = 0; u < 16; ++u)
        if (u < nblk) s += pre->b[u];
      f.bs[tid] = s;
    }
    if (tid < K) {
      int n = 0;
#pragma unroll
      for (int u = 0; u < 16; ++u) n += pre->n[u];
      f.ns[tid] = n;
    }
  } else {
  for (int i = tid; i < CSP * CSP; i += kUpdThreads) f.Gs[i] = Gc[(size_t)mf * p.B * CSP * CSP + i];
  for (int i = tid; i < K * CSP; i += kUpdThreads) f.Ds[i] = Din[i];
  for (int i = tid; i < K * CSP; i += kUpdThreads) {
    double s = 0.0;
    for (int b0 = 0; b0 < nblk; b0 += 8) {  // blocks in order, 8 loads in flight
      double v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = b0 + u < nblk ? bins[(size_t)(b0 + u) * K * CSP + i] : 0.0;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (b0 + u < nblk) s += v[u];
    }
    f.bs[i] = s;
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
    f.ns[k] = n;
  }
  }
  __syncthreads();
  constexpr int SOLVERS = fit_solvers<CSP>();
  for (int k0 = 0; k0 < K; k0 += SOLVERS) {
    const int k = k0 + tid;
    if (tid < SOLVERS && k < K && f.ns[k] > 0) {
      double bk[CSP], x[CSP];
#pragma unroll
      for (int i = 0; i < CSP; ++i) bk[i] = f.bs[k * CSP + i];
      if constexpr (fit_solve_lds<CSP>() > 0) {
        solve_normal<CSP>(f.Gs, bk, f.Aw + (size_t)tid * CSP * CSP, x);
      } else {
        double A[CSP * CSP];
        solve_normal<CSP>(f.Gs, bk, A, x);
      }
#pragma unroll
      for (int i = 0; i < CSP; ++i) f.Ds[k * CSP + i] = x[i] / f.ns[k];
    }
  }
  __syncthreads();
  for (int k = tid; k < K; k += kUpdThreads) {  // D_k^T G D_k
    double s = 0.0;
#pragma unroll
    for (int i = 0; i < CSP; ++i) {
      double g = 0.0;
#pragma unroll
      for (int b = 0; b < CSP; ++b) g += f.Gs[i * CSP + b] * f.Ds[k * CSP + b];
      s += f.Ds[k * CSP + i] * g;
    }
    f.qs[k] = s;
  }
  __syncthreads();
}

// One pass over E for kPassCh channels and every image (kPassThreads /
// kPassCh chunks of kPassChunk images per round of 256), between the batch of
// Lp subspaces starting at mp0 (all fitted; Lp = 0: none) and the batch of
// Ln subspaces starting at mn0 (Ln = 0: none):
//   assign:  the last subspace of the previous batch, ml = mp0 + Lp - 1, by
//            Eq. (12) from P (still that subspace's) and its last fit, which
//            every workgroup makes from the last prep kernel's bins (Din in,
//            Dout out, stored by workgroup 0); the chunk-0
//            threads store the codes;
//   apply:   for i < Lp in order, E[n][c] -= sum_j S[n][(mp0+i) C's + j]
//            dW_i[j][c] (dW_i = D_new[k_new] - D_old[k_old] of step i: from
//            the prep kernels, the last one here), with the block sum of E^2
//            after each into opart[i][block];
//   collect: X[j][a][c] = sum_n S[n][(mn0+j) C's + a] E[n][c] for j < Ln;
//   rows:    Wb[j][a][c] = D^(mn0+j)[k(c)][a] for j < Lw (read before this
//            pass's assignment and before the previous batch's commit, so
//            only for batches that share no subspace with the previous one).
// Per round the images' S columns of both batches are staged in LDS; the
// chunk's E is loaded into registers (all loads in flight) before any of it
// is written.  Each thread keeps its sums of E^2 (one per step) and its X
// partials (B C's of them) in registers; at the end the four chunks of a
// wave are added by shuffles, then the waves in order through LDS (a fixed
// order throughout).  Eight waves per workgroup and ~71 KB of LDS, so that
// two waves share each SIMD.
template <int CSP, int B>
__global__ __launch_bounds__(kPassThreads) void ec_pass_kernel(const float* __restrict__ S, EcParams p,
                                                             double* __restrict__ E, int mp0, int Lp,
                                                             const double* __restrict__ P,
                                                             const double* __restrict__ bins,
                                                             const int* __restrict__ nbin, int nblk,
                                                             const double* __restrict__ Gc,
                                                             const double* __restrict__ Din,
                                                             double* __restrict__ Dout, uint8_t* __restrict__ ct,
                                                             const double* __restrict__ D64,
                                                             const uint8_t* __restrict__ codes_old,
                                                             const double* __restrict__ dW, int mn0, int Ln,
                                                             double* __restrict__ X, double* __restrict__ opart,
                                                             double* __restrict__ Wb, int Lw,
                                                             unsigned* __restrict__ bar) {
  // LDS: dW [B][16][C's], the per-wave sums of E^2 [B][waves], then one area
  // that holds the fit of ml (its D and q) for the assignment, then per round
  // the images' S columns ([chunk][image][2 B C's]: the previous batch's,
  // then the next one's), and at the end the waves' X partials [wave][B C's][16].
  extern __shared__ double sh[];
  constexpr int NCH = kPassThreads / kPassCh;             // image chunks
  constexpr int NW = kPassThreads / kWave;                // waves
  constexpr int kRound = kPassChunk * NCH;                // images per round
  constexpr int BC = B * CSP;
  constexpr int kChunkF = kPassChunk * 2 * BC + 4;        // floats per chunk in the stage (padded: no bank conflicts)
  constexpr int kStage = kRound * 2 * BC;
  static_assert(kWave % kPassCh == 0, "a wave holds whole chunks");
  double* dws = sh;
  double* red = dws + (size_t)B * kPassCh * CSP;  // [B][waves]
  double* area = red + B * NW;
  float* ss = reinterpret_cast<float*>(area);
  double* xw = area;
  const int tid = threadIdx.x, cl = tid % kPassCh, chunk = tid / kPassCh;
  const int lane = tid & (kWave - 1), wave = tid / kWave;
  const int c = blockIdx.x * kPassCh + cl;
  const bool col = c < p.Ct;
  const int cc = col ? c : p.Ct - 1;  // a valid column for loads whose value is not used
  if (blockIdx.x == 0 && tid == 0) *bar = 0;  // for the steps kernel that follows
  // the next batch's weight rows W^(mn0+s)_c = D^(mn0+s)[k(c)], s < Lw, for its
  // prep kernels (Lw = 0 when the two batches share subspaces: ec_rows_kernel
  // gathers them after the commit)
  for (int t = tid; t < Lw * CSP * kPassCh; t += kPassThreads) {
    const int ch = t % kPassCh, sa = t / kPassCh, s = sa / CSP, a = sa - s * CSP;
    const int c2 = blockIdx.x * kPassCh + ch;
    if (c2 < p.Ct) {
      const int kk = ct[(size_t)(mn0 + s) * p.Ct + c2];
      Wb[(size_t)sa * p.Ct + c2] = D64[((size_t)(mn0 + s) * p.K + kk) * CSP + a];
    }
  }
  double xacc[BC], sq[B];
#pragma unroll
  for (int i = 0; i < BC; ++i) xacc[i] = 0.0;
#pragma unroll
  for (int i = 0; i < B; ++i) sq[i] = 0.0;
  if (Lp > 0) {
    const int ml = mp0 + Lp - 1;
    // dW of the batch's earlier steps for the block's channels (zeros past the block)
    for (int t = tid; t < (Lp - 1) * kPassCh * CSP; t += kPassThreads) {
      const int i = t / (kPassCh * CSP), r = t % (kPassCh * CSP), ch = r / CSP, a = r % CSP;
      const int c2 = blockIdx.x * kPassCh + ch;
      dws[t] = c2 < p.Ct ? dW[((size_t)i * CSP + a) * p.Ct + c2] : 0.0;
    }
    const int vt = tid < kUpdThreads ? tid : kUpdThreads + tid;  // the fit's first kUpdThreads threads
    FitRegs pre;
    ec_fit_issue<CSP>(bins, nbin, nblk, p, ml, Gc, Din, pre, vt);
    double pc[CSP];
#pragma unroll
    for (int j = 0; j < CSP; ++j) pc[j] = P[(size_t)j * p.Ct + cc];
    const double* wo = D64 + ((size_t)ml * p.K + codes_old[(size_t)(Lp - 1) * p.Ct + cc]) * CSP;
    double dwo[CSP];
#pragma unroll
    for (int j = 0; j < CSP; ++j) dwo[j] = wo[j];
    const FitLds f = fit_lds<CSP>(area, p.K);
    ec_fit_wg<CSP>(bins, nbin, nblk, p, ml, Gc, Din, f, &pre, vt);  // ends with a barrier
    if (blockIdx.x == 0)
      for (int i = tid; i < p.K * CSP; i += kPassThreads) Dout[i] = f.Ds[i];
    const double* sd = f.Ds;
    if (chunk == 0) {
      const int knew = ec_best<CSP>(sd, f.qs, p.K, pc);
      if (col) ct[(size_t)ml * p.Ct + c] = (uint8_t)knew;
#pragma unroll
      for (int j = 0; j < CSP; ++j)
        dws[((size_t)(Lp - 1) * kPassCh + cl) * CSP + j] = col ? sd[knew * CSP + j] - dwo[j] : 0.0;
    }
  }
  for (int r0 = 0; r0 < p.N; r0 += kRound) {
    __syncthreads();  // the assignment table or the previous round's stage may still be read
    constexpr int kPer = kStage / kPassThreads;  // stage values per thread, all loads in flight
    static_assert(kStage % kPassThreads == 0 && kPer <= 64, "stage share per thread");
    {
      float v[kPer];
#pragma unroll
      for (int u = 0; u < kPer; ++u) {  // straight-line: every load issued, unused values masked
        const int t = u * kPassThreads + tid;
        const int img = t / (2 * BC), col2 = t % (2 * BC);
        const int half = col2 / BC, c3 = col2 % BC;
        const int len = half == 0 ? Lp : Ln, m0 = half == 0 ? mp0 : mn0;
        const bool ok = r0 + img < p.N && c3 < len * CSP;
        const size_t at = ok ? (size_t)(r0 + img) * p.Cs + (size_t)m0 * CSP + c3 : 0;
        const float x = S[at];
        v[u] = ok ? x : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kPer; ++u) {
        const int t = u * kPassThreads + tid;
        const int img = t / (2 * BC);
        ss[(img / kPassChunk) * kChunkF + (img % kPassChunk) * 2 * BC + t % (2 * BC)] = v[u];
      }
    }
    __syncthreads();
    const int n0 = r0 + chunk * kPassChunk;
    // images past N: E read at a valid row and zeroed (their S is 0 too)
    double e[kPassChunk];
#pragma unroll
    for (int i = 0; i < kPassChunk; ++i) {
      const double v = E[(size_t)min(n0 + i, p.N - 1) * p.Ct + cc];
      e[i] = col && n0 + i < p.N ? v : 0.0;
    }
    const float* sr = ss + (size_t)chunk * kChunkF;  // [image][2 B C's] of this chunk
#pragma unroll
    for (int s = 0; s < B; ++s) {
      if (s < Lp) {
        double dw[CSP];
#pragma unroll
        for (int j = 0; j < CSP; ++j) dw[j] = dws[((size_t)s * kPassCh + cl) * CSP + j];
        double sqs = 0.0;
#pragma unroll
        for (int i = 0; i < kPassChunk; ++i) {
          const float* srow = sr + i * 2 * BC + s * CSP;
          double d = 0.0;
#pragma unroll
          for (int j = 0; j < CSP; ++j) d += (double)srow[j] * dw[j];
          e[i] -= d;
          sqs += e[i] * e[i];
        }
        sq[s] += sqs;
      }
    }
    if (Lp > 0 && col) {
#pragma unroll
      for (int i = 0; i < kPassChunk; ++i)
        if (n0 + i < p.N) E[(size_t)(n0 + i) * p.Ct + c] = e[i];
    }
#pragma unroll
    for (int s = 0; s < B; ++s) {
      if (s < Ln) {
#pragma unroll
        for (int i = 0; i < kPassChunk; ++i) {
          const float* srow = sr + i * 2 * BC + BC + s * CSP;
#pragma unroll
          for (int j = 0; j < CSP; ++j) xacc[s * CSP + j] += (double)srow[j] * e[i];
        }
      }
    }
  }
  // the block sums of E^2 after each step: per wave in a fixed shuffle
  // order, then the waves in order
  if (Lp > 0) {
#pragma unroll
    for (int s = 0; s < B; ++s) {
      if (s < Lp) {
        double v = sq[s];
        for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_down(v, off, kWave);
        if (lane == 0) red[s * NW + wave] = v;
      }
    }
    __syncthreads();
    if (tid < Lp) {
      double v = 0.0;
      for (int w = 0; w < NW; ++w) v += red[tid * NW + w];
      opart[(size_t)tid * gridDim.x + blockIdx.x] = v;
    }
  }
  if (Ln > 0) {
    // X partials: the wave's four chunks of each channel by shuffles, then
    // the waves in order
    __syncthreads();  // the last round's stage is no longer read
#pragma unroll
    for (int sj = 0; sj < BC; ++sj) {
      if (sj < Ln * CSP) {
        double v = xacc[sj];
        for (int off = kWave / 2; off >= kPassCh; off >>= 1) v += __shfl_down(v, off, kWave);
        if (lane < kPassCh) xw[((size_t)wave * BC + sj) * kPassCh + lane] = v;
      }
    }
    __syncthreads();
    for (int t = tid; t < kPassCh * Ln * CSP; t += kPassThreads) {
      const int ch = t % kPassCh, sj = t / kPassCh;  // sj = s C's + j
      const int c2 = blockIdx.x * kPassCh + ch;
      double v = 0.0;
      for (int w = 0; w < NW; ++w) v += xw[((size_t)w * BC + sj) * kPassCh + ch];
      if (c2 < p.Ct) X[(size_t)sj * p.Ct + c2] = v;
    }
  }
}

template <int CSP, int B> size_t pass_lds_bytes(int K) {
  constexpr int NCH = kPassThreads / kPassCh, NW = kPassThreads / kWave;
  const size_t fixed = ((size_t)B * kPassCh * CSP + (size_t)B * NW) * sizeof(double);
  const size_t fit = fit_lds_bytes<CSP>(K);
  const size_t stage = (size_t)NCH * (kPassChunk * 2 * B * CSP + 4) * sizeof(float);
  const size_t xpart = (size_t)NW * B * CSP * kPassCh * sizeof(double);
  return fixed + std::max({fit, stage, xpart});
}

// After a batch's pass: D64[mp0 + i] = Dnew[i] for i < Lp (the batch's final
// sub-codebooks), and objective[s] = the sum over the blocks of
// opart[s][block] for s < rows <= 16, in a fixed order: 16 threads per row
// each add a strided share of the blocks in order, then a fixed tree over
// the 16.  One workgroup of kUpdThreads threads; red: kUpdThreads doubles of
// LDS.
struct EcCommit {
  const double* opart;
  int nblk, rows;
  double* objective;  // null: the sub-codebooks only
  const double* Dnew;
  double* D64;
  int mp0, Lp, kc;
};

__device__ void ec_commit_wg(const EcCommit& c, double* red) {
  const int tid = threadIdx.x;
  for (int i = tid; i < c.Lp * c.kc; i += kUpdThreads) c.D64[(size_t)c.mp0 * c.kc + i] = c.Dnew[i];
  if (!c.objective) return;  // uniform
  const int s = tid / 16, t = tid % 16;
  double v = 0.0;
  if (s < c.rows)
    for (int b0 = t; b0 < c.nblk; b0 += 16 * 16) {  // 16 loads in flight, added in order
      double x[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) x[u] = b0 + 16 * u < c.nblk ? c.opart[(size_t)s * c.nblk + b0 + 16 * u] : 0.0;
#pragma unroll
      for (int u = 0; u < 16; ++u) v += x[u];
    }
  red[tid] = v;
  __syncthreads();
  for (int h = 8; h > 0; h >>= 1) {
    if (t < h) red[tid] += red[tid + h];
    __syncthreads();
  }
  if (t == 0 && s < c.rows) c.objective[s] = red[tid];
}

__global__ __launch_bounds__(kUpdThreads) void ec_commit_kernel(EcCommit c) {
  __shared__ double red[kUpdThreads];
  ec_commit_wg(c, red);
}

// Wb[s][a][c] = D64[m0 + s][ct[m0 + s][c]][a] for s < L: a batch's weight
// rows at its start, when the pass cannot gather them (the batch shares
// subspaces with the previous one, whose assignment and commit come first).
__global__ __launch_bounds__(kEcThreads) void ec_rows_kernel(EcParams p, const double* __restrict__ D64,
                                                           const uint8_t* __restrict__ ct, int m0, int L,
                                                           double* __restrict__ Wb) {
  const size_t t = (size_t)blockIdx.x * kEcThreads + threadIdx.x;
  if (t >= (size_t)L * p.Csp * p.Ct) return;
  const int c = (int)(t % p.Ct);
  const int sa = (int)(t / p.Ct), s = sa / p.Csp, a = sa - s * p.Csp;
  const int kk = ct[(size_t)(m0 + s) * p.Ct + c];
  Wb[t] = D64[((size_t)(m0 + s) * p.K + kk) * p.Csp + a];
}

// LDS of the prep kernel: a fit, then P of the block in sorted order and
// the counting sort's counts and offsets.
template <int CSP> size_t prep_lds_bytes(int K) {
  return fit_lds_bytes<CSP>(K) + (size_t)kEcThreads * CSP * sizeof(double) +
         ((size_t)(kEcThreads / kWave) * K + 2 * (size_t)K) * sizeof(int);
}

// Per block of 256 output channels, step j of the batch (subspace m = m0 + j),
// round `it` of Eq. (11)-(12):
//   first (fm >= 0), the fit this step depends on, as ec_fit_wg (every
//   workgroup computes it; workgroup 0 stores it in Dout): that of the last
//   round of m - 1 (it == 0) or of round it - 1 of m;
//   it == 0: if j > 0, the assignment of m - 1 (Eq. (12)) with that fit,
//            dW_{j-1}[a][c] = D_new[k_new][a] - D64[m-1][k_old][a] stored;
//            then P_c = X^(j)_c - sum_{i<j} Gc[m][j-i] dW_i[.][c]
//            + G W^(m)_c, stored, and codes_old[j] = the codes of m;
//   it >= 1: the codes of m by Eq. (12) from P and the fit;
// then the block's sums over the channels assigned to each sub-codeword,
// in channel order: bins[block][k][j] = sum of P_c[j], nbin[block][k] the
// count.  The sums come from a counting sort in LDS: per wave, the lanes
// sharing a code find their rank with ballots; codes x waves give each
// channel its place, and one thread per (k, j) adds its run in order.
template <int CSP, int B>
__device__ __forceinline__ void ec_prep_step(const EcParams& p, int m0, int j, int it, int fm,
                                             const double* __restrict__ Din, const double* __restrict__ bins_in,
                                             const int* __restrict__ nbin_in, int nblk, double* __restrict__ Dout,
                                             const double* __restrict__ X, const double* __restrict__ Gc,
                                             const double* __restrict__ Wb, uint8_t* __restrict__ ct,
                                             double* __restrict__ P, double* __restrict__ dW,
                                             uint8_t* __restrict__ codes_old, double* __restrict__ bins,
                                             int* __restrict__ nbin, double* sp) {
  const FitLds f = fit_lds<CSP>(sp, p.K);
  double* Ps = reinterpret_cast<double*>(reinterpret_cast<char*>(sp) + fit_lds_bytes<CSP>(p.K));  // [256][C's]
  int* cnt = reinterpret_cast<int*>(Ps + (size_t)kEcThreads * CSP);  // [waves][K]
  int* tot = cnt + (kEcThreads / kWave) * p.K;                       // [K]
  int* base = tot + p.K;                                             // [K]
  const int tid = threadIdx.x, c = blockIdx.x * kEcThreads + tid;
  const int lane = tid & (kWave - 1), wave = tid / kWave;
  const bool col = c < p.Ct;
  const int m = m0 + j;
  const double* gm = Gc + (size_t)m * p.B * CSP * CSP;  // Gc[m][d] = gm + d C's^2
  // the fit's loads and those that do not depend on it, issued first
  FitRegs pre;
  pre.on = false;
  if (fm >= 0) ec_fit_issue<CSP>(bins_in, nbin_in, nblk, p, fm, Gc, Din, pre);
  double pc[CSP], pp[CSP], dlast[CSP], wrow[CSP], worow[CSP];
#pragma unroll
  for (int a = 0; a < CSP; ++a) dlast[a] = 0.0;
  int k = 0;
  double dwv[B][CSP];  // dW of the steps before the previous one
  if (col) {
    if (it == 0) {
#pragma unroll
      for (int a = 0; a < CSP; ++a) pc[a] = X[((size_t)j * CSP + a) * p.Ct + c];
#pragma unroll
      for (int i = 0; i < B; ++i)
        if (i < j - 1)
#pragma unroll
          for (int a = 0; a < CSP; ++a) dwv[i][a] = dW[((size_t)i * CSP + a) * p.Ct + c];
      k = ct[(size_t)m * p.Ct + c];
      // W^(m)_c and W^(m-1)_c as they were when the batch began (gathered by the pass)
#pragma unroll
      for (int a = 0; a < CSP; ++a) {
        wrow[a] = Wb[((size_t)j * CSP + a) * p.Ct + c];
        worow[a] = Wb[((size_t)(j > 0 ? j - 1 : j) * CSP + a) * p.Ct + c];
      }
    }
    if (it > 0 || j > 0)
#pragma unroll
      for (int a = 0; a < CSP; ++a) pp[a] = P[(size_t)a * p.Ct + c];
  }
  if (fm >= 0) {
    ec_fit_wg<CSP>(bins_in, nbin_in, nblk, p, fm, Gc, Din, f, &pre);
    if (blockIdx.x == 0)
      for (int i = tid; i < p.K * CSP; i += kEcThreads) Dout[i] = f.Ds[i];
  }
  if (col) {
    if (it == 0) {
      if (j > 0) {  // m - 1 with its last fit
        const int knew = ec_best<CSP>(f.Ds, f.qs, p.K, pp);
        ct[(size_t)(m - 1) * p.Ct + c] = (uint8_t)knew;
#pragma unroll
        for (int a = 0; a < CSP; ++a) {
          dlast[a] = f.Ds[knew * CSP + a] - worow[a];
          dW[((size_t)(j - 1) * CSP + a) * p.Ct + c] = dlast[a];
        }
      }
#pragma unroll
      for (int i = 0; i < B; ++i) {
        if (i < j) {
          const bool last = i == j - 1;
          const double* g = gm + (size_t)(j - i) * CSP * CSP;
#pragma unroll
          for (int a = 0; a < CSP; ++a) {
            double s = 0.0;
#pragma unroll
            for (int b = 0; b < CSP; ++b) s += g[a * CSP + b] * (last ? dlast[b] : dwv[i][b]);
            pc[a] -= s;
          }
        }
      }
#pragma unroll
      for (int a = 0; a < CSP; ++a) {
        double s = 0.0;
#pragma unroll
        for (int b = 0; b < CSP; ++b) s += gm[a * CSP + b] * wrow[b];
        pc[a] += s;
        P[(size_t)a * p.Ct + c] = pc[a];
      }
      codes_old[(size_t)j * p.Ct + c] = (uint8_t)k;
    } else {
#pragma unroll
      for (int a = 0; a < CSP; ++a) pc[a] = pp[a];
      k = ec_best<CSP>(f.Ds, f.qs, p.K, pc);
      ct[(size_t)m * p.Ct + c] = (uint8_t)k;
    }
  }
  // ---- counting sort of the block's channels by code
  for (int i = lane; i < p.K; i += kWave) cnt[wave * p.K + i] = 0;
  // (each wave clears and fills only its own row of counts)
  // the lanes holding this lane's code: matched bit by bit over the code's
  // bits, one ballot per bit
  int rank = 0;
  {
    uint64_t same = __ballot(col);
    for (int bit = 0; (1 << bit) < p.K; ++bit) {
      const bool one = ((k >> bit) & 1) != 0;
      const uint64_t ones = __ballot(col && one);
      same &= one ? ones : ~ones;
    }
    if (col) {
      rank = __popcll(same & ((1ull << lane) - 1ull));
      if (rank == 0) cnt[wave * p.K + k] = __popcll(same);  // the code's lowest lane
    }
  }
  __syncthreads();
  for (int kk = tid; kk < p.K; kk += kEcThreads) {
    int t = 0;
    for (int w = 0; w < kEcThreads / kWave; ++w) t += cnt[w * p.K + kk];
    tot[kk] = t;
  }
  __syncthreads();
  if (p.K <= kWave) {  // exclusive prefix of tot by one wave's shuffles
    if (wave == 0) {
      const int t = lane < p.K ? tot[lane] : 0;
      int v = t;
      for (int off = 1; off < kWave; off <<= 1) {
        const int u = __shfl_up(v, off, kWave);
        if (lane >= off) v += u;
      }
      if (lane < p.K) base[lane] = v - t;
    }
  } else {
    for (int kk = tid; kk < p.K; kk += kEcThreads) {
      int b0 = 0;
      for (int i = 0; i < kk; ++i) b0 += tot[i];
      base[kk] = b0;
    }
  }
  __syncthreads();
  if (col) {
    int pos = base[k] + rank;
    for (int w = 0; w < wave; ++w) pos += cnt[w * p.K + k];
#pragma unroll
    for (int a = 0; a < CSP; ++a) Ps[(size_t)pos * CSP + a] = pc[a];
  }
  __syncthreads();
  for (int t = tid; t < p.K * CSP; t += kEcThreads) {
    const int kk = t / CSP, a = t % CSP;
    const int n = tot[kk];
    const double* run = Ps + (size_t)base[kk] * CSP + a;
    double s = 0.0;
    int i = 0;
    for (; i + 8 <= n; i += 8) {  // eight reads in flight, added in order
      double v[8];
#pragma unroll
      for (int x = 0; x < 8; ++x) v[x] = run[(size_t)(i + x) * CSP];
#pragma unroll
      for (int x = 0; x < 8; ++x) s += v[x];
    }
    for (; i < n; ++i) s += run[(size_t)i * CSP];
    bins[((size_t)blockIdx.x * p.K + kk) * CSP + a] = s;
  }
  for (int kk = tid; kk < p.K; kk += kEcThreads) nbin[(size_t)blockIdx.x * p.K + kk] = tot[kk];
}

template <int CSP, int B>
__global__ __launch_bounds__(kEcThreads) void ec_prep_kernel(EcParams p, int m0, int j, int it, int fm,
                                                           const double* __restrict__ Din,
                                                           const double* __restrict__ bins_in,
                                                           const int* __restrict__ nbin_in, int nblk,
                                                           double* __restrict__ Dout, const double* __restrict__ X,
                                                           const double* __restrict__ Gc,
                                                           const double* __restrict__ Wb, uint8_t* __restrict__ ct,
                                                           double* __restrict__ P, double* __restrict__ dW,
                                                           uint8_t* __restrict__ codes_old,
                                                           double* __restrict__ bins, int* __restrict__ nbin,
                                                           EcCommit cm) {
  extern __shared__ double sp[];
  if ((int)blockIdx.x >= nblk) {  // the workgroup past the channel blocks: the previous batch's commit
    ec_commit_wg(cm, sp);
    return;
  }
  ec_prep_step<CSP, B>(p, m0, j, it, fm, Din, bins_in, nbin_in, nblk, Dout, X, Gc, Wb, ct, P, dW, codes_old, bins,
                       nbin, sp);
}

// Buffers of a batch's steps (the workspace slices of launch_ec_csp).
struct EcSteps {
  const double* X;
  const double* Wb;   // [B][C's][C_t]: the batch's weight rows at its start
  const double* Gc;
  double* D64;
  uint8_t* ct;
  double* P;
  double* dW;
  uint8_t* codes_old;
  double* bins;       // [2][blocks][K][C's]
  int* nbin;          // [2][blocks][K]
  double* Dnew;       // [B][K][C's]: each step's last fit
  double* Dpp;        // [2][K][C's]: the fits of the inner rounds before the last
  unsigned* bar;      // arrival count of the grid barriers (0 at launch)
  int* fail;          // set when a barrier gives up waiting
};

// Polls of a grid barrier before it gives up (each a memory round trip and
// ~64 clocks of sleep: about a second, against microseconds when every
// workgroup is resident).
constexpr int kBarrierPolls = 1 << 20;

// Every workgroup of the grid arrives here before any leaves: the writes
// before it (global memory, every thread) are visible after it to every
// workgroup.  Arrivals count up on *bar; `target` is the count once every
// workgroup has arrived at this barrier.  Requires every workgroup of the
// grid to be resident (a cooperative launch).  The wait is bounded: after
// kBarrierPolls polls the workgroup sets *fail and goes on, and once *fail
// is set a barrier gives up within 256 polls.
__device__ __forceinline__ void grid_barrier(unsigned* bar, unsigned target, int* fail) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  __syncthreads();
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_add(bar, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    for (int polls = 0; __hip_atomic_load(bar, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target; ++polls) {
      if (polls >= kBarrierPolls) {
        __hip_atomic_store(fail, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
      if ((polls & 255) == 255 && __hip_atomic_load(fail, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) break;
      __builtin_amdgcn_s_sleep(1);
    }
  }
  __syncthreads();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
}

// Every step of a batch (subspaces m0 .. m0 + L - 1, `inner` rounds each) in
// one launch, one workgroup per block of 256 channels as ec_prep_kernel,
// the steps separated by grid barriers instead of kernel boundaries (the
// batch's last fit is made by the pass that follows).  The step sequence, its inputs and outputs and every sum's
// order are those of the per-step kernels, so the results are the same bit
// for bit.  sel0: the bins buffer the step before the batch wrote.
template <int CSP, int B>
__global__ __launch_bounds__(kEcThreads) void ec_steps_kernel(EcParams p, int m0, int L, int sel0, EcSteps b) {
  extern __shared__ double sp[];
  const int kc = p.K * CSP, nblk = gridDim.x;
  auto bins_at = [&](int sel) { return b.bins + (size_t)sel * nblk * kc; };
  auto nbin_at = [&](int sel) { return b.nbin + (size_t)sel * nblk * p.K; };
  auto fit_in = [&](int m, int r) -> const double* {
    return r == 0 ? b.D64 + (size_t)m * kc : b.Dpp + (size_t)((r - 1) % 2) * kc;
  };
  auto fit_out = [&](int jj, int r) -> double* {
    return r == p.inner - 1 ? b.Dnew + (size_t)jj * kc : b.Dpp + (size_t)(r % 2) * kc;
  };
  int sel = sel0;
  unsigned target = 0;
  for (int j = 0; j < L; ++j) {
    for (int it = 0; it < p.inner; ++it) {
      int fm = -1, fj = 0, fr = 0;  // the fit this step waits for, as in the per-step launches
      if (it > 0) {
        fm = m0 + j;
        fj = j;
        fr = it - 1;
      } else if (j > 0) {
        fm = m0 + j - 1;
        fj = j - 1;
        fr = p.inner - 1;
      }
      if (fm >= 0) {  // the previous step's bins (and fit) from every workgroup
        target += (unsigned)nblk;
        grid_barrier(b.bar, target, b.fail);
      }
      ec_prep_step<CSP, B>(p, m0, j, it, fm, fm >= 0 ? fit_in(fm, fr) : b.D64, bins_at(sel), nbin_at(sel), nblk,
                           fm >= 0 ? fit_out(fj, fr) : b.Dpp, b.X, b.Gc, b.Wb, b.ct, b.P, b.dW, b.codes_old,
                           bins_at(sel ^ 1), nbin_at(sel ^ 1), sp);
      sel ^= 1;
    }
  }
}

// codebooks = fp32(D64) (all NaN if a grid barrier of the call gave up
// waiting), codes[c][m] = ct[m][c].
__global__ __launch_bounds__(kEcThreads) void ec_finish_kernel(const double* __restrict__ D64, EcParams p,
                                                             const uint8_t* __restrict__ ct,
                                                             const int* __restrict__ fail,
                                                             float* __restrict__ D, uint8_t* __restrict__ codes) {
  const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x, stride = (size_t)gridDim.x * blockDim.x;
  const size_t nd = (size_t)p.M * p.K * p.Csp, nc = (size_t)p.M * p.Ct;
  const bool bad = *fail != 0;  // a grid barrier gave up: the results are not the method's
  for (size_t i = tid; i < nd; i += stride) D[i] = bad ? __builtin_nanf("") : (float)D64[i];
  for (size_t i = tid; i < nc; i += stride) codes[i] = ct[(i % p.M) * p.Ct + i / p.M];
}

}  // namespace

template <int CSP>
hipError_t launch_ec_csp(int N, int Cs, int Ct, int M, int K, const float* S, const float* T, float* D,
                         uint8_t* codes, int sweeps, int inner, double* objective, hipStream_t stream) {
  constexpr int Csp = CSP;
  constexpr int B = ec_batch<CSP>();
  EcParams p{N, Cs, Ct, M, K, Csp, inner, B};
  const int cblocks = ceil_div(Ct, kEcThreads);     // prep workgroups (channel blocks)
  const int pblocks = ceil_div(Ct, kPassCh);        // pass workgroups
  const int sblocks_c = ceil_div(Ct, kStartTile), sblocks_n = ceil_div(N, kStartTile);
  const int nstart = sblocks_c * sblocks_n;         // start kernel's block sums
  const int kc = K * Csp;
  auto pass = ec_pass_kernel<CSP, B>;
  auto prep = ec_prep_kernel<CSP, B>;
  auto steps = ec_steps_kernel<CSP, B>;
  const size_t pass_lds = pass_lds_bytes<CSP, B>(K);
  const size_t prep_lds = prep_lds_bytes<CSP>(K);
  if (pass_lds > kLdsBytes || prep_lds > kLdsBytes) return hipErrorInvalidValue;
  hipError_t e;
  if ((e = allow_max_lds((const void*)pass)) != hipSuccess) return e;
  if ((e = allow_max_lds((const void*)prep)) != hipSuccess) return e;
  if ((e = allow_max_lds((const void*)steps)) != hipSuccess) return e;
  // QCNN_EC_STEPS=batch (read per call): a batch's steps in one cooperative
  // launch with grid barriers between them, where the device supports it and
  // every channel block's workgroup can be resident at once.  Not the
  // default: on the fc6 shape a step then takes ~16 us of the kernel against
  // 12.7 us for a prep kernel of its own (a barrier's fences and memory-side
  // atomics across the XCDs cost more than a kernel boundary).
  bool coop = false;
  {
    const char* env = getenv("QCNN_EC_STEPS");
    int dev = 0, attr = 0, cus = 0, per_cu = 0;
    if (env && strcmp(env, "batch") == 0 && hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&attr, hipDeviceAttributeCooperativeLaunch, dev) == hipSuccess && attr &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void*)steps, kEcThreads, prep_lds) ==
            hipSuccess)
      coop = (long long)per_cu * cus >= cblocks;
  }
  // workspace slices, each rounded up to 256 bytes
  const size_t sizes[] = {
      (size_t)N * Ct * 8,                                  // E
      (size_t)B * Csp * Ct * 8,                            // X
      (size_t)B * Csp * Ct * 8,                            // Wb
      (size_t)Csp * Ct * 8,                                // P
      (size_t)B * Csp * Ct * 8,                            // dW
      (size_t)M * B * Csp * Csp * 8,                       // Gc
      (size_t)M * kc * 8,                                  // D64
      (size_t)B * kc * 8,                                  // Dnew
      (size_t)2 * kc * 8,                                  // Dpp (fits of the inner rounds)
      (size_t)std::max(nstart, B * pblocks) * 8,           // objective block sums
      (size_t)2 * cblocks * kc * 8,                        // bins (two buffers)
      (size_t)2 * cblocks * K * 4,                         // nbin (two buffers)
      (size_t)B * Ct,                                      // codes_old
      (size_t)M * Ct,                                      // codes, [M][C_t]
      sizeof(unsigned),                                    // grid barrier arrivals
      sizeof(int),                                         // grid barrier failure flag
  };
  size_t total = 0;
  for (size_t b : sizes) total += (b + 255) & ~(size_t)255;
  Scratch scratch;
  if ((e = scratch.acquire(stream, total)) != hipSuccess) return e;
  char* w = scratch.get();
  int si = 0;
  auto take = [&]() {
    char* r = w;
    w += (sizes[si++] + 255) & ~(size_t)255;
    return r;
  };
  double* E = reinterpret_cast<double*>(take());
  double* X = reinterpret_cast<double*>(take());
  double* Wb = reinterpret_cast<double*>(take());
  double* P = reinterpret_cast<double*>(take());
  double* dW = reinterpret_cast<double*>(take());
  double* Gc = reinterpret_cast<double*>(take());
  double* D64 = reinterpret_cast<double*>(take());
  double* Dnew = reinterpret_cast<double*>(take());
  double* Dpp = reinterpret_cast<double*>(take());
  double* opart = reinterpret_cast<double*>(take());
  double* bins = reinterpret_cast<double*>(take());
  int* nbin = reinterpret_cast<int*>(take());
  uint8_t* codes_old = reinterpret_cast<uint8_t*>(take());
  uint8_t* ct = reinterpret_cast<uint8_t*>(take());
  unsigned* bar = reinterpret_cast<unsigned*>(take());
  int* fail = reinterpret_cast<int*>(take());
  auto bins_at = [&](int sel) { return bins + (size_t)sel * cblocks * kc; };
  auto nbin_at = [&](int sel) { return nbin + (size_t)sel * cblocks * K; };

  const size_t ninit = std::max<size_t>({(size_t)M * Ct, (size_t)M * kc, (size_t)M * B * Csp * Csp});
  const unsigned iblocks = (unsigned)std::min<size_t>(8192, ceil_div_z(ninit, kEcThreads));
  hipLaunchKernelGGL(ec_init_kernel, dim3(iblocks), dim3(kEcThreads), 0, stream, S, D, (const uint8_t*)codes, p,
                     D64, ct, Gc, fail);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(ec_start_kernel<CSP>, dim3((unsigned)sblocks_c, (unsigned)sblocks_n), dim3(kEcThreads), 0,
                     stream, S, T, p, (const double*)D64, (const uint8_t*)ct, E, opart);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (objective) {
    hipLaunchKernelGGL(ec_commit_kernel, dim3(1), dim3(kUpdThreads), 0, stream,
                       EcCommit{opart, nstart, 1, objective, Dnew, D64, 0, 0, kc});
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  // Input of the fit of round r of subspace m: D64[m] for r = 0, else the
  // previous round's fit (Dpp[(r - 1) % 2]); its output: Dpp[r % 2], or
  // Dnew[j] for the last round.  No fit reads the buffer it writes.
  auto fit_in = [&](int m, int r) -> const double* {
    return r == 0 ? D64 + (size_t)m * kc : Dpp + (size_t)((r - 1) % 2) * kc;
  };
  auto fit_out = [&](int j, int r) -> double* {
    return r == inner - 1 ? Dnew + (size_t)j * kc : Dpp + (size_t)(r % 2) * kc;
  };
  int sel = 0;            // bins buffer the last prep kernel wrote
  int nstep = 0;          // subspace steps whose objective is recorded
  int mp0 = -1, Lp = 0;   // the previous batch (fitted but for its last round, updates not yet in E)
  // The previous batch's commit after its pass: run by an extra workgroup of
  // the next batch's first prep kernel (it touches only that batch's rows of
  // D64 and the pass's block sums, which no prep kernel reads), else by a
  // kernel of its own (after the last pass, with the batch launches, and when
  // the next batch shares subspaces with the previous one).
  EcCommit pending{};
  bool has_pending = false;
  auto launch_pending = [&]() -> hipError_t {
    if (!has_pending) return hipSuccess;
    has_pending = false;
    hipLaunchKernelGGL(ec_commit_kernel, dim3(1), dim3(kUpdThreads), 0, stream, pending);
    return hipGetLastError();
  };
  auto close_and_pass = [&](int mn0, int Ln) -> hipError_t {
    hipError_t r;
    // one batch per sweep (M <= B): the next batch is the previous one again
    const bool shared = Lp > 0 && Ln > 0 && mp0 < mn0 + Ln && mn0 < mp0 + Lp;
    // the last fit of the previous batch is made inside the pass
    const int ml = Lp > 0 ? mp0 + Lp - 1 : 0;
    hipLaunchKernelGGL(pass, dim3((unsigned)pblocks), dim3(kPassThreads), pass_lds, stream, S, p, E, mp0, Lp,
                       (const double*)P, (const double*)bins_at(sel), (const int*)nbin_at(sel), cblocks,
                       (const double*)Gc, fit_in(ml, inner - 1), fit_out(Lp > 0 ? Lp - 1 : 0, inner - 1), ct,
                       (const double*)D64, (const uint8_t*)codes_old, (const double*)dW, mn0, Ln, X, opart, Wb,
                       shared ? 0 : Ln, bar);
    if ((r = hipGetLastError()) != hipSuccess) return r;
    if (Lp > 0) {
      pending = EcCommit{opart, pblocks, Lp, objective ? objective + 1 + nstep : nullptr, Dnew, D64, mp0, Lp, kc};
      has_pending = true;
      if ((coop || Ln == 0 || shared) && (r = launch_pending()) != hipSuccess) return r;
    }
    if (shared) {
      const size_t nrows = (size_t)Ln * Csp * Ct;
      hipLaunchKernelGGL(ec_rows_kernel, dim3((unsigned)ceil_div_z(nrows, kEcThreads)), dim3(kEcThreads), 0, stream, p,
                         (const double*)D64, (const uint8_t*)ct, mn0, Ln, Wb);
      if ((r = hipGetLastError()) != hipSuccess) return r;
    }
    nstep += Lp;
    return hipSuccess;
  };
  for (int s = 0; s < sweeps; ++s) {
    for (int m0 = 0; m0 < M; m0 += B) {
      const int L = std::min(B, M - m0);
      if ((e = close_and_pass(m0, L)) != hipSuccess) return e;
      if (coop) {
        EcSteps sb{X, Wb, Gc, D64, ct, P, dW, codes_old, bins, nbin, Dnew, Dpp, bar, fail};
        int a_m0 = m0, a_L = L, a_sel = sel;
        void* args[] = {&p, &a_m0, &a_L, &a_sel, &sb};
        if ((e = hipLaunchCooperativeKernel((const void*)steps, dim3((unsigned)cblocks), dim3(kEcThreads), args,
                                            (unsigned)prep_lds, stream)) != hipSuccess)
          return e;
        sel ^= (L * inner) & 1;
        mp0 = m0;
        Lp = L;
        continue;
      }
      for (int j = 0; j < L; ++j) {
        for (int it = 0; it < inner; ++it) {
          // the fit this step waits for: the last round of m - 1, or round it - 1 of m
          int fm = -1, fj = 0, fr = 0;
          if (it > 0) {
            fm = m0 + j;
            fj = j;
            fr = it - 1;
          } else if (j > 0) {
            fm = m0 + j - 1;
            fj = j - 1;
            fr = inner - 1;
          }
          const double* din = fm >= 0 ? fit_in(fm, fr) : D64;
          double* dout = fm >= 0 ? fit_out(fj, fr) : Dpp;
          const bool with_commit = has_pending;  // the batch's first step
          hipLaunchKernelGGL(prep, dim3((unsigned)(cblocks + (with_commit ? 1 : 0))), dim3(kEcThreads), prep_lds,
                             stream, p, m0, j, it, fm, din, (const double*)bins_at(sel), (const int*)nbin_at(sel),
                             cblocks, dout, (const double*)X, (const double*)Gc, (const double*)Wb, ct, P, dW,
                             codes_old, bins_at(sel ^ 1), nbin_at(sel ^ 1), pending);
          if ((e = hipGetLastError()) != hipSuccess) return e;
          has_pending = false;
          sel ^= 1;
        }
      }
      mp0 = m0;
      Lp = L;
    }
  }
  if (Lp > 0 && (e = close_and_pass(-1, 0)) != hipSuccess) return e;  // finish the last batch
  hipLaunchKernelGGL(ec_finish_kernel, dim3(iblocks), dim3(kEcThreads), 0, stream, (const double*)D64, p,
                     (const uint8_t*)ct, (const int*)fail, D, codes);
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
