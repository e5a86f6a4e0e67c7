// Parameter quantization on the GPU: the k-means that produces the
// sub-codebooks and codes the forward uses (Sec. 3.1, Eq. (4): per subspace,
// minimise || D^(m) B^(m) - W^(m) ||_F^2 by k-means over the sub-vectors;
// Sec. 3.2, Eq. (6): a conv layer shares D^(m) over every kernel position,
// so the k-means of subspace m runs over the sub-vectors of all (c_t, p_k)).
//
// Weights W [C_t][C_s][d_k][d_k] (FC: d_k = 1); the sub-vector i = c_t P + p
// (P = d_k^2 kernel positions) of subspace m is W[c_t][m C'_s + j][p],
// j < C'_s.  Codes [C_t][d_k][d_k][M] = [n][M], codebooks [M][K][C'_s].
//
// * Assignment (pq_assign_kernel): one thread per sub-vector, the subspace's
//   codebook in LDS (every thread reads the same sub-codeword at a time, a
//   broadcast); for a fully-connected layer pq_assign_fc_kernel reads whole
//   runs of weight rows instead (below), with the same arithmetic.  The distance is accumulated in fp32 as
//   d = fma(w_j - c_j, w_j - c_j, d) over j in order and the first minimum
//   wins, so the decision is reproducible bit for bit.  The minimum
//   distances are summed in float64 in a fixed tree order per block, then
//   per subspace (pq_objective_kernel).
// * Update (pq_update_kernel): one workgroup per subspace (XCD-major) and
//   one thread per sub-codeword.  Chunks of the subspace's sub-vectors and their codes are
//   staged in LDS with coalesced loads and sorted stably by code; thread k
//   adds the sub-vectors coded k in float64 in sub-vector order, so each mean
//   is summed in a fixed order and rounded once to fp32.  A sub-codeword that
//   no sub-vector chose keeps its value.
#include "qcnn_internal.h"

namespace qcnn {
namespace {

constexpr int kQThreads = 256;
constexpr int kMaxCsp = 16;
constexpr int kChunkFloats = 4096;  // LDS floats of staged sub-vectors per update chunk

struct QShape {
  int Ct, Cs, P, M, K, Csp;
  int n;  // sub-vectors per subspace, C_t P
};

__device__ __forceinline__ double block_sum_fixed(double v, double* red) {
  // Tree over the wave (fixed shuffle order), then the waves in order.
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_down(v, off, kWave);
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  if (lane == 0) red[wave] = v;
  __syncthreads();
  double s = 0.0;
  if (threadIdx.x == 0)
    for (int w = 0; w < (int)(blockDim.x / kWave); ++w) s += red[w];
  return s;
}

// CSP > 0: C'_s fixed at compile time (the loops over a sub-vector are
// exact); CSP = 0: any C'_s up to kMaxCsp, read at run time.
template <int CSP>
__global__ __launch_bounds__(kQThreads) void pq_assign_kernel(const float* __restrict__ W,
                                                              const float* __restrict__ D, QShape q,
                                                              uint8_t* __restrict__ codes,
                                                              double* __restrict__ part) {
  constexpr int NJ = CSP > 0 ? CSP : kMaxCsp;
  const int csp = CSP > 0 ? CSP : q.Csp;
  extern __shared__ float cb[];  // K x C'_s sub-codewords of subspace m
  __shared__ double red[kQThreads / kWave];
  const int m = blockIdx.y;
  const float* Dm = D + (size_t)m * q.K * csp;
  for (int i = threadIdx.x; i < q.K * csp; i += kQThreads) cb[i] = Dm[i];
  __syncthreads();
  const int i = blockIdx.x * kQThreads + threadIdx.x;
  double mine = 0.0;
  if (i < q.n) {
    const int t = i / q.P, p = i - t * q.P;
    const float* src = W + ((size_t)t * q.Cs + (size_t)m * csp) * q.P + p;
    float w[NJ];
#pragma unroll
    for (int j = 0; j < NJ; ++j) w[j] = j < csp ? src[(size_t)j * q.P] : 0.f;
    int best = 0;
    float bd = 0.f;
    for (int k = 0; k < q.K; ++k) {
      const float* c = cb + k * csp;
      float d = 0.f;
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        if (j < csp) {
          const float diff = w[j] - c[j];
          d = fmaf(diff, diff, d);
        }
      }
      if (k == 0 || d < bd) {
        bd = d;
        best = k;
      }
    }
    codes[(size_t)i * q.M + m] = (uint8_t)best;
    mine = (double)bd;
  }
  const double s = block_sum_fixed(mine, red);
  if (threadIdx.x == 0) part[(size_t)m * gridDim.x + blockIdx.x] = s;
}

// Assignment of a fully-connected layer (one kernel position): a workgroup
// takes kFcRows output channels x kFcSubs consecutive subspaces; thread
// (r, s) decides rows r, r + 8, ... of subspace m0 + s.  Neighbouring lanes
// read neighbouring subspaces of one weight row (kFcSubs C'_s contiguous
// floats) and write neighbouring code bytes; the sub-codewords of the
// workgroup's subspaces sit in LDS as [k][s][C'_s], so the lanes of one k
// read consecutive addresses.  The distance and the first-minimum rule are
// those of pq_assign_kernel; the minimum distances of each subspace are
// summed per workgroup in a fixed order (each thread's rows in order, then
// the 8 row groups in order) into part[m][row block].
constexpr int kFcRows = 256;
constexpr int kFcSubs = 32;

template <int CSP>
__global__ __launch_bounds__(kQThreads) void pq_assign_fc_kernel(const float* __restrict__ W,
                                                                 const float* __restrict__ D, QShape q,
                                                                 uint8_t* __restrict__ codes,
                                                                 double* __restrict__ part) {
  extern __shared__ float cbs[];  // [K][kFcSubs][C'_s]
  __shared__ double red[kQThreads / kFcSubs][kFcSubs];
  const int m0 = blockIdx.y * kFcSubs;
  const int ns = min(kFcSubs, q.M - m0);
  // staged with 16-byte loads: quad e covers (sub, k, 4 coordinates); the
  // subspaces' codebooks are contiguous in D
  static_assert(CSP % 4 == 0, "16-byte staging");
  for (int e = threadIdx.x; e < q.K * kFcSubs * (CSP / 4); e += kQThreads) {
    const int sub = e / (q.K * (CSP / 4)), r = e % (q.K * (CSP / 4)), k = r / (CSP / 4), j4 = r % (CSP / 4);
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (sub < ns) v = *reinterpret_cast<const float4*>(D + ((size_t)(m0 + sub) * q.K + k) * CSP + 4 * j4);
    *reinterpret_cast<float4*>(cbs + ((size_t)k * kFcSubs + sub) * CSP + 4 * j4) = v;
  }
  __syncthreads();
  const int sub = threadIdx.x % kFcSubs, r0 = threadIdx.x / kFcSubs;
  const int m = m0 + sub;
  double mine = 0.0;
  if (sub < ns) {
    // four rows at a time: their loads in flight together (rows past C_t read
    // row C_t - 1 and are dropped)
    constexpr int RS = kQThreads / kFcSubs;  // row stride
    for (int r = r0; r < kFcRows; r += 4 * RS) {
      float w[4][CSP];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int t = min(blockIdx.x * kFcRows + r + u * RS, q.Ct - 1);
        const float* src = W + (size_t)t * q.Cs + (size_t)m * CSP;
#pragma unroll
        for (int j4 = 0; j4 < CSP / 4; ++j4) {
          const float4 v = *reinterpret_cast<const float4*>(src + 4 * j4);
          w[u][4 * j4] = v.x;
          w[u][4 * j4 + 1] = v.y;
          w[u][4 * j4 + 2] = v.z;
          w[u][4 * j4 + 3] = v.w;
        }
      }
      int best[4] = {0, 0, 0, 0};
      float bd[4] = {0.f, 0.f, 0.f, 0.f};
      for (int k = 0; k < q.K; ++k) {
        const float* c = cbs + ((size_t)k * kFcSubs + sub) * CSP;
        float cv[CSP];
#pragma unroll
        for (int j = 0; j < CSP; ++j) cv[j] = c[j];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          float d = 0.f;
#pragma unroll
          for (int j = 0; j < CSP; ++j) {
            const float diff = w[u][j] - cv[j];
            d = fmaf(diff, diff, d);
          }
          if (k == 0 || d < bd[u]) {
            bd[u] = d;
            best[u] = k;
          }
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int t = blockIdx.x * kFcRows + r + u * RS;
        if (t < q.Ct) {
          codes[(size_t)t * q.M + m] = (uint8_t)best[u];
          mine += (double)bd[u];
        }
      }
    }
  }
  red[r0][sub] = mine;
  __syncthreads();
  if (r0 == 0 && sub < ns) {
    double v = 0.0;
    for (int g = 0; g < kQThreads / kFcSubs; ++g) v += red[g][sub];
    part[(size_t)m * gridDim.x + blockIdx.x] = v;
  }
}

// obj_m[m] = sum over the assignment blocks of subspace m, in block order.
__global__ __launch_bounds__(kQThreads) void pq_objective_kernel(const double* __restrict__ part, int nblk, int M,
                                                                 double* __restrict__ obj_m) {
  const int m = blockIdx.x * kQThreads + threadIdx.x;
  if (m >= M) return;
  double s = 0.0;
  for (int b = 0; b < nblk; ++b) s += part[(size_t)m * nblk + b];
  obj_m[m] = s;
}

// total = the sum over m of obj_m (per-thread runs in m order, then a fixed tree).
__global__ __launch_bounds__(kQThreads) void pq_total_kernel(const double* __restrict__ obj_m, int M,
                                                             double* __restrict__ total) {
  __shared__ double red[kQThreads / kWave];
  double mine = 0.0;
  for (int m = threadIdx.x; m < M; m += kQThreads) mine += obj_m[m];
  const double s = block_sum_fixed(mine, red);
  if (threadIdx.x == 0) *total = s;
}

// Update of one subspace per workgroup.  Sub-vectors are taken in chunks:
// the chunk's sub-vectors and codes are staged in LDS, a stable counting sort
// by code lists every sub-codeword's members in sub-vector order, and one
// thread per (sub-codeword k, coordinate j) then adds coordinate j of k's
// members in that order (float64, eight members' reads in flight),
// continuing its sum from the previous chunk.  The stable order comes from wave ballots: the lanes
// holding the same code are found bit by bit, a lane's rank is the number of
// such lanes below it, earlier waves of the same round and earlier rounds
// add their counts.
// Subspaces are mapped XCD-major (blocks b, b+8, ... on one XCD take
// consecutive subspaces), so the workgroups that share the cache lines of a
// weight row (neighbouring subspaces of a fully-connected layer) share an L2.
template <int CSP>
__global__ __launch_bounds__(kQThreads) void pq_update_kernel(const float* __restrict__ W,
                                                              const uint8_t* __restrict__ codes, QShape q,
                                                              float* __restrict__ D, int* __restrict__ counts) {
  constexpr int NJ = CSP > 0 ? CSP : kMaxCsp;
  __shared__ float sv[kChunkFloats];        // staged sub-vectors, [il][C'_s]
  __shared__ uint8_t sc[kChunkFloats];      // their codes
  __shared__ uint16_t perm[kChunkFloats];   // chunk positions sorted by code, stable
  __shared__ int cnt[256], start[256], run[256];
  __shared__ int wcnt[kQThreads / kWave][256];
  const int per_xcd = (q.M + 7) / 8;
  const int m = (int)(blockIdx.x & 7) * per_xcd + (int)(blockIdx.x >> 3);
  if (m >= q.M) return;  // whole workgroup, before any barrier
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int csp = CSP > 0 ? CSP : q.Csp;
  const int chunk = kChunkFloats / csp;
  // Thread tid owns the pairs (k, j) = pair tid + kQThreads u, pair = k C'_s + j
  // (at most NJ of them: K <= 256).
  double sum[NJ];
  int total[NJ];  // members of the pair's sub-codeword over all chunks
#pragma unroll
  for (int u = 0; u < NJ; ++u) {
    sum[u] = 0.0;
    total[u] = 0;
  }
  const int npairs = q.K * csp;
  for (int base = 0; base < q.n; base += chunk) {
    const int len = min(chunk, q.n - base);
    __syncthreads();  // the previous chunk is done
    {
      // Element (il, j).  Conv: j slowest, so that consecutive threads read
      // consecutive kernel positions of one input channel; FC (one position):
      // j fastest, so that they read the contiguous C'_s floats of a row.
      // Every load of the chunk is issued before any is stored.
      constexpr int EPT = kChunkFloats / kQThreads;  // elements per thread
      constexpr int CPT = (kChunkFloats + kQThreads - 1) / kQThreads;  // codes per thread (>= len / kQThreads)
      float v[EPT];
      uint8_t cv[CPT];
#pragma unroll
      for (int u = 0; u < EPT; ++u) {
        const int e = tid + u * kQThreads;
        const bool ok = e < len * csp;
        int j, il;
        if (q.P == 1) {
          il = e / csp;
          j = e - il * csp;
        } else {
          j = e / len;
          il = e - j * len;
        }
        const int i = base + il;
        const int t = i / q.P, p = i - t * q.P;
        const float x = W[ok ? ((size_t)t * q.Cs + (size_t)m * csp + j) * q.P + p : 0];
        v[u] = x;
      }
#pragma unroll
      for (int u = 0; u < CPT; ++u) {
        const int il = tid + u * kQThreads;
        const uint8_t c = codes[il < len ? (size_t)(base + il) * q.M + m : 0];
        cv[u] = c;
      }
#pragma unroll
      for (int u = 0; u < EPT; ++u) {
        const int e = tid + u * kQThreads;
        if (e < len * csp) {
          int j, il;
          if (q.P == 1) {
            il = e / csp;
            j = e - il * csp;
          } else {
            j = e / len;
            il = e - j * len;
          }
          sv[il * csp + j] = v[u];
        }
      }
#pragma unroll
      for (int u = 0; u < CPT; ++u) {
        const int il = tid + u * kQThreads;
        if (il < len) sc[il] = cv[u];
      }
    }
    for (int k = tid; k < 256; k += kQThreads) {
      cnt[k] = 0;
      run[k] = 0;
    }
    for (int k = tid; k < (kQThreads / kWave) * 256; k += kQThreads) (&wcnt[0][0])[k] = 0;
    __syncthreads();
    for (int il = tid; il < len; il += kQThreads) atomicAdd(&cnt[sc[il]], 1);  // counts: order-free
    __syncthreads();
    {  // exclusive scan of the 256 counts: within each wave, then across waves
      static_assert(kQThreads == 256, "one count per thread");
      const int own = cnt[tid];
      int incl = own;
#pragma unroll
      for (int off = 1; off < kWave; off <<= 1) {
        const int o = __shfl_up(incl, off, kWave);
        if (lane >= off) incl += o;
      }
      if (lane == kWave - 1) wcnt[wave][0] = incl;  // wave totals (wcnt is zero again below)
      __syncthreads();
      int before = 0;
      for (int w = 0; w < wave; ++w) before += wcnt[w][0];
      start[tid] = before + incl - own;
      __syncthreads();
      if (lane == kWave - 1) wcnt[wave][0] = 0;
      __syncthreads();
    }
    for (int r0 = 0; r0 < len; r0 += kQThreads) {
      const int il = r0 + tid;
      const bool valid = il < len;
      const uint32_t c = valid ? sc[il] : 0u;
      uint64_t same = __ballot(valid);
#pragma unroll
      for (int b = 0; b < 8; ++b) {
        const uint64_t ones = __ballot(valid && ((c >> b) & 1u));
        same &= ((c >> b) & 1u) ? ones : ~ones;
      }
      const int below = __popcll(same & ((1ull << lane) - 1ull));
      if (valid && below == 0) wcnt[wave][c] = __popcll(same);  // the group's lowest lane
      __syncthreads();
      if (valid) {
        int off = start[c] + run[c] + below;
        for (int w = 0; w < wave; ++w) off += wcnt[w][c];
        perm[off] = (uint16_t)il;
      }
      __syncthreads();
      for (int k = tid; k < 256; k += kQThreads) {
        int add = 0;
        for (int w = 0; w < kQThreads / kWave; ++w) {
          add += wcnt[w][k];
          wcnt[w][k] = 0;
        }
        run[k] += add;
      }
      __syncthreads();
    }
#pragma unroll
    for (int u = 0; u < NJ; ++u) {
      const int pr = tid + u * kQThreads;
      if (pr < npairs) {
        const int k = pr / csp, j = pr - k * csp;
        const int s0 = start[k], n_k = cnt[k];
        double acc = sum[u];
        int r = 0;
        for (; r + 8 <= n_k; r += 8) {  // the members' reads first, then the adds in order
          int pi[8];
          float v[8];
#pragma unroll
          for (int x = 0; x < 8; ++x) pi[x] = perm[s0 + r + x];
#pragma unroll
          for (int x = 0; x < 8; ++x) v[x] = sv[pi[x] * csp + j];
#pragma unroll
          for (int x = 0; x < 8; ++x) acc += (double)v[x];
        }
        for (; r < n_k; ++r) acc += (double)sv[perm[s0 + r] * csp + j];
        sum[u] = acc;
        total[u] += n_k;
      }
    }
  }
#pragma unroll
  for (int u = 0; u < NJ; ++u) {
    const int pr = tid + u * kQThreads;
    if (pr < npairs) {
      const int k = pr / csp, j = pr - k * csp;
      if (total[u]) D[((size_t)m * q.K + k) * csp + j] = (float)(sum[u] / (double)total[u]);
      if (counts && j == 0) counts[(size_t)m * q.K + k] = total[u];
    }
  }
}

QShape make_shape(int Ct, int Cs, int dk, int M, int K, int Csp) {
  return QShape{Ct, Cs, dk * dk, M, K, Csp, Ct * dk * dk};
}

// Assignment plus the objective reduction: obj_m ([M], may be null) and
// total (may be null); obj_tmp is room for M doubles when obj_m is null.
// True when the fully-connected assignment kernel serves this layer.
bool fc_assign(const QShape& q, const float* W, const float* D) {
  // 16-byte loads of the weight rows and codebooks: C_s and the base
  // addresses must keep every sub-vector 16-byte aligned
  return q.P == 1 && (q.Csp == 4 || q.Csp == 8) && q.Cs % 4 == 0 && ((uintptr_t)W & 15) == 0 &&
         ((uintptr_t)D & 15) == 0 && (size_t)q.K * kFcSubs * q.Csp * sizeof(float) <= 64 * 1024;
}

// Blocks per subspace of the assignment (the objective partials per subspace).
int assign_blocks(const QShape& q, bool fc) { return fc ? ceil_div(q.Ct, kFcRows) : ceil_div(q.n, kQThreads); }

hipError_t assign(const QShape& q, const float* W, const float* D, uint8_t* codes, double* part, double* obj_m,
                  double* obj_tmp, double* total, hipStream_t stream) {
  const bool fc = fc_assign(q, W, D);
  const int nblk = assign_blocks(q, fc);
  if (fc) {
    auto k = q.Csp == 4 ? pq_assign_fc_kernel<4> : pq_assign_fc_kernel<8>;
    hipLaunchKernelGGL(k, dim3((unsigned)nblk, (unsigned)ceil_div(q.M, kFcSubs)), dim3(kQThreads),
                       (size_t)q.K * kFcSubs * q.Csp * sizeof(float), stream, W, D, q, codes, part);
  } else {
    auto k = pq_assign_kernel<0>;
    if (q.Csp == 4) k = pq_assign_kernel<4>;
    else if (q.Csp == 8) k = pq_assign_kernel<8>;
    else if (q.Csp == 3) k = pq_assign_kernel<3>;
    hipLaunchKernelGGL(k, dim3((unsigned)nblk, (unsigned)q.M), dim3(kQThreads),
                       (size_t)q.K * q.Csp * sizeof(float), stream, W, D, q, codes, part);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || (!obj_m && !total)) return e;
  double* om = obj_m ? obj_m : obj_tmp;
  hipLaunchKernelGGL(pq_objective_kernel, dim3((unsigned)ceil_div(q.M, kQThreads)), dim3(kQThreads), 0, stream,
                     part, nblk, q.M, om);
  e = hipGetLastError();
  if (e != hipSuccess || !total) return e;
  hipLaunchKernelGGL(pq_total_kernel, dim3(1), dim3(kQThreads), 0, stream, om, q.M, total);
  return hipGetLastError();
}

hipError_t update(const QShape& q, const float* W, const uint8_t* codes, float* D, int* counts,
                  hipStream_t stream) {
  auto k = pq_update_kernel<0>;
  if (q.Csp == 4) k = pq_update_kernel<4>;
  else if (q.Csp == 8) k = pq_update_kernel<8>;
  else if (q.Csp == 3) k = pq_update_kernel<3>;
  const unsigned blocks = (unsigned)(ceil_div(q.M, 8) * 8);
  hipLaunchKernelGGL(k, dim3(blocks), dim3(kQThreads), 0, stream, W, codes, q, D, counts);
  return hipGetLastError();
}

// Workspace: the per-block objective partials, then M doubles.
// (room for either assignment kernel's partials)
size_t part_bytes(const QShape& q) {
  const int nb = std::max(assign_blocks(q, true), assign_blocks(q, false));
  return ((size_t)q.M * nb + q.M) * sizeof(double);
}

}  // namespace

hipError_t launch_pq_assign(int Ct, int Cs, int dk, const float* W, const float* D, int M, int K, int Csp,
                            uint8_t* codes, double* objective, hipStream_t stream) {
  const QShape q = make_shape(Ct, Cs, dk, M, K, Csp);
  Scratch scratch;
  hipError_t e = scratch.acquire(stream, part_bytes(q));
  if (e != hipSuccess) return e;
  KernelTimer timer(stream);
  double* part = reinterpret_cast<double*>(scratch.get());
  return assign(q, W, D, codes, part, objective, nullptr, nullptr, stream);
}

hipError_t launch_pq_update(int Ct, int Cs, int dk, const float* W, const uint8_t* codes, int M, int K, int Csp,
                            float* D, int* counts, hipStream_t stream) {
  const QShape q = make_shape(Ct, Cs, dk, M, K, Csp);
  KernelTimer timer(stream);
  return update(q, W, codes, D, counts, stream);
}

hipError_t launch_pq_kmeans(int Ct, int Cs, int dk, const float* W, int M, int K, int Csp, int iters, float* D,
                            uint8_t* codes, double* objective, hipStream_t stream) {
  const QShape q = make_shape(Ct, Cs, dk, M, K, Csp);
  Scratch scratch;
  hipError_t e = scratch.acquire(stream, part_bytes(q));
  if (e != hipSuccess) return e;
  double* part = reinterpret_cast<double*>(scratch.get());
  KernelTimer timer(stream);
  for (int it = 0; it <= iters && e == hipSuccess; ++it) {
    e = assign(q, W, D, codes, part, nullptr,
               part + (size_t)q.M * std::max(assign_blocks(q, true), assign_blocks(q, false)),
               objective ? objective + it : nullptr, stream);
    if (e == hipSuccess && it < iters) e = update(q, W, codes, D, nullptr, stream);
  }
  return e;
}

}  // namespace qcnn
