// PQ fully-connected layer: tables of 4 subspaces per phase in LDS, 128-bit
// gathers over images.
//
// Paper: Sec. 3.1, Eq. (5) and the test-phase paragraph after it:
//     T(c_t) = sum_m < D^(m)_{k_m(c_t)}, S^(m) > = sum_m L[m][ k_m(c_t) ],
// with L[m][k] = < D^(m)_k, S^(m) > computed once per input.  Table 1: C_s K
// multiply-adds for the tables plus C_t M additions for the responses.
//
// MI355X mapping:
//   * a workgroup owns NS = 4 LPC images (64 or 128), a block of output
//     channels and a range of subspaces; per subspace its table
//     lut[k][image] (K rows of NS floats) is built in LDS by MFMA
//     (v_mfma_f32_16x16x4_f32: 16 codewords x 16 images x 4 input channels);
//   * a gather instruction serves 64 / LPC output channels: LPC lanes per
//     channel, each lane reading the 16-byte quad of 4 images of that
//     channel's table row, so every table read is one aligned ds_read_b128
//     and four fp32 adds per lane, without lane shifts;
//   * subspaces go in phases of 4 with double-buffered tables: the tables of
//     phase c+1 are built (operands loaded during the gather) while phase c
//     is gathered, one barrier per phase;
//   * the codes are re-laid out once per call to one dword per (4 subspaces,
//     channel), clamped to K-1; each lane loads the dword of its channel for
//     the next phase while the current one is gathered;
//   * the subspaces may be split over workgroups so that the chip fills: the
//     partial sums go to a stream-ordered buffer [split][channel][image] and
//     a second kernel adds them in a fixed order (deterministic), applies
//     bias and ReLU and transposes them to [image][channel] through LDS.
#include <stdio.h>
#include <stdlib.h>

#include "qcnn_internal.h"

namespace qcnn {

struct FcTParams {
  int N, Cs, M, K, Csp, Ct;
  int NS, RS;              // images per workgroup (4 LPC), table row stride in floats
  int KP;                  // table rows: K rounded up to 16
  int mgroups;             // ceil(M / 4): dword code groups
  int MC, nphases;         // subspaces per phase (4 or 8), ceil(M / MC)
  int tc, tblocks, nblocks, splits, ph_per_split;
  int work, per_xcd;
  int ct_pad;
  int relu;
};

namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;
constexpr int kNI = 8;   // gather instructions per wave and subspace

typedef float f4v __attribute__((ext_vector_type(4)));

// LPC: lanes per channel (16 or 32); NC: 4-channel groups of a subspace (1
// or 2); KB: 16-row codeword blocks (1..4); MC: subspaces per phase (4 or 8,
// i.e. one or two code dwords per channel).
template <int LPC, int NC, int KB, int MC>
__global__ __launch_bounds__(kThreads, 1) void fc_tiled_kernel(const float* __restrict__ x,
                                                               const float* __restrict__ D,
                                                               const uint32_t* __restrict__ codes4,
                                                               const float* __restrict__ bias,
                                                               float* __restrict__ y, float* __restrict__ partial,
                                                               FcTParams p) {
  extern __shared__ float4 lut4[];
  float* lut = reinterpret_cast<float*>(lut4);
  constexpr int CPI = kWave / LPC;        // channels per gather instruction
  constexpr int TW = kNI * CPI;           // channels per wave
  constexpr int NS = 4 * LPC;             // images per workgroup
  constexpr int NB = NS / 16;             // 16-image blocks
  constexpr int GPP = MC / 4;             // code dwords per channel and phase
  constexpr int TASKS = MC * NB;          // (subspace, image block) MFMA tasks per phase
  constexpr int TPW = (TASKS + kWaves - 1) / kWaves;  // tasks per wave (1 or 2)
  constexpr int PD = 8;                   // table reads kept in flight
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int g = lane / LPC, qd = lane % LPC;

  // Work item, XCD-major; the channel blocks of one (image block, split)
  // are consecutive, so they share an XCD and its L2 for x and D.
  const int b = blockIdx.x;
  const int w = (b & 7) * p.per_xcd + (b >> 3);
  if (w >= p.work) return;
  const int tb = w % p.tblocks;
  const int r0 = w / p.tblocks;
  const int split = r0 % p.splits;
  const int nblk = r0 / p.splits;
  const int n0 = nblk * NS;
  const int t0 = tb * p.tc + wave * TW;
  const int ph0 = split * p.ph_per_split;
  const int ph1 = min(p.nphases, ph0 + p.ph_per_split);

  constexpr uint32_t kOOB = 0x80000000u;
  const int arow = lane & 15, acol = lane >> 4;
  const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(x), 0, (int)((size_t)p.N * p.Cs * 4), 0x00020000);
  const __amdgpu_buffer_rsrc_t dres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(D), 0, (int)((size_t)p.M * p.K * p.Csp * 4), 0x00020000);
  const int tbuf = p.KP * p.RS;  // floats per subspace table

  // ---- build operands of phase ph (subspaces ph MC ..): task k of this
  // wave is (subspace ml, image block nb) = ((wave + 16 k) / NB, % NB).
  // A operand (x): image n0 + 16 nb + l % 16, channel m C's + 4 c + l / 16;
  // B operand (D): codeword 16 kb + l % 16 of subspace m, channel 4 c + l / 16.
  // Offsets past a buffer's end (image >= N, channel >= C's, codeword >= K,
  // subspace >= M) read 0.
  float av[TPW][NC], bv[TPW][KB][NC];
  auto load_ops = [&](int ph) {
#pragma unroll
    for (int k = 0; k < TPW; ++k) {
      const int task = wave + kWaves * k;
      const int ml = task / NB, nb = task - ml * NB;
      const int m = ph * MC + ml;
      const bool mok = task < TASKS && m < p.M;
      const int n = n0 + nb * 16 + arow;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int j = 4 * c + acol;
        const bool ok = mok && n < p.N && j < p.Csp;
        const uint32_t off = ok ? (uint32_t)(((size_t)n * p.Cs + (size_t)m * p.Csp + j) * 4) : kOOB;
        av[k][c] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(xres, off, 0, 0));
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
          const int kk = kb * 16 + arow;
          const bool okd = mok && kk < p.K && j < p.Csp;
          const uint32_t offd = okd ? (uint32_t)((((size_t)m * p.K + kk) * p.Csp + j) * 4) : kOOB;
          bv[k][kb][c] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(dres, offd, 0, 0));
        }
      }
    }
  };
  // MFMA with the codebook as the A operand: d[r] = table value of codeword
  // 16 kb + 4 (l / 16) + r at image 16 nb + l % 16.  Each 32-bit store then
  // writes 16 consecutive images of one row per 16-lane group (rows whose
  // stride is a multiple of 256 bytes would make a 16-rows-per-store layout
  // conflict 16 ways).
  auto build = [&](int buf) {
#pragma unroll
    for (int k = 0; k < TPW; ++k) {
      const int task = wave + kWaves * k;
      if (task < TASKS) {
        const int ml = task / NB, nb = task - ml * NB;
        float* base = lut + (buf * MC + ml) * tbuf + nb * 16 + arow;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
          f4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int c = 0; c < NC; ++c) d = __builtin_amdgcn_mfma_f32_16x16x4f32(bv[k][kb][c], av[k][c], d, 0, 0, 0);
#pragma unroll
          for (int r = 0; r < 4; ++r) base[(kb * 16 + 4 * acol + r) * p.RS] = d[r];
        }
      }
    }
  };
  // Codes of a phase: instruction i serves channel t0 + i CPI + g; dword gg
  // holds that channel's codes of the phase's subspaces 4 gg .. 4 gg + 3.
  uint32_t cur[GPP][kNI], nxt[GPP][kNI];
  auto load_codes = [&](int ph, uint32_t (&dst)[GPP][kNI]) {
#pragma unroll
    for (int gg = 0; gg < GPP; ++gg) {
      const uint32_t* src = codes4 + (size_t)(ph * GPP + gg) * p.ct_pad + t0 + g;
#pragma unroll
      for (int i = 0; i < kNI; ++i) dst[gg][i] = src[i * CPI];
    }
  };

  float acc[kNI][4];
#pragma unroll
  for (int i = 0; i < kNI; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[i][r] = 0.f;

  // Row stride in bytes in a VGPR: address = code * stride + base is one v_mad_u32_u24.
  uint32_t row_bytes = (uint32_t)p.RS * 4u;
  asm volatile("" : "+v"(row_bytes));
  const uint32_t lane_off = (uint32_t)qd * 16u;
  const char* lbase = reinterpret_cast<const char*>(lut4);

  if (ph0 < ph1) {
    load_ops(ph0);
    load_codes(ph0, cur);
    build(0);
    // Settle the first codes here: the loop below is entered with no load
    // pending on them, so its start does not wait for the next phase's loads
    // (the load counter is in order).
#pragma unroll
    for (int gg = 0; gg < GPP; ++gg)
#pragma unroll
      for (int i = 0; i < kNI; ++i) asm volatile("" : "+v"(cur[gg][i]));
  }
  int buf = 0;
  for (int ph = ph0; ph < ph1; ++ph) {
    const bool more = ph + 1 < ph1;
    if (more) {
      load_ops(ph + 1);
      load_codes(ph + 1, nxt);
    }
    __syncthreads();  // tables of this phase are complete; the other buffer is free
    // ---- gather, Eq. (5): MC subspaces x kNI instructions
#pragma unroll
    for (int ml = 0; ml < MC; ++ml) {
      if (ph * MC + ml >= p.M) break;  // the last phase may hold fewer subspaces
      const uint32_t tb_off = (uint32_t)((buf * MC + ml) * tbuf) * 4u + lane_off;
      f4v qb[PD];
      auto addr = [&](int i) -> uint32_t {
        const uint32_t code = (cur[ml >> 2][i] >> (8 * (ml & 3))) & 0xffu;
        return __umul24(code, row_bytes) + tb_off;
      };
#pragma unroll
      for (int i = 0; i < PD && i < kNI; ++i) qb[i] = *reinterpret_cast<const f4v*>(lbase + addr(i));
#pragma unroll
      for (int i = 0; i < kNI; ++i) {
        const f4v q = qb[i % PD];
        if (i + PD < kNI) qb[i % PD] = *reinterpret_cast<const f4v*>(lbase + addr(i + PD));
        acc[i][0] += q[0];
        acc[i][1] += q[1];
        acc[i][2] += q[2];
        acc[i][3] += q[3];
      }
    }
    if (more) {
      build(buf ^ 1);
#pragma unroll
      for (int gg = 0; gg < GPP; ++gg)
#pragma unroll
        for (int i = 0; i < kNI; ++i) {
          cur[gg][i] = nxt[gg][i];
          asm volatile("" : "+v"(cur[gg][i]));
        }
    }
    buf ^= 1;
  }

  // ---- epilogue: lane holds images n0 + 4 qd + r of channel t0 + i CPI + g
#pragma unroll
  for (int i = 0; i < kNI; ++i) {
    const int t = t0 + i * CPI + g;
    if (partial) {
      float* dst = partial + ((size_t)split * p.ct_pad + t) * (size_t)(p.nblocks * NS) + n0 + 4 * qd;
#pragma unroll
      for (int r = 0; r < 4; ++r) dst[r] = acc[i][r];
    } else if (t < p.Ct) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int n = n0 + 4 * qd + r;
        if (n < p.N) {
          float v = acc[i][r] + (bias ? bias[t] : 0.f);
          if (p.relu) v = fmaxf(v, 0.f);
          y[(size_t)n * p.Ct + t] = v;
        }
      }
    }
  }
}

// codes4[gq][t] = the codes of subspaces 4 gq .. 4 gq + 3 of channel t, one
// byte each (clamped to K-1; subspaces past M and channels past C_t give 0).
// A transpose of [C_t][M] bytes into [M / 4][ct_pad] dwords through LDS:
// a 64 (t) x 64 (gq) tile per workgroup, read along the subspaces, written
// along the channels.
__global__ __launch_bounds__(256) void fc_codes_kernel(CodeStream codes, int Ct, int M, int K,
                                                       int mgroups, int ct_pad, uint32_t* __restrict__ codes4) {
  __shared__ uint32_t tile[64][65];
  const int gq0 = blockIdx.x * 64, tt0 = blockIdx.y * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;  // 64 x 4
  const uint32_t kmax = (uint32_t)(K - 1);
  // All 16 loads of a thread are issued before its first LDS store (one
  // load latency per workgroup instead of 16).
  uint32_t words[16];
  // One byte per code and M % 4 == 0: every row starts 4-byte aligned (so
  // does the caller's array) and a dword holds the 4 codes of a group.
  const bool aligned = codes.bits == 8 && (M & 3) == 0;
  const int gq = gq0 + tx;
  // Groups past the last subspace (mgroups rounds M up to whole phases) hold
  // no code: nothing of the caller's array is read for them.
  const bool has_codes = gq < mgroups && 4 * gq < M;
  if (aligned) {
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) {
      const int t = tt0 + ty + 4 * rr;
      words[rr] = (t < Ct && has_codes) ? *reinterpret_cast<const uint32_t*>(codes.p + (size_t)t * M + 4 * gq) : 0u;
    }
  } else if (codes.bits == 8) {
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) {
      const int t = tt0 + ty + 4 * rr;
      uint32_t word = 0;
      if (t < Ct && has_codes) {
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (4 * gq + k < M) word |= code_at(codes, (size_t)t * M + 4 * gq + k) << (8 * k);
      }
      words[rr] = word;
    }
  } else {
    // Packed codes: the group's (up to) 4 codes are 4 b <= 28 consecutive
    // stream bits, read as one 64-bit window of two aligned dwords (the
    // second only when the bits reach into it, so it is inside the stream).
    const uint32_t* w = reinterpret_cast<const uint32_t*>(codes.p);
    const int b = codes.bits;
    const uint32_t mask = b ? (1u << b) - 1u : 0u;
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) {
      const int t = tt0 + ty + 4 * rr;
      uint32_t word = 0;
      if (t < Ct && has_codes && b > 0) {
        const int n = min(4, M - 4 * gq);  // >= 1 here
        const size_t bit = ((size_t)t * M + 4 * gq) * (size_t)b;
        const uint32_t sh = (uint32_t)(bit & 31);
        uint64_t win = w[bit >> 5];
        if (sh + (uint32_t)(n * b) > 32u) win |= (uint64_t)w[(bit >> 5) + 1] << 32;
        win >>= sh;
        for (int k = 0; k < n; ++k) word |= (uint32_t)((win >> (k * b)) & mask) << (8 * k);
      }
      words[rr] = word;
    }
  }
#pragma unroll
  for (int rr = 0; rr < 16; ++rr) {
    uint32_t out = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint32_t c = (words[rr] >> (8 * k)) & 0xffu;
      out |= (c < kmax ? c : kmax) << (8 * k);
    }
    tile[ty + 4 * rr][tx] = out;
  }
  __syncthreads();
#pragma unroll
  for (int rr = 0; rr < 16; ++rr) {
    const int r = ty + 4 * rr;
    const int gq = gq0 + r, t = tt0 + tx;
    if (gq < mgroups && t < ct_pad) codes4[(size_t)gq * ct_pad + t] = tile[tx][r];
  }
}

// y[n][t] = sum over splits (in split order) of partial[split][t][n] + bias,
// then ReLU.  A 64 (t) x 64 (n) tile per 1024-thread workgroup: read along
// n with the loads of 4 splits x 4 rows in flight per thread, transposed
// through LDS, written along t.
__global__ __launch_bounds__(1024) void fc_tiled_reduce_kernel(const float* __restrict__ partial, FcTParams p,
                                                               const float* __restrict__ bias,
                                                               float* __restrict__ y) {
  __shared__ float tile[64][65];
  const int NT = p.nblocks * p.NS;
  const int tt0 = blockIdx.y * 64, nn0 = blockIdx.x * 64;
  const size_t split_stride = (size_t)p.ct_pad * NT;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;  // 64 x 16
  const int n = nn0 + tx;
  float s[4] = {0.f, 0.f, 0.f, 0.f};
  bool rok[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) rok[k] = n < NT && tt0 + ty + 16 * k < p.ct_pad;
  const float* src = partial + (size_t)(tt0 + ty) * NT + n;
  int sp = 0;
  for (; sp + 4 <= p.splits; sp += 4) {
    float v[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int k = 0; k < 4; ++k)
        v[u][k] = rok[k] ? src[(size_t)(sp + u) * split_stride + (size_t)16 * k * NT] : 0.f;
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int k = 0; k < 4; ++k) s[k] += v[u][k];
  }
  for (; sp < p.splits; ++sp)
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (rok[k]) s[k] += src[(size_t)sp * split_stride + (size_t)16 * k * NT];
#pragma unroll
  for (int k = 0; k < 4; ++k) tile[ty + 16 * k][tx] = s[k];
  __syncthreads();
  const int t = tt0 + tx;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int nn = nn0 + ty + 16 * k;
    if (nn < p.N && t < p.Ct) {
      float v = tile[tx][ty + 16 * k] + (bias ? bias[t] : 0.f);
      if (p.relu) v = fmaxf(v, 0.f);
      y[(size_t)nn * p.Ct + t] = v;
    }
  }
}

struct FcPlan {
  FcTParams p;
  int LPC, NC, KB;
  size_t lds;
};

double fc_cost(const FcTParams& p, int LPC) {
  const int CPI = kWave / LPC;
  const double vals = 40.0;  // table values gathered per clock per CU
  const double gather = (double)kWaves * kNI * kWave * 4 / vals;             // per subspace
  const double build = (double)p.NS * p.KP * 4 * ((p.Csp + 3) / 4) * 2 / 256.0;  // MFMA flops / 256 per clock
  const double per_wg = (double)p.ph_per_split * (p.MC * (gather + build) + 800.0);
  const double rounds = (double)((p.work + 255) / 256);
  double cost = rounds * per_wg;
  if (p.splits > 1) cost += (double)p.splits * 2.0 * p.ct_pad * p.nblocks * p.NS * 4 / 2.0e3;
  (void)CPI;
  return cost;
}

bool make_fc_plan(int N, int Cs, int M, int K, int Csp, int Ct, FcPlan* out) {
  if (K > 64 || Csp > 8) return false;
  if ((long long)N * Cs * 4 > (1LL << 31) - 1 || (long long)M * K * Csp * 4 > (1LL << 31) - 1) return false;
  bool found = false;
  double best = 0;
  for (int LPC : {16, 32})
  for (int MC : {4, 8}) {
    const int NS = 4 * LPC;
    if (LPC == 32 && (K > 32 || N <= 64)) continue;
    FcTParams p{};
    p.N = N; p.Cs = Cs; p.M = M; p.K = K; p.Csp = Csp; p.Ct = Ct;
    p.NS = NS;
    // Rows a multiple of 256 bytes apart: every 16-lane group of a gather
    // then reads one aligned 256-byte run, which the LDS serves at full
    // rate even when the groups read different rows (rows offset by other
    // amounts cost about 40 %).
    p.RS = NS;
    p.KP = (K + 15) / 16 * 16;
    p.MC = MC;
    p.nphases = ceil_div(M, MC);
    p.mgroups = p.nphases * (MC / 4);  // code dwords per channel, whole phases
    const size_t lds = (size_t)2 * MC * p.KP * p.RS * sizeof(float);
    if (lds > kLdsBytes || (MC == 8 && (LPC != 16 || p.KP > 32))) continue;
    p.tc = kWaves * kNI * (kWave / LPC);
    p.tblocks = ceil_div(Ct, p.tc);
    p.nblocks = ceil_div(N, NS);
    p.ct_pad = p.tblocks * p.tc;
    if ((long long)p.nblocks * NS * p.ct_pad * 16 > (1LL << 40)) continue;
    for (int splits = 1; splits <= 64 && splits <= p.nphases; ++splits) {
      FcTParams q = p;
      q.ph_per_split = ceil_div(p.nphases, splits);
      q.splits = ceil_div(p.nphases, q.ph_per_split);
      if (q.splits != splits) continue;
      const long long work = (long long)p.nblocks * p.tblocks * q.splits;
      if (work > (1LL << 30)) continue;
      q.work = (int)work;
      q.per_xcd = ceil_div(q.work, 8);
      const double c = fc_cost(q, LPC);
      if (!found || c < best) {
        found = true;
        best = c;
        *out = {q, LPC, Csp <= 4 ? 1 : 2, p.KP / 16, lds};
      }
    }
  }
  return found;
}

template <int LPC, int NC, int KB>
hipError_t launch_t(const FcPlan& pl, const float* x, const float* D, const uint32_t* codes4, const float* bias,
                    float* y, float* partial, hipStream_t stream, LaunchTimer* timer) {
  auto k = fc_tiled_kernel<LPC, NC, KB, 4>;
  if constexpr (LPC == 16 && KB <= 2) {  // the only tables small enough for 8 subspaces per phase
    if (pl.p.MC == 8) k = fc_tiled_kernel<LPC, NC, KB, 8>;
  }
  hipError_t e = allow_max_lds((const void*)k);
  if (e != hipSuccess) return e;
  return timed_launch(timer, k, dim3(8 * pl.p.per_xcd), dim3(kThreads), (uint32_t)pl.lds, stream, x, D, codes4, bias, y,
                      partial, pl.p);
}

template <int LPC, int NC>
hipError_t launch_kb(const FcPlan& pl, const float* x, const float* D, const uint32_t* codes4, const float* bias,
                     float* y, float* partial, hipStream_t stream, LaunchTimer* timer) {
  switch (pl.KB) {
    case 1: return launch_t<LPC, NC, 1>(pl, x, D, codes4, bias, y, partial, stream, timer);
    case 2: return launch_t<LPC, NC, 2>(pl, x, D, codes4, bias, y, partial, stream, timer);
    case 3: return launch_t<LPC, NC, 3>(pl, x, D, codes4, bias, y, partial, stream, timer);
    default: return launch_t<LPC, NC, 4>(pl, x, D, codes4, bias, y, partial, stream, timer);
  }
}

}  // namespace

bool fc_tiled_supported(int N, int Cs, int M, int K, int Csp, int Ct) {
  FcPlan pl;
  return make_fc_plan(N, Cs, M, K, Csp, Ct, &pl);
}

namespace {

bool fc_plan(int N, int Cs, int M, int K, int Csp, int Ct, int relu, FcPlan* pl) {
  if (!make_fc_plan(N, Cs, M, K, Csp, Ct, pl)) return false;
  pl->p.relu = relu;
  static const bool trace = getenv("QCNN_TRACE_PLAN") && *getenv("QCNN_TRACE_PLAN") == '1';
  if (trace)
    fprintf(stderr, "qcnn fc_tiled: LPC=%d NC=%d KB=%d MC=%d NS=%d tc=%d tblocks=%d nblocks=%d splits=%d "
            "phases/split=%d work=%d lds=%zu\n", pl->LPC, pl->NC, pl->KB, pl->p.MC, pl->p.NS, pl->p.tc,
            pl->p.tblocks, pl->p.nblocks, pl->p.splits, pl->p.ph_per_split, pl->p.work, pl->lds);
  return true;
}

size_t code_bytes_of(const FcTParams& p) { return ((size_t)p.mgroups * p.ct_pad * 4 + 255) & ~(size_t)255; }

hipError_t launch_codes(const FcTParams& p, CodeStream codes, int Ct, int M, int K, uint32_t* codes4,
                        hipStream_t stream) {
  hipLaunchKernelGGL(fc_codes_kernel, dim3((unsigned)ceil_div(p.mgroups, 64), (unsigned)ceil_div(p.ct_pad, 64)),
                     dim3(256), 0, stream, codes, Ct, M, K, p.mgroups, p.ct_pad, codes4);
  return hipGetLastError();
}

// The kernels of a call after the code re-layout: the main kernel, then (split
// plans) the split sum.
hipError_t run_fc(const FcPlan& pl, const float* x, const float* D, const uint32_t* codes4, const float* bias,
                  float* y, float* partial, hipStream_t stream) {
  const FcTParams& p = pl.p;
  hipError_t e;
  {
    LaunchTimer timer;
    if (pl.LPC == 16)
      e = pl.NC == 1 ? launch_kb<16, 1>(pl, x, D, codes4, bias, y, partial, stream, &timer)
                     : launch_kb<16, 2>(pl, x, D, codes4, bias, y, partial, stream, &timer);
    else
      e = pl.NC == 1 ? launch_kb<32, 1>(pl, x, D, codes4, bias, y, partial, stream, &timer)
                     : launch_kb<32, 2>(pl, x, D, codes4, bias, y, partial, stream, &timer);
  }
  if (e == hipSuccess && partial) {
    const int NT = p.nblocks * p.NS;
    hipLaunchKernelGGL(fc_tiled_reduce_kernel, dim3((unsigned)ceil_div(NT, 64), (unsigned)ceil_div(p.ct_pad, 64)),
                       dim3(1024), 0, stream, partial, p, bias, y);
    e = hipGetLastError();
  }
  return e;
}

size_t partial_bytes_of(const FcTParams& p) {
  return p.splits > 1 ? (size_t)p.splits * p.ct_pad * p.nblocks * p.NS * sizeof(float) : 0;
}

}  // namespace

hipError_t launch_fc_tiled(int N, int Cs, int M, int K, int Csp, int Ct, const float* x, const float* D,
                           CodeStream codes, const float* bias, int relu, float* y, hipStream_t stream) {
  FcPlan pl;
  if (!fc_plan(N, Cs, M, K, Csp, Ct, relu, &pl)) return hipErrorInvalidConfiguration;
  const size_t code_bytes = code_bytes_of(pl.p);
  Scratch scratch;
  hipError_t e = scratch.acquire(stream, code_bytes + partial_bytes_of(pl.p));
  if (e != hipSuccess) return e;
  char* base = scratch.get();
  uint32_t* codes4 = reinterpret_cast<uint32_t*>(base);
  float* partial = pl.p.splits > 1 ? reinterpret_cast<float*>(base + code_bytes) : nullptr;
  e = launch_codes(pl.p, codes, Ct, M, K, codes4, stream);
  if (e != hipSuccess) return e;
  return run_fc(pl, x, D, codes4, bias, y, partial, stream);
}

size_t fc_tiled_code_bytes(int N, int Cs, int M, int K, int Csp, int Ct) {
  FcPlan pl;
  return make_fc_plan(N, Cs, M, K, Csp, Ct, &pl) ? code_bytes_of(pl.p) : 0;
}

hipError_t launch_fc_tiled_codes(int N, int Cs, int M, int K, int Csp, int Ct, CodeStream codes, uint32_t* codes4,
                                 hipStream_t stream) {
  FcPlan pl;
  if (!make_fc_plan(N, Cs, M, K, Csp, Ct, &pl)) return hipErrorInvalidConfiguration;
  return launch_codes(pl.p, codes, Ct, M, K, codes4, stream);
}

hipError_t launch_fc_tiled_relaid(int N, int Cs, int M, int K, int Csp, int Ct, const float* x, const float* D,
                                  const uint32_t* codes4, const float* bias, int relu, float* y,
                                  hipStream_t stream) {
  FcPlan pl;
  if (!fc_plan(N, Cs, M, K, Csp, Ct, relu, &pl)) return hipErrorInvalidConfiguration;
  const size_t part = partial_bytes_of(pl.p);
  Scratch scratch;
  hipError_t e = scratch.acquire(stream, part);
  if (e != hipSuccess) return e;
  return run_fc(pl, x, D, codes4, bias, y, part ? reinterpret_cast<float*>(scratch.get()) : nullptr, stream);
}

}  // namespace qcnn
