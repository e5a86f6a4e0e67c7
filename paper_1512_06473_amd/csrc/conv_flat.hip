// Stride-1 PQ convolution on a flattened, zero-padded image grid.
//
// Paper: Sec. 3.2, Eq. (7): each response sums, over the receptive-field
// pairs (p_k, p_s) and the subspaces m, the table entry <D^(m)_k, S^(m)_{p_s}>
// selected by the code k = k_m(c_t, p_k); the table is pre-computed over the
// input positions (paragraph after Eq. (7); Table 1 term d_s^2 C_s K).
//
// Layout.  All N images are stacked into one flat grid of width Wg = W + pad
// whose rows are the padded image rows; the right padding of a row is the
// left padding of the next one and the bottom padding of an image is the top
// padding of the next, so every halo cell is a zero shared by its neighbours.
// Output (n, yo, xo) is grid slot s = (n (H + pad) + yo) Wg + xo, and kernel
// tap (ky, kx) reads grid position s + ky Wg + kx: one uniform shift per tap.
// Slots with yo >= H_o or xo >= W_o are computed and discarded.
//
// Work split.  A tile is 252 consecutive slots: lane l of every wave owns
// the quad of slots 4l .. 4l+3 (lane 63 only supplies neighbour values; the
// next tile recomputes its slots).  For one subspace m the workgroup builds,
// in LDS, the table rows of every grid position the tile can touch,
// lut[k][0 .. P_T), with MFMA (v_mfma_f32_16x16x4_f32: 16 positions x 16
// codewords x 4 input channels per instruction).  Each wave then owns TW
// output channels; per (channel, tap) the code is a wave-uniform scalar, the
// lane reads the aligned 16-byte quad of its row at the tap's quad offset,
// and the 0..3 elements that fall past the quad come from lane l+1 through a
// DPP wave shift.  So a tap costs one ds_read_b128, one address add and four
// fp32 adds per lane, all reads are aligned and bank-conflict free.
//
// Codes are re-laid out once per call to codes8[m][t][tap] (clamped to K-1),
// so that one wave's codes for a subspace are a few contiguous dwords that
// scalar loads bring into SGPRs before the table build; the gather then needs
// one scalar extract and multiply per code.  The subspaces may be
// split over workgroups (partial sums reduced in a fixed order by a second
// kernel); blocks are mapped so that the workgroups of one tile share an XCD
// (and its L2) for the input reads of the table build.
#include <stdio.h>
#include <stdlib.h>

#include "qcnn_internal.h"

namespace qcnn {

struct FlatParams {
  int N, Cs, H, W, M, K, Csp, Ct, dk, pad, Ho, Wo;
  int Wg, Hg;            // grid width W + pad, grid rows per image H + pad
  int grid_pos;          // positions that hold input or halo: (N Hg + pad) Wg
  int tiles;             // ceil(N Hg Wg / 252)
  int PR;                // table row stride in floats (PR / 4 odd: conflict-free MFMA stores)
  int npb;               // 16-position blocks per table tile
  int tc, tblocks, splits, m_per_split;
  int work, per_xcd;
  int ct_pad;            // layout of the relaid codes: [M][ct_pad][taps] uint8
  int relu;
};

namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;
constexpr int kTileSlots = 252;
constexpr int kMaxPB = 2;   // 16-position table blocks per wave
constexpr int kMaxKB = 8;   // 16-codeword blocks (K <= 128)

typedef float f4v __attribute__((ext_vector_type(4)));

// acc += (value of v in lane l+1)
__device__ __forceinline__ void add_from_next_lane(float& acc, float v) {
  asm("v_add_f32_dpp %0, %1, %0 wave_shl:1 row_mask:0xf bank_mask:0xf" : "+v"(acc) : "v"(v));
}

template <int R>
__device__ __forceinline__ void tap_add(float (&a)[4], const f4v& q) {
  const float e[4] = {q[0], q[1], q[2], q[3]};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (j + R < 4)
      a[j] += e[j + R];
    else
      add_from_next_lane(a[j], e[j + R - 4]);
  }
}

template <int DK, int WG4, int NC, int TW>
__global__ __launch_bounds__(kThreads, 1) void conv_flat_kernel(const float* __restrict__ x,
                                                                 const float* __restrict__ D,
                                                                 const uint8_t* __restrict__ codes8,
                                                                 const float* __restrict__ bias,
                                                                 float* __restrict__ y, float* __restrict__ partial,
                                                                 FlatParams p) {
  extern __shared__ float4 lut4[];
  float* lut = reinterpret_cast<float*>(lut4);
  constexpr int TAPS = DK * DK;
  constexpr int NQ = TW * TAPS;        // table reads per wave and subspace
  constexpr int CW = (NQ + 3) / 4;     // code dwords per wave and subspace
  constexpr int PD = 8;                // table reads kept in flight
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);

  // Work item of this block, XCD-major: blocks b, b+8, b+16, ... run on one XCD.
  const int b = blockIdx.x;
  const int w = (b & 7) * p.per_xcd + (b >> 3);
  if (w >= p.work) return;
  const int per_tile = p.tblocks * p.splits;
  const int tile = w / per_tile;
  const int rem = w - tile * per_tile;
  const int tb = rem / p.splits;
  const int split = rem - tb * p.splits;
  const int s0 = tile * kTileSlots;
  const int t0 = tb * p.tc + wave * TW;
  const int m0 = split * p.m_per_split;
  const int m1 = min(p.M, m0 + p.m_per_split);
  const int HW = p.H * p.W;

  // ---- table-build operands that do not depend on m.  A operand: lane
  // supplies row l % 16 (a position) and column l / 16 (an input channel of
  // the subspace); B operand: row l / 16 (channel), column l % 16 (codeword).
  // Both are read with raw buffer loads: an offset past the buffer's end
  // returns 0, which is exactly the value of a halo position, of a channel
  // beyond C'_s and of a codeword beyond K.
  constexpr uint32_t kOOB = 0x80000000u;
  const int arow = lane & 15, acol = lane >> 4;
  // LDS byte address of this lane's quad for each tap, relative to a table row:
  // the tap shifts the quad index by (ky Wg + kx) / 4.
  uint32_t tapbase[TAPS];
#pragma unroll
  for (int tap = 0; tap < TAPS; ++tap)
    tapbase[tap] = (uint32_t)(lane + (((tap / DK) * p.Wg + (tap % DK)) >> 2)) * 16u;
  // Table row stride in bytes, held in a VGPR so that code * stride + tap
  // base is one v_mad_u32_u24 (codes < 256, strides < 2^16).
  uint32_t row_bytes = (uint32_t)p.PR * 4u;
  asm volatile("" : "+v"(row_bytes));
  // Input element (n, m C's + j, yy, xx) sits at byte ((n Cs + j) HW + yy W + xx) * 4
  // + m C's HW * 4; the subspace part goes into the scalar offset.  Only
  // the per-lane (vector) offset is range checked, so every lane whose value
  // must be 0 gets an offset past the end on its own.
  uint32_t xoff[kMaxPB][NC];
#pragma unroll
  for (int i = 0; i < kMaxPB; ++i) {
    const int pb = wave + kWaves * i;
    const int f = s0 + 16 * pb + arow;
    const int row = f / p.Wg, c = f - row * p.Wg;
    const int n = row / p.Hg, yy = row - n * p.Hg - p.pad, xx = c - p.pad;
    const bool ok = pb < p.npb && f < p.grid_pos && n < p.N && yy >= 0 && xx >= 0;
#pragma unroll
    for (int cc = 0; cc < NC; ++cc) {
      const int j = 4 * cc + acol;
      xoff[i][cc] = (ok && j < p.Csp) ? (uint32_t)((n * p.Cs + j) * HW + yy * p.W + xx) * 4u : kOOB;
    }
  }
  // Codebook entry (k, j) of subspace m sits at byte (k C's + j) * 4 of that
  // subspace's codebook; rows k >= K and channels j >= C's are past the end.
  uint32_t doff[kMaxKB][NC];
#pragma unroll
  for (int kb = 0; kb < kMaxKB; ++kb)
#pragma unroll
    for (int cc = 0; cc < NC; ++cc) {
      const int k = kb * 16 + arow, j = 4 * cc + acol;
      doff[kb][cc] = (k < p.K && j < p.Csp) ? (uint32_t)(k * p.Csp + j) * 4u : kOOB;
    }
  const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(x), 0, (int)((size_t)p.N * p.Cs * HW * 4), 0x00020000);

  float acc[TW][4];
#pragma unroll
  for (int i = 0; i < TW; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;

  const int kblocks = (p.K + 15) >> 4;
  const f4v zero4 = {0.f, 0.f, 0.f, 0.f};

  // Table-build operands, double-buffered: those of subspace m+1 are loaded
  // while the waves gather from the table of subspace m.
  float av[kMaxPB][NC], bv[kMaxKB][NC];
  auto load_operands = [&](int mm, float (&a)[kMaxPB][NC], float (&bb)[kMaxKB][NC]) {
    const __amdgpu_buffer_rsrc_t dres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(D + (size_t)mm * p.K * p.Csp), 0, p.K * p.Csp * 4, 0x00020000);
#pragma unroll
    for (int i = 0; i < kMaxPB; ++i)
#pragma unroll
      for (int c = 0; c < NC; ++c)
        a[i][c] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(xres, xoff[i][c], mm * p.Csp * HW * 4, 0));
#pragma unroll
    for (int kb = 0; kb < kMaxKB; ++kb)
#pragma unroll
      for (int c = 0; c < NC; ++c)
        bb[kb][c] = kb < kblocks ? __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(dres, doff[kb][c], 0, 0)) : 0.f;
  };
  load_operands(m0, av, bv);
  // This wave's codes for subspace m: TW x TAPS consecutive bytes, in SGPRs.
  auto load_codes = [&](int mm, uint32_t (&w)[CW]) {
    const uint32_t* ow = reinterpret_cast<const uint32_t*>(codes8 + ((size_t)mm * p.ct_pad + t0) * TAPS);
#pragma unroll
    for (int k = 0; k < CW; ++k) w[k] = ow[k];
  };
  uint32_t cw[CW];
  load_codes(m0, cw);

  for (int m = m0; m < m1; ++m) {
    __syncthreads();  // every wave is done reading the previous table
    // ---- table build: lut[k][pos] = sum_j D[m][k][j] x[pos][m C's + j]
#pragma unroll
    for (int kb = 0; kb < kMaxKB; ++kb) {
#pragma unroll
      for (int i = 0; i < kMaxPB; ++i) {
        const int pb = wave + kWaves * i;
        if (kb < kblocks && pb < p.npb) {
          f4v d = zero4;
#pragma unroll
          for (int c = 0; c < NC; ++c) d = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i][c], bv[kb][c], d, 0, 0, 0);
          // d[r] = lut[k = kb*16 + lane%16][pos = 16 pb + 4 (lane/16) + r]; rows k >= K are never read
          *reinterpret_cast<f4v*>(lut + (kb * 16 + arow) * p.PR + 16 * pb + 4 * acol) = d;
        }
      }
    }
    if (m + 1 < m1) load_operands(m + 1, av, bv);  // registers are free again after the build
    __syncthreads();
    // ---- gather-accumulate, Eq. (7).  The (channel, tap) pairs of this wave
    // form one stream of NQ table reads; PD of them are kept in flight.
    auto tap_addr = [&](int k) -> uint32_t {
      const uint32_t code = (cw[k >> 2] >> (8 * (k & 3))) & 0xffu;
      return __umul24(code, row_bytes) + tapbase[k % TAPS];
    };
    const char* lbase = reinterpret_cast<const char*>(lut4);
    f4v qb[PD];
#pragma unroll
    for (int k = 0; k < PD && k < NQ; ++k) qb[k] = *reinterpret_cast<const f4v*>(lbase + tap_addr(k));
#pragma unroll
    for (int k = 0; k < NQ; ++k) {
      const f4v q = qb[k % PD];
      if (k + PD < NQ) qb[k % PD] = *reinterpret_cast<const f4v*>(lbase + tap_addr(k + PD));
      const int i = k / TAPS, tap = k % TAPS;
      switch ((((tap / DK) * WG4) + (tap % DK)) & 3) {
        case 0: tap_add<0>(acc[i], q); break;
        case 1: tap_add<1>(acc[i], q); break;
        case 2: tap_add<2>(acc[i], q); break;
        default: tap_add<3>(acc[i], q); break;
      }
    }
    if (m + 1 < m1) load_codes(m + 1, cw);  // latency hidden by the next table build
  }

  // ---- epilogue
  if (lane == kWave - 1) return;  // its slots belong to the next tile
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int s = s0 + 4 * lane + j;
    const int row = s / p.Wg, xo = s - row * p.Wg;
    const int n = row / p.Hg, yo = row - n * p.Hg;
    if (n >= p.N || yo >= p.Ho || xo >= p.Wo) continue;
#pragma unroll
    for (int i = 0; i < TW; ++i) {
      const int t = t0 + i;
      if (t >= p.Ct) break;
      const size_t o = (((size_t)n * p.Ct + t) * p.Ho + yo) * p.Wo + xo;
      if (partial) {
        partial[(size_t)split * p.N * p.Ct * p.Ho * p.Wo + o] = acc[i][j];
      } else {
        float v = acc[i][j] + (bias ? bias[t] : 0.f);
        if (p.relu) v = fmaxf(v, 0.f);
        y[o] = v;
      }
    }
  }
}

// codes8[m][t][tap] = min(code, K-1); channels past C_t are 0.  One thread
// writes one dword (4 consecutive bytes of the [m][t][tap] order); the bytes
// it reads are scattered, but the whole code array is small and L2-resident.
__global__ __launch_bounds__(256) void flat_codes_kernel(const uint8_t* __restrict__ codes, int Ct, int taps, int M,
                                                         int K, int ct_pad, uint32_t* __restrict__ codes8) {
  const int nwords = (M * ct_pad * taps + 3) / 4;  // the plan keeps M ct_pad taps below 2^31
  const int per_m = ct_pad * taps;
  for (int wi = blockIdx.x * blockDim.x + threadIdx.x; wi < nwords; wi += gridDim.x * blockDim.x) {
    uint32_t word = 0;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int o = wi * 4 + b;
      const int m = o / per_m;
      const int r = o - m * per_m;
      const int t = r / taps, tap = r - t * taps;
      uint32_t v = 0;
      if (m < M && t < Ct) {
        v = codes[((size_t)t * taps + tap) * M + m];
        v = v < (uint32_t)(K - 1) ? v : (uint32_t)(K - 1);
      }
      word |= v << (8 * b);
    }
    codes8[wi] = word;
  }
}

// y = sum over splits in order + bias, then ReLU (y is NCHW, bias per channel).
__global__ __launch_bounds__(256) void split_reduce_kernel(const float* __restrict__ partial, int splits,
                                                           size_t total, int plane, int Ct,
                                                           const float* __restrict__ bias, int relu,
                                                           float* __restrict__ y) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  float s = partial[i];
  for (int k = 1; k < splits; ++k) s += partial[(size_t)k * total + i];
  if (bias) s += bias[(i / plane) % Ct];
  if (relu) s = fmaxf(s, 0.f);
  y[i] = s;
}

constexpr size_t kLdsMax = 160 * 1024;


struct FlatPlan {
  FlatParams p;
  int TW;
  size_t lds;
};

// Estimated cost (arbitrary units ~ CU clocks) of a plan, for the choice of
// channel block and subspace split.
double plan_cost(const FlatParams& p, int TW) {
  const double vals = 51.0;     // lookups per clock per CU (VALU bound, 1.25 ops / lookup)
  const double mfma = 256.0;    // f32 MFMA flops per clock per CU
  const int taps = p.dk * p.dk;
  const double mper = (double)p.m_per_split;
  const double gather = (double)kWaves * TW * taps * 256 / vals;
  const double build = (double)p.npb * 16 * 16 * ((p.K + 15) / 16) * 4 * ((p.Csp + 3) / 4) * 2 / mfma;
  const double per_wg = mper * (gather + build + 400.0);
  const double rounds = (double)((p.work + 255) / 256);
  double cost = rounds * per_wg;
  if (p.splits > 1) cost += (double)p.splits * 2.0 * p.N * p.Ct * p.Ho * p.Wo * 4 / 3.0e3;  // ~3 kB/clk chip-wide
  return cost;
}

bool make_plan(const ConvShape& s, FlatPlan* out) {
  if (s.stride != 1 || s.pad > s.dk - 1) return false;
  if (s.dk != 1 && s.dk != 3) return false;
  if (s.Csp > 8 || s.K > 16 * kMaxKB) return false;
  FlatParams p{};
  p.N = s.N; p.Cs = s.Cs; p.H = s.H; p.W = s.W; p.M = s.M; p.K = s.K; p.Csp = s.Csp; p.Ct = s.Ct;
  p.dk = s.dk; p.pad = s.pad; p.Ho = s.Ho; p.Wo = s.Wo;
  p.Wg = s.W + s.pad;
  p.Hg = s.H + s.pad;
  const long long slots = (long long)s.N * p.Hg * p.Wg;
  const long long gpos = ((long long)s.N * p.Hg + s.pad) * p.Wg;
  if (gpos + 4096 > (1LL << 31) || (long long)s.N * s.Cs * s.H * s.W * 4 > (1LL << 31) - 1) return false;
  p.grid_pos = (int)gpos;
  p.tiles = (int)((slots + kTileSlots - 1) / kTileSlots);
  const int dmax = (s.dk - 1) * p.Wg + (s.dk - 1);
  const int PT = 4 * (kWave + (dmax >> 2));
  const int PT16 = (PT + 15) / 16 * 16;
  p.npb = PT16 / 16;
  if (p.npb > kWaves * kMaxPB) return false;
  p.PR = (PT16 / 4) % 2 == 1 ? PT16 : PT16 + 4;
  const size_t lds = (size_t)((s.K + 15) / 16 * 16) * p.PR * sizeof(float);
  (void)kMaxKB;
  if (lds > kLdsMax) return false;
  bool found = false;
  double best = 0;
  for (int TW : {12}) {
    const int tc = kWaves * TW;
    const int tblocks = ceil_div(s.Ct, tc);
    for (int splits = 1; splits <= 16 && splits <= s.M; ++splits) {
      FlatParams q = p;
      q.tc = tc;
      q.tblocks = tblocks;
      q.m_per_split = ceil_div(s.M, splits);
      q.splits = ceil_div(s.M, q.m_per_split);
      if (q.splits != splits) continue;
      const long long work = (long long)p.tiles * tblocks * q.splits;
      if (work > (1LL << 30)) continue;
      q.work = (int)work;
      q.per_xcd = ceil_div(q.work, 8);
      q.ct_pad = tblocks * tc;
      if ((long long)s.M * q.ct_pad * s.dk * s.dk + 4 > (1LL << 31)) continue;
      const double c = plan_cost(q, TW);
      if (!found || c < best) {
        found = true;
        best = c;
        *out = {q, TW, lds};
      }
    }
  }
  return found;
}

template <int DK, int WG4, int NC, int TW>
hipError_t launch_main(const FlatPlan& pl, const float* x, const float* D, const uint8_t* codes8, const float* bias,
                       float* y, float* partial, hipStream_t stream) {
  auto k = conv_flat_kernel<DK, WG4, NC, TW>;
  hipError_t e = hipFuncSetAttribute((const void*)k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)pl.lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k, dim3(8 * pl.p.per_xcd), dim3(kThreads), pl.lds, stream, x, D, codes8, bias, y, partial, pl.p);
  return hipGetLastError();
}

template <int DK, int WG4, int NC>
hipError_t launch_tw(const FlatPlan& pl, const float* x, const float* D, const uint8_t* codes8, const float* bias,
                     float* y, float* partial, hipStream_t stream) {
  return launch_main<DK, WG4, NC, 12>(pl, x, D, codes8, bias, y, partial, stream);
}

template <int DK, int WG4>
hipError_t launch_nc(const FlatPlan& pl, const float* x, const float* D, const uint8_t* codes8, const float* bias,
                     float* y, float* partial, hipStream_t stream) {
  if (pl.p.Csp <= 4) return launch_tw<DK, WG4, 1>(pl, x, D, codes8, bias, y, partial, stream);
  return launch_tw<DK, WG4, 2>(pl, x, D, codes8, bias, y, partial, stream);
}

template <int DK>
hipError_t launch_wg(const FlatPlan& pl, const float* x, const float* D, const uint8_t* codes8, const float* bias,
                     float* y, float* partial, hipStream_t stream) {
  if constexpr (DK == 1) return launch_nc<DK, 0>(pl, x, D, codes8, bias, y, partial, stream);  // one tap: no shift
  else switch (pl.p.Wg & 3) {
    case 0: return launch_nc<DK, 0>(pl, x, D, codes8, bias, y, partial, stream);
    case 1: return launch_nc<DK, 1>(pl, x, D, codes8, bias, y, partial, stream);
    case 2: return launch_nc<DK, 2>(pl, x, D, codes8, bias, y, partial, stream);
    default: return launch_nc<DK, 3>(pl, x, D, codes8, bias, y, partial, stream);
  }
}

}  // namespace

bool conv_flat_supported(const ConvShape& s) {
  FlatPlan pl;
  return make_plan(s, &pl);
}

hipError_t launch_conv_flat(const ConvShape& s, const float* x, const float* D, const uint8_t* codes,
                            const float* bias, int relu, float* y, hipStream_t stream) {
  FlatPlan pl;
  if (!make_plan(s, &pl)) return hipErrorInvalidConfiguration;
  pl.p.relu = relu;
  static const bool trace = getenv("QCNN_TRACE_PLAN") && *getenv("QCNN_TRACE_PLAN") == '1';
  if (trace)
    fprintf(stderr, "qcnn conv_flat: tiles=%d tc=%d tblocks=%d splits=%d work=%d PR=%d npb=%d lds=%zu\n",
            pl.p.tiles, pl.p.tc, pl.p.tblocks, pl.p.splits, pl.p.work, pl.p.PR, pl.p.npb, pl.lds);
  const FlatParams& p = pl.p;
  const size_t n_codes = (size_t)p.M * p.ct_pad * p.dk * p.dk;
  const size_t out_elems = (size_t)p.N * p.Ct * p.Ho * p.Wo;
  const size_t code_bytes = (n_codes + 4 + 255) & ~(size_t)255;  // + the tail of the last dword load
  const size_t ws = code_bytes + (p.splits > 1 ? (size_t)p.splits * out_elems * sizeof(float) : 0);
  char* base = nullptr;
  hipError_t e = hipMallocAsync((void**)&base, ws, stream);
  if (e != hipSuccess) return e;
  uint8_t* codes8 = reinterpret_cast<uint8_t*>(base);
  float* partial = p.splits > 1 ? reinterpret_cast<float*>(base + code_bytes) : nullptr;
  const size_t nwords = (n_codes + 3) / 4;
  hipLaunchKernelGGL(flat_codes_kernel, dim3((unsigned)std::min<size_t>(2048, ceil_div_z(nwords, 256))), dim3(256), 0,
                     stream, codes, p.Ct, p.dk * p.dk, p.M, p.K, p.ct_pad, reinterpret_cast<uint32_t*>(codes8));
  e = hipGetLastError();
  if (e == hipSuccess) {
    KernelTimer timer(stream);
    switch (p.dk) {
      case 1: e = launch_wg<1>(pl, x, D, codes8, bias, y, partial, stream); break;
      case 3: e = launch_wg<3>(pl, x, D, codes8, bias, y, partial, stream); break;
      default: e = hipErrorInvalidConfiguration; break;
    }
  }
  if (e == hipSuccess && partial) {
    hipLaunchKernelGGL(split_reduce_kernel, dim3((unsigned)ceil_div_z(out_elems, 256)), dim3(256), 0, stream,
                       partial, p.splits, out_elems, p.Ho * p.Wo, p.Ct, bias, relu, y);
    e = hipGetLastError();
  }
  hipError_t e2 = hipFreeAsync(base, stream);
  return e == hipSuccess ? e2 : e;
}

}  // namespace qcnn
