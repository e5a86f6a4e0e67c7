// PQ convolution on a flattened image grid, with the table in LDS.
//
// Paper: Sec. 3.2, Eq. (7): each response sums, over the receptive-field
// pairs (p_k, p_s) and the subspaces m, the table entry <D^(m)_k, S^(m)_{p_s}>
// selected by the code k = k_m(c_t, p_k); the table is pre-computed over the
// input positions (paragraph after Eq. (7); Table 1 term d_s^2 C_s K).
//
// Layout.  The output maps are stacked into one flat grid of width Wg; grid
// slot s = ((n S + strip) Hg + yo) Wg + xl holds output (n, yo, strip sw + xl)
// (S column strips of sw outputs per image; S = 1 for maps that fit).
//
// Virtual subspaces.  The sum of Eq. (7) is split into pieces that are each
// a stride-1 correlation with a small ROWS x COLS tap grid on that layout:
//   * stride s: a kernel tap (ky, kx) = (s u + a, s v + b) reads input
//     (s (yo + u) + a - pad, s (xo + v) + b - pad), so for a fixed phase
//     (a, b) the tap is a shift (u, v) of the output slot over a table built
//     at the phase's input positions;
//   * large kernels: the kernel rows are cut into G groups of ROWS rows, and
//     group g's table is built at input rows shifted by s g ROWS.
// A virtual subspace v = (m, a, b, g) has its own table (subspace m's
// codewords against the inputs it samples); its taps are the ROWS x COLS
// grid (u', v') with kernel tap ky = s (g ROWS + u') + a, kx = s v' + b, and
// grid entries past the kernel read a row of zeros.  Tap (u', v') of slot s
// reads table position s + u' Wg + v': one uniform shift per tap.
// For stride 1 with ROWS <= the rows the halo absorbs, neighbouring images
// share their zero halo (Wg = W + pad, Hg = H + pad: the right padding of a
// row is the left padding of the next one); otherwise each image keeps its
// own margin (Hg = H_o + ROWS - 1, Wg = sw + COLS - 1) and every table value
// comes from its own coordinates.
//
// Work split.  A tile is 252 consecutive slots: lane l of every wave owns
// the quad of slots 4l .. 4l+3 (lane 63 only supplies neighbour values; the
// next tile recomputes its slots).  For one virtual subspace the workgroup
// builds, in LDS, the table rows of every position the tile can touch,
// lut[k][0 .. P_T), with MFMA (v_mfma_f32_16x16x4_f32: 16 positions x 16
// codewords x 4 input channels per instruction).  Each wave then owns TW
// output channels; per (channel, tap) the code is a wave-uniform scalar, the
// lane reads the aligned 16-byte quad of its row at the tap's quad offset,
// and the 0..3 elements that fall past the quad come from lane l+1 through a
// DPP wave shift.  So a tap costs one ds_read_b128, one address
// multiply-add and four fp32 adds per lane, all reads are aligned and
// bank-conflict free.
//
// Codes are re-laid out (once per call, or once per prepared plan) to
// codes8[v][t][tap] (clamped to K-1, the zero row for grid taps past the
// kernel; each channel's taps padded to a stride that keeps every wave's run
// dword aligned), so that one wave's codes for a virtual subspace are a few
// contiguous dwords that scalar loads bring into SGPRs during the table
// build.  The virtual subspaces may be split over
// workgroups: each then stores its partial sums tile by tile (whole cache
// lines per store instruction) and a second kernel adds them in a fixed
// order.  Blocks are mapped so that the workgroups of one tile share an XCD
// (and its L2) for the input reads of the table build.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "qcnn_internal.h"

namespace qcnn {

struct FlatParams {
  int N, Cs, H, W, M, K, Csp, Ct, dk, stride, pad, Ho, Wo;
  int S, sw;             // column strips per image, output columns per strip (S = 1: sw = W_o)
  int Wg, Hg;            // grid width, grid rows per image
  int grid_pos;          // grid positions that may hold input (beyond: zero)
  int tiles;             // ceil(N S Hg Wg / 252)
  int G, V;              // kernel-row groups; virtual subspaces M s^2 G
  int zrow;              // table row of zeros for grid taps past the kernel, or -1
  int dstage;            // float offset in LDS of the staged codebook (after the table)
  int PR;                // table row stride in floats (PR / 4 odd: conflict-free MFMA stores)
  int npb;               // 16-position blocks per table tile
  int tc, tblocks, splits, v_per_split;
  int work, per_xcd;
  int ct_pad;            // layout of the relaid codes: [V][ct_pad][taps] uint8
  int relu;
};

namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;
constexpr int kTileSlots = 252;
constexpr int kMaxPB = 2;   // 16-position table blocks per wave
constexpr int kMaxKB = 8;   // 16-codeword blocks (K <= 128)

typedef float f4v __attribute__((ext_vector_type(4)));

// Bytes per channel of the re-laid codes: the tap count, padded so that a
// wave's run of TW channels is a whole number of dwords (a wave reads its
// codes with scalar dword loads, whose addresses must be 4-byte aligned;
// every run starts at a multiple of TW channels).
__host__ __device__ constexpr int code_stride(int TW, int taps) {
  int c = taps;
  while ((TW * c) % 4 != 0) ++c;
  return c;
}

// acc += (value of v in lane l+1): a wave_shl:1 DPP move the compiler folds
// into the add (v_add_f32_dpp), with the wait states a DPP read needs after a
// VALU write inserted by the compiler.  Lane 63 gets 0 (bound_ctrl off and
// old value 0); its slots belong to the next tile and are never stored.
__device__ __forceinline__ void add_from_next_lane(float& acc, float v) {
  acc += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x130, 0xf, 0xf, false));
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

// Kernel rows ky = s u + a (u = 0, 1, ...) of stride phase a.
__device__ __forceinline__ int s_rows_in_kernel(const FlatParams& p, int a) {
  return (p.dk - a + p.stride - 1) / p.stride;
}

// Gather-accumulate of Eq. (7) over one virtual subspace's table: the
// (channel, tap) pairs of a wave form one stream of table reads, PD of them
// kept in flight.  Per read: the code byte (a scalar), one address
// multiply-add, one 128-bit LDS read and four adds.  LAST_ROW_AT_END: the
// taps of the grid's last row come at the end of the stream (every channel's
// other rows first), and the stream stops before them when that row lies past
// the kernel (the last row group, or a stride phase with fewer rows: those
// taps would read the zero row); only the PD reads already in flight are
// spent on it.  The stream is unrolled by template recursion (a counted loop
// this long exceeds the compiler's unroll limit).  PRIO: a
// wave steps its issue priority down along its stream, 3 for the first 5/8
// of its reads, 2 until 13/16, 1 until 15/16, then the base level, so that
// waves ahead of the others yield the SIMD to the ones behind and the waves
// of a workgroup finish their gathers closer together (the last ones alone
// do not keep the LDS busy).  Measured on the AlexNet conv3 layer against
// other schedules: one drop from 1 to 0 at 3/4 gave a 2 % longer kernel,
// a single drop at 7/8 4 % longer, steps that start at 3/4 2 % longer, and
// steps that start at 1/4 or 1/2 up to 3 % longer.  With LAST_ROW_AT_END the
// steps span the reads before the last row (AlexNet conv2: 593 -> 587 us
// with the pooled split sum).  Only for a workgroup that has its CU to
// itself: beside a second workgroup, the priority starves that one's table
// build.
template <int ROWS, int COLS, int TW, int CW, bool LAST_ROW_AT_END, bool PRIO>
struct GatherStream {
  static constexpr int TAPS = ROWS * COLS;
  static constexpr int NS = TW * TAPS;
  static constexpr int B = LAST_ROW_AT_END ? TW * (ROWS - 1) * COLS : NS;  // first read of the last row
  // stream position k -> (channel, tap) index of the full tap grid
  static constexpr int full(int k) {
    if (k < B) {
      constexpr int per = LAST_ROW_AT_END ? (ROWS - 1) * COLS : TAPS;
      return (k / per) * TAPS + k % per;
    }
    return ((k - B) / COLS) * TAPS + (ROWS - 1) * COLS + (k - B) % COLS;
  }

  const uint32_t (&cw)[CW];
  const uint32_t (&tapbase)[TAPS];
  uint32_t row_bytes;
  const char* lbase;
  bool last_row;  // read the last row's taps

  static constexpr int CS = code_stride(TW, TAPS);

  template <int KF>
  __device__ __forceinline__ f4v read() const {
    constexpr int cb = (KF / TAPS) * CS + KF % TAPS;  // byte of the code in the wave's run
    const uint32_t code = (cw[cb >> 2] >> (8 * (cb & 3))) & 0xffu;
    return *reinterpret_cast<const f4v*>(lbase + __umul24(code, row_bytes) + tapbase[KF % TAPS]);
  }

  template <int K, int WG4, int PD>
  __device__ __forceinline__ void step(float (&acc)[TW][4], f4v (&qb)[PD]) const {
    if constexpr (K < NS) {
      // With an early stop the steps run over the reads before it (steps
      // placed after it made the compiler spill 66-160 registers).
      constexpr int PN = LAST_ROW_AT_END ? B : NS;
      if constexpr (PRIO && K == 0) __builtin_amdgcn_s_setprio(3);
      if constexpr (PRIO && K == (5 * PN) / 8) __builtin_amdgcn_s_setprio(2);
      if constexpr (PRIO && K == (13 * PN) / 16) __builtin_amdgcn_s_setprio(1);
      if constexpr (PRIO && K == (15 * PN) / 16) __builtin_amdgcn_s_setprio(0);
      if constexpr (K == B) {
        if (!last_row) return;  // wave-uniform
      }
      const f4v q = qb[K % PD];
      if constexpr (K + PD < NS) qb[K % PD] = read<full(K + PD)>();
      constexpr int kf = full(K), i = kf / TAPS, tap = kf % TAPS;
      constexpr int R = ((tap / COLS) * WG4 + tap % COLS) & 3;
      tap_add<R>(acc[i], q);
      step<K + 1, WG4, PD>(acc, qb);
    }
  }

  template <int K, int PD>
  __device__ __forceinline__ void prime(f4v (&qb)[PD]) const {
    if constexpr (K < PD && K < NS) {
      qb[K] = read<full(K)>();
      prime<K + 1, PD>(qb);
    }
  }
};

template <int ROWS, int COLS, int WG4, int TW, int PD, bool LAST_ROW_AT_END, bool PRIO, int CW>
__device__ __forceinline__ void gather_stream(float (&acc)[TW][4], const uint32_t (&cw)[CW],
                                              const uint32_t (&tapbase)[ROWS * COLS], uint32_t row_bytes,
                                              const char* lbase, bool last_row) {
  const GatherStream<ROWS, COLS, TW, CW, LAST_ROW_AT_END, PRIO> gs{cw, tapbase, row_bytes, lbase, last_row};
  f4v qb[PD];
  gs.template prime<0, PD>(qb);
  gs.template step<0, WG4, PD>(acc, qb);
}

// GEN = false: one virtual subspace per subspace (stride 1, one row group),
// so the input offsets of the table build are fixed per lane.  GEN = true:
// stride phases and/or row groups; the offsets move with the virtual subspace.
//
// VALU = true (comparison variant, stride 1 only): the table is built with
// fused multiply-adds on the vector ALUs instead of MFMA, into the same
// layout.  Lane l computes lut[16 kb + l % 16][16 pb + 4 (l / 16) + r],
// r < 4: its C's codebook values come from the staged codebook in LDS and
// its 4 x C's input values from the lanes that loaded them for the MFMA
// operand layout, through ds_bpermute.
template <int ROWS, int COLS, int WG4, int NC, int TW, bool GEN, bool PRIO, bool VALU = false>
__global__ __launch_bounds__(kThreads, 1) void conv_flat_kernel(const float* __restrict__ x,
                                                                 const float* __restrict__ D,
                                                                 const uint8_t* __restrict__ codes8,
                                                                 const float* __restrict__ bias,
                                                                 float* __restrict__ y, float* __restrict__ partial,
                                                                 FlatParams p) {
  extern __shared__ float4 lut4[];
  float* lut = reinterpret_cast<float*>(lut4);
  constexpr int TAPS = ROWS * COLS;
  constexpr int CS = code_stride(TW, TAPS);  // code bytes per channel
  constexpr int CW = (TW * CS + 3) / 4;      // code dwords per wave and virtual subspace
  constexpr int PD = 6;                // table reads kept in flight (4 to 6 equal, 8 ~1 % slower)
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
  const int v0 = split * p.v_per_split;
  const int v1 = min(p.V, v0 + p.v_per_split);
  const int HW = p.H * p.W;

  if (p.zrow >= 0)  // the zero row; the build never writes it, the first barrier publishes it
    for (int i = threadIdx.x; i < p.PR; i += kThreads) lut[p.zrow * p.PR + i] = 0.f;

  // ---- table-build operands.  A operand: lane supplies row l % 16 (a
  // position) and column l / 16 (an input channel of the subspace); B
  // operand: row l / 16 (channel), column l % 16 (codeword).  Both are read
  // with raw buffer loads: an offset past the buffer's end returns 0, which
  // is exactly the value of a halo position, of a channel beyond C'_s and of
  // a codeword beyond K.
  constexpr uint32_t kOOB = 0x80000000u;
  const int arow = lane & 15, acol = lane >> 4;
  // LDS byte address of this lane's quad for each tap, relative to a table
  // row: tap (u', v') shifts the quad index by (u' Wg + v') / 4.
  uint32_t tapbase[TAPS];
#pragma unroll
  for (int tap = 0; tap < TAPS; ++tap)
    tapbase[tap] = (uint32_t)(lane + (((tap / COLS) * p.Wg + (tap % COLS)) >> 2)) * 16u;
  // Table row stride in bytes, held in a VGPR so that code * stride + tap
  // base is one v_mad_u32_u24 (codes < 256, strides < 2^16).
  uint32_t row_bytes = (uint32_t)p.PR * 4u;
  asm volatile("" : "+v"(row_bytes));
  // Input element (n, m C's + j, yy, xx) sits at byte ((n Cs + j) HW + yy W + xx) * 4
  // + m C's HW * 4; the subspace part goes into the scalar offset.  Only the
  // per-lane (vector) offset is range checked, so every lane whose value must
  // be 0 gets an offset past the end on its own.  Grid position f of this
  // lane: input row s i - pad (+ the virtual subspace's row shift), column
  // s (strip sw + c) - pad (+ its column shift).
  uint32_t xoff[kMaxPB][NC];   // !GEN: final offsets
  int ybase[kMaxPB], xbase[kMaxPB];  // GEN: input row / column before the shift (invalid: a large negative)
  int xb[kMaxPB][NC];          // GEN: offset before the shift
#pragma unroll
  for (int i = 0; i < kMaxPB; ++i) {
    const int pb = wave + kWaves * i;
    const int f = s0 + 16 * pb + arow;
    const int row = f / p.Wg, c = f - row * p.Wg;
    const int g = row / p.Hg, n = g / p.S, strip = g - n * p.S;
    const int yy = p.stride * (row - g * p.Hg) - p.pad, xx = p.stride * (strip * p.sw + c) - p.pad;
    const bool ok = pb < p.npb && f < p.grid_pos && n < p.N;
    if constexpr (GEN) {
      ybase[i] = ok ? yy : -(1 << 28);
      xbase[i] = xx;
    }
#pragma unroll
    for (int cc = 0; cc < NC; ++cc) {
      const int j = 4 * cc + acol;
      if constexpr (GEN) {
        xb[i][cc] = j < p.Csp ? (n * p.Cs + j) * HW + yy * p.W + xx : -(1 << 30);
      } else {
        const bool in = ok && j < p.Csp && yy >= 0 && yy < p.H && xx >= 0 && xx < p.W;
        xoff[i][cc] = in ? (uint32_t)((n * p.Cs + j) * HW + yy * p.W + xx) * 4u : kOOB;
      }
    }
  }
  // Codebook entry (k, j) of subspace m sits at byte (k C's + j) * 4 of that
  // subspace's codebook.  Rows k >= K fall past the buffer's end by
  // themselves; channels j >= C's get an offset past the end here.
  uint32_t dlane[NC];
#pragma unroll
  for (int cc = 0; cc < NC; ++cc) {
    const int j = 4 * cc + acol;
    dlane[cc] = j < p.Csp ? (uint32_t)(arow * p.Csp + j) * 4u : kOOB;
  }
  const uint32_t dstep = (uint32_t)(16 * p.Csp * 4);  // bytes from one 16-row block to the next
  const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(x), 0, (int)((size_t)p.N * p.Cs * HW * 4), 0x00020000);

  float acc[TW][4];
#pragma unroll
  for (int i = 0; i < TW; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;

  const int kblocks = (p.K + 15) >> 4;
  const f4v zero4 = {0.f, 0.f, 0.f, 0.f};

  // Table-build operands, double-buffered: those of virtual subspace v+1 are
  // loaded while the waves gather from the table of v.
  // The codebook of a subspace (the B operands of every wave) is staged in
  // LDS, dstage[(kb NC + c) 64 + l] = D[m][16 kb + l % 16][4 c + l / 16]:
  // wave q < kMaxKB NC loads entry q of each lane's set once for the whole
  // workgroup (a load per wave per 16-codeword block made the build issue
  // bound on vector memory instructions), and writes it to LDS near the end
  // of the previous gather.  Waves past the last entry keep 0 in slots
  // that no build reads.
  static_assert(kMaxKB * NC <= kWaves, "one staging wave per codebook block and channel group");
  float* dstage = lut + p.dstage;
  const bool dloader = wave < kMaxKB * NC;
  const int dkb = wave / NC, dc = wave % NC;
  float av[kMaxPB][NC], dnext = 0.f;
  auto load_operands = [&](int vv, float (&a)[kMaxPB][NC], float& dv) {
    int m = vv, dy = 0, dx = 0;
    if constexpr (GEN) {  // v = ((m s + a) s + b) G + g
      const int g = vv % p.G;
      int r = vv / p.G;
      dx = r % p.stride;
      r /= p.stride;
      dy = r % p.stride + p.stride * g * ROWS;
      m = r / p.stride;
    }
    const __amdgpu_buffer_rsrc_t dres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(D + (size_t)m * p.K * p.Csp), 0, p.K * p.Csp * 4, 0x00020000);
#pragma unroll
    for (int i = 0; i < kMaxPB; ++i) {
      bool in = true;
      if constexpr (GEN) {
        const int yy = ybase[i] + dy, xx = xbase[i] + dx;
        in = yy >= 0 && yy < p.H && xx >= 0 && xx < p.W;
      }
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        uint32_t off;
        if constexpr (GEN)
          off = (in && xb[i][c] >= -(1 << 29)) ? (uint32_t)((xb[i][c] + dy * p.W + dx) * 4) : kOOB;
        else
          off = xoff[i][c];
        a[i][c] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(xres, off, m * p.Csp * HW * 4, 0));
      }
    }
    // Blocks kb >= kblocks hold codewords >= K: their offsets are past the
    // buffer's end, so the loads return 0 without a branch.
    if (dloader) {
      uint32_t off = kOOB;
#pragma unroll
      for (int c = 0; c < NC; ++c)
        if (c == dc) off = dlane[c] + dkb * dstep;
      dv = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(dres, off, 0, 0));
    }
  };
  load_operands(v0, av, dnext);
  dstage[wave * 64 + lane] = dnext;  // published by the loop's first barrier
  // This wave's codes for virtual subspace v: TW x TAPS consecutive bytes, in SGPRs.
  auto load_codes = [&](int vv, uint32_t (&cwv)[CW]) {
    const uint32_t* ow = reinterpret_cast<const uint32_t*>(codes8 + ((size_t)vv * p.ct_pad + t0) * CS);
#pragma unroll
    for (int k = 0; k < CW; ++k) cwv[k] = ow[k];
  };
  uint32_t cw[CW];

  for (int v = v0; v < v1; ++v) {
    __syncthreads();  // every wave is done reading the previous table
    // The build's B operands are read from the staged codebook before any
    // table store (as far as the compiler knows, the stores could overwrite
    // them) and waited for before the codes' scalar loads are issued: LDS
    // reads and scalar loads share one wait counter, so a later wait for the
    // operands would also wait for the codes.
    float bv[kMaxKB][NC];
    if constexpr (!VALU) {
#pragma unroll
      for (int kb = 0; kb < kMaxKB; ++kb)
#pragma unroll
        for (int c = 0; c < NC; ++c) bv[kb][c] = dstage[(kb * NC + c) * 64 + lane];
#pragma unroll
      for (int kb = 0; kb < kMaxKB; ++kb)
#pragma unroll
        for (int c = 0; c < NC; ++c) asm volatile("" ::"v"(bv[kb][c]));
    }
    __builtin_amdgcn_sched_barrier(0);
    // The codes of v arrive during the build.  (A barrier waits for every
    // outstanding scalar load, so issuing them before one would expose their
    // latency.)
    load_codes(v, cw);
    // ---- table build: lut[k][pos] = sum_j D[m][k][j] x[pos][m C's + j]
    // d[r] = lut[k = kb*16 + lane%16][pos = 16 pb + 4 (lane/16) + r]
    float xq[NC][4][4];  // VALU: x[16 pb + 4 (l / 16) + r][4 c + jj] in [c][jj][r]
    auto tile = [&](int i, int kb) -> f4v {
      f4v d = zero4;
      if constexpr (VALU) {
#pragma unroll
        for (int c = 0; c < NC; ++c)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj) {
            const float dk = dstage[(kb * NC + c) * 64 + jj * 16 + arow];  // D[16 kb + l % 16][4 c + jj]
#pragma unroll
            for (int r = 0; r < 4; ++r) d[r] = fmaf(dk, xq[c][jj][r], d[r]);
          }
      } else {
#pragma unroll
        for (int c = 0; c < NC; ++c)
          d = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i][c], bv[kb][c], d, 0, 0, 0);
      }
      return d;
    };
    auto put = [&](int i, int kb, const f4v& d) {
      *reinterpret_cast<f4v*>(lut + (kb * 16 + arow) * p.PR + 16 * (wave + kWaves * i) + 4 * acol) = d;
    };
#pragma unroll
    for (int i = 0; i < kMaxPB; ++i) {
      if (wave + kWaves * i >= p.npb) continue;  // wave-uniform
      if constexpr (VALU) {
        // av[i][c] of lane q holds x[16 pb + q % 16][4 c + q / 16].
#pragma unroll
        for (int c = 0; c < NC; ++c)
#pragma unroll
          for (int jj = 0; jj < 4; ++jj)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              xq[c][jj][r] = __int_as_float(
                  __builtin_amdgcn_ds_bpermute((4 * acol + r + 16 * jj) * 4, __float_as_int(av[i][c])));
      }
      if (kblocks == kMaxKB) {
        // All blocks: straight-line code, each store one MFMA behind so
        // that the next MFMA is issued while the previous result drains.
        f4v prev = tile(i, 0);
#pragma unroll
        for (int kb = 1; kb < kMaxKB; ++kb) {
          const f4v d = tile(i, kb);
          put(i, kb - 1, prev);
          prev = d;
        }
        put(i, kMaxKB - 1, prev);
      } else {
#pragma unroll
        for (int kb = 0; kb < kMaxKB; ++kb)
          if (kb < kblocks) put(i, kb, tile(i, kb));  // rows k >= kblocks*16 are not in the table
      }
    }
    __syncthreads();
    // Operands of v+1, issued after the barrier: issued before it, the burst
    // of loads held every wave at the barrier for about as long as the build.
    if (v + 1 < v1) load_operands(v + 1, av, dnext);
    // ---- gather-accumulate, Eq. (7), over the grid rows and columns of this
    // virtual subspace that lie inside the kernel.
    const char* lbase = reinterpret_cast<const char*>(lut4);
    // Waves whose channels all lie past C_t (a channel block wider than the
    // layer) skip the gather: wave-uniform, they only help build the tables.
    if (t0 < p.Ct) {
      if constexpr (GEN) {
        // Grid row u' is kernel row s (g ROWS + u') + a.
        const int g = v % p.G, a = (v / p.G / p.stride) % p.stride;
        const bool last_row = s_rows_in_kernel(p, a) - g * ROWS >= ROWS;
        gather_stream<ROWS, COLS, WG4, TW, PD, (ROWS > 1), PRIO>(acc, cw, tapbase, row_bytes, lbase, last_row);
      } else {
        gather_stream<ROWS, COLS, WG4, TW, PD, false, PRIO>(acc, cw, tapbase, row_bytes, lbase, true);
      }
    }
    // Stage the codebook of v+1 (its loads have had the whole gather to land).
    // Every wave stores, into a slot of its own, without a branch: a branch
    // here made the compiler spill the accumulators.  After the last subspace
    // the store rewrites what is already there.
    dstage[wave * 64 + lane] = dnext;
  }

  // ---- epilogue
  if (lane == kWave - 1) return;  // its slots belong to the next tile
  if (partial) {
    // partial[split][tile][t][j][lane] holds slot 4 lane + j of the tile:
    // every store instruction writes 256 contiguous bytes.
    float* dst = partial + (((size_t)split * p.tiles + tile) * p.ct_pad + t0) * 256 + lane;
#pragma unroll
    for (int i = 0; i < TW; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) dst[(size_t)i * 256 + 64 * j] = acc[i][j];
    return;
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int s = s0 + 4 * lane + j;
    const int row = s / p.Wg, xl = s - row * p.Wg;
    const int g = row / p.Hg, yo = row - g * p.Hg;
    const int n = g / p.S, xo = (g - n * p.S) * p.sw + xl;
    if (n >= p.N || yo >= p.Ho || xl >= p.sw || xo >= p.Wo) continue;
#pragma unroll
    for (int i = 0; i < TW; ++i) {
      const int t = t0 + i;
      if (t >= p.Ct) break;
      const size_t o = (((size_t)n * p.Ct + t) * p.Ho + yo) * p.Wo + xo;
      float v = acc[i][j] + (bias ? bias[t] : 0.f);
      if (p.relu) v = fmaxf(v, 0.f);
      y[o] = v;
    }
  }
}

// codes8[v][t][tap]: the code of kernel tap (ky, kx) = (s (g ROWS + u') + a,
// s v' + b) of subspace m for virtual subspace v = ((m s + a) s + b) G + g
// and grid tap (u', v') = (tap / COLS, tap % COLS), clamped to K-1; grid taps
// past the kernel get the zero row; channels past C_t and the padding bytes
// of a channel (tap >= ROWS COLS, up to the code stride) get 0.  One thread
// writes one dword (4 consecutive bytes); the bytes it reads are scattered,
// but the whole code array is small and L2-resident.
struct CodeMap {
  int Ct, dk, stride, M, G, rows, cols, K, ct_pad, zrow, V;
  int cstride;  // bytes per channel (>= rows cols; the bytes past the taps are 0 and never read)
};

__global__ __launch_bounds__(256) void flat_codes_kernel(CodeStream codes, CodeMap q,
                                                         uint32_t* __restrict__ codes8) {
  const int taps = q.rows * q.cols;
  const int per_v = q.ct_pad * q.cstride;
  const int nwords = (q.V * per_v + 3) / 4;  // the plan keeps V ct_pad taps below 2^31
  const bool plain = q.G == 1 && q.stride == 1;  // v = m, tap = (ky, kx)
  for (int wi = blockIdx.x * blockDim.x + threadIdx.x; wi < nwords; wi += gridDim.x * blockDim.x) {
    // (v, t, tap) of the word's first byte; the other three follow by
    // stepping tap, then t, then v (no division per byte).
    const int o = wi * 4;
    int v = o / per_v;
    const int r = o - v * per_v;
    int t = r / q.cstride, tap = r - t * q.cstride;
    uint32_t word = 0;
#pragma unroll
    for (int bb = 0; bb < 4; ++bb) {
      uint32_t val = 0;
      if (v < q.V && t < q.Ct && tap < taps) {
        int m = v, ky = tap / q.cols, kx = tap - ky * q.cols;
        if (!plain) {
          const int g = v % q.G;
          int rr = v / q.G;
          const int pb = rr % q.stride;
          rr /= q.stride;
          const int pa = rr % q.stride;
          m = rr / q.stride;
          ky = q.stride * (g * q.rows + ky) + pa;
          kx = q.stride * kx + pb;
        }
        if (ky < q.dk && kx < q.dk) {
          val = code_at(codes, (((size_t)t * q.dk + ky) * q.dk + kx) * q.M + m);
          val = val < (uint32_t)(q.K - 1) ? val : (uint32_t)(q.K - 1);
        } else {
          val = (uint32_t)q.zrow;
        }
      }
      word |= val << (8 * bb);
      if (++tap == q.cstride) {
        tap = 0;
        if (++t == q.ct_pad) {
          t = 0;
          ++v;
        }
      }
    }
    codes8[wi] = word;
  }
}

// y = sum over splits in order + bias, then ReLU.  One thread per stored
// partial value, in the partials' own order [tile][t][j][lane] (so every
// split's values are read with whole cache lines); the thread finds the
// output element of its slot, if the slot is one, and writes it.
__global__ __launch_bounds__(256) void split_reduce_kernel(const float* __restrict__ partial, FlatParams p,
                                                           const float* __restrict__ bias, float* __restrict__ y) {
  const size_t per_split = (size_t)p.tiles * p.ct_pad * 256;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= per_split) return;
  const int lane = (int)(i & 63), j = (int)((i >> 6) & 3);
  if (lane == kWave - 1) return;  // that lane's slots belong to the next tile (not stored)
  const size_t r = i >> 8;
  const int t = (int)(r % p.ct_pad);
  const int tile = (int)(r / p.ct_pad);
  const int slot = tile * kTileSlots + 4 * lane + j;
  const int row = slot / p.Wg, xl = slot - row * p.Wg;
  const int g = row / p.Hg, yo = row - g * p.Hg;
  const int n = g / p.S, xo = (g - n * p.S) * p.sw + xl;
  if (t >= p.Ct || n >= p.N || yo >= p.Ho || xl >= p.sw || xo >= p.Wo) return;
  // Loads of four splits in flight at a time; the sum is still taken in split order.
  float s = 0.f;
  int k = 0;
  for (; k + 4 <= p.splits; k += 4) {
    float v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = partial[(size_t)(k + u) * per_split + i];
#pragma unroll
    for (int u = 0; u < 4; ++u) s += v[u];
  }
  for (; k < p.splits; ++k) s += partial[(size_t)k * per_split + i];
  if (bias) s += bias[t];
  if (p.relu) s = fmaxf(s, 0.f);
  y[(((size_t)n * p.Ct + t) * p.Ho + yo) * p.Wo + xo] = s;
}

// split_reduce_kernel followed by max pooling, in one pass: one workgroup
// per channel t and group of G consecutive images (G H_o W_o <=
// kPoolMapMax).  The group's grid slots are one run of consecutive tiles;
// for each tile the workgroup reads the channel's 1 KB block of partials of
// every split (one float per thread, whole cache lines; two tiles' loads in
// flight), adds the splits in order, adds the bias and rectifies exactly as
// above, and puts each valid output of the group into LDS; the pooled
// outputs are then window maxima over LDS, written as runs of H_p W_p
// contiguous values.  The result equals the split sum followed by the
// max-pool kernel bit for bit; the full map never goes to memory.  Groups
// are mapped XCD-major with the image group fastest, so the tile two
// neighbouring groups share is read from the same L2.
constexpr int kPoolMapMax = 8192;
constexpr int kPoolImages = 8;

struct PoolGroups {
  int G, groups;  // images per workgroup, image groups
};

__device__ __forceinline__ float split_sum(const float* __restrict__ partial, size_t per_split, size_t idx,
                                           int splits) {
  float s = 0.f;
  int k = 0;
  for (; k + 4 <= splits; k += 4) {
    float v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = partial[(size_t)(k + u) * per_split + idx];
#pragma unroll
    for (int u = 0; u < 4; ++u) s += v[u];
  }
  for (; k < splits; ++k) s += partial[(size_t)k * per_split + idx];
  return s;
}

__global__ __launch_bounds__(256) void split_reduce_pool_kernel(const float* __restrict__ partial, FlatParams p,
                                                                PoolSpec q, PoolGroups pg,
                                                                const float* __restrict__ bias,
                                                                float* __restrict__ y) {
  extern __shared__ float map[];  // [G][H_o][W_o] outputs of the group
  const int units = p.Ct * pg.groups;
  const int per_xcd = (units + 7) / 8;
  const int w = (int)(blockIdx.x & 7) * per_xcd + (int)(blockIdx.x >> 3);
  if (w >= units) return;  // whole workgroup, before the barrier
  const int grp = w % pg.groups, t = w / pg.groups;
  const int n0 = grp * pg.G, nimg = min(pg.G, p.N - n0);
  const int plane = p.S * p.Hg * p.Wg;  // grid slots of one image
  const int start = n0 * plane, end = start + nimg * plane;
  const size_t per_split = (size_t)p.tiles * p.ct_pad * 256;
  const int lane = threadIdx.x & 63, j = threadIdx.x >> 6;
  const float b = bias ? bias[t] : 0.f;
  auto place = [&](int tile, float s) {
    const int slot = tile * kTileSlots + 4 * lane + j;
    if (lane == kWave - 1 || slot < start || slot >= end) return;
    const int local = slot - start;
    const int img = local / plane, rem = local - img * plane;
    const int row = rem / p.Wg, xl = rem - row * p.Wg;
    const int strip = row / p.Hg, yo = row - strip * p.Hg;
    const int xo = strip * p.sw + xl;
    if (yo >= p.Ho || xl >= p.sw || xo >= p.Wo) return;
    if (bias) s += b;
    if (p.relu) s = fmaxf(s, 0.f);
    map[(img * p.Ho + yo) * p.Wo + xo] = s;
  };
  const int t_end = (end - 1) / kTileSlots;
  int tile = start / kTileSlots;
  for (; tile + 1 <= t_end; tile += 2) {
    const size_t idx = ((size_t)tile * p.ct_pad + t) * 256 + threadIdx.x;
    const float s0 = split_sum(partial, per_split, idx, p.splits);
    const float s1 = split_sum(partial, per_split, idx + (size_t)p.ct_pad * 256, p.splits);
    place(tile, s0);
    place(tile + 1, s1);
  }
  if (tile <= t_end) place(tile, split_sum(partial, per_split, ((size_t)tile * p.ct_pad + t) * 256 + threadIdx.x,
                                           p.splits));
  __syncthreads();
  const int per_img = q.Hp * q.Wp;
  for (int i = threadIdx.x; i < nimg * per_img; i += blockDim.x) {
    const int img = i / per_img, r = i - img * per_img;
    const int py = r / q.Wp, px = r - py * q.Wp;
    const float* win = map + (img * p.Ho + py * q.s) * p.Wo + px * q.s;
    float best = win[0];
    for (int dy = 0; dy < q.k; ++dy)
      for (int dx = 0; dx < q.k; ++dx) best = fmaxf(best, win[dy * p.Wo + dx]);
    y[((size_t)(n0 + img) * p.Ct + t) * per_img + r] = best;
  }
}



struct FlatPlan {
  FlatParams p;
  int rows, cols;  // tap grid of a virtual subspace
  bool gen;        // offsets move with the virtual subspace
  int TW;
  size_t lds;
  bool prio;  // one workgroup per CU: the plain-grid kernels step their waves' issue priority
  bool valu = false;  // build the tables on the vector ALUs (comparison variant, stride 1 only)
};

// Estimated cost (arbitrary units ~ CU clocks) of a plan, for the choice of
// layout, strips, channel block and subspace split.
double plan_cost(const FlatParams& p, int taps, int TW) {
  const double vals = 40.0;     // table values gathered per clock per CU
  const double mfma = 256.0;    // f32 MFMA flops per clock per CU
  const double vper = (double)p.v_per_split;
  const double gather = (double)kWaves * TW * taps * 256 / vals;
  const double build = (double)p.npb * 16 * 16 * ((p.K + 15) / 16) * 4 * ((p.Csp + 3) / 4) * 2 / mfma;
  const double per_wg = vper * (gather + build + 1500.0);
  const double rounds = (double)((p.work + 255) / 256);
  double cost = rounds * per_wg;
  if (p.splits > 1)  // partial sums written, then read back (~3 kB per clock chip-wide)
    cost += (double)p.splits * 2.0 * p.tiles * p.ct_pad * 256 * 4 / 3.0e3;
  return cost;
}

// A family of layouts: tap grid rows x cols, G row groups, and whether
// neighbouring images share their zero halo.
struct Layout {
  int rows, cols, G;
  bool shared, gen;
};

// Grid geometry for layout L with S strips per image; false when the table
// does not fit.
bool set_geometry(const ConvShape& s, const Layout& L, int S, FlatParams* p, size_t* lds) {
  if (S == 1) {
    p->sw = s.Wo;
    p->Wg = L.shared ? s.W + s.pad : s.Wo + L.cols - 1;
  } else {
    p->sw = ceil_div(s.Wo, S);
    if ((S - 1) * p->sw >= s.Wo) return false;  // an empty last strip
    p->Wg = p->sw + L.cols - 1;
  }
  p->S = S;
  p->Hg = L.shared ? s.H + s.pad : s.Ho + L.rows - 1;
  p->G = L.G;
  const long long slots = (long long)s.N * S * p->Hg * p->Wg;
  const long long gpos = ((long long)s.N * S * p->Hg + (L.shared ? s.pad : 0)) * p->Wg;
  if (gpos + 4096 > (1LL << 31)) return false;
  p->grid_pos = (int)gpos;
  p->tiles = (int)((slots + kTileSlots - 1) / kTileSlots);
  const int dmax = (L.rows - 1) * p->Wg + (L.cols - 1);
  const int PT = 4 * (kWave + (dmax >> 2));
  const int PT16 = (PT + 15) / 16 * 16;
  p->npb = PT16 / 16;
  if (p->npb > kWaves * kMaxPB) return false;
  p->PR = (PT16 / 4) % 2 == 1 ? PT16 : PT16 + 4;
  const int kpad = (s.K + 15) / 16 * 16;
  const bool dummies = s.stride * s.stride * L.G * L.rows * L.cols > s.dk * s.dk;
  p->zrow = dummies ? kpad : -1;
  p->dstage = (kpad + (dummies ? 1 : 0)) * p->PR;
  *lds = ((size_t)p->dstage + (size_t)kThreads) * sizeof(float);
  return *lds <= kLdsBytes;
}

bool make_plan(const ConvShape& s, FlatPlan* out) {
  if (s.Csp > 8 || s.K > 16 * kMaxKB) return false;
  if ((long long)s.N * s.Cs * s.H * s.W * 4 > (1LL << 31) - 1) return false;  // 32-bit buffer offsets
  // Candidate layouts.  Shared halos need stride 1, pad <= d_k - 1, and for
  // several row groups pad + ROWS - 1 < d_k (no output reads a neighbour's
  // rows through a shifted group).
  Layout cand[4];
  int nc = 0;
  if (s.stride == 1 && (s.dk == 1 || s.dk == 3) && s.pad <= s.dk - 1) cand[nc++] = {s.dk, s.dk, 1, true, false};
  if (s.stride == 1 && s.dk == 5 && s.pad + 1 < 5) cand[nc++] = {2, 5, 3, true, true};
  const int r = ceil_div(s.dk, s.stride);  // tap grid of a stride phase
  if ((r == 2 || r == 3) && !(s.stride == 1 && s.dk == 1)) cand[nc++] = {r, r, 1, false, true};
  if (s.stride == 1 && s.dk == 1) cand[nc++] = {1, 1, 1, true, false};
  FlatParams p{};
  p.N = s.N; p.Cs = s.Cs; p.H = s.H; p.W = s.W; p.M = s.M; p.K = s.K; p.Csp = s.Csp; p.Ct = s.Ct;
  p.dk = s.dk; p.stride = s.stride; p.pad = s.pad; p.Ho = s.Ho; p.Wo = s.Wo;
  bool found = false;
  double best = 0;
  for (int ci = 0; ci < nc; ++ci) {
    const Layout& L = cand[ci];
    const int taps = L.rows * L.cols;
    p.V = s.M * s.stride * s.stride * L.G;
    for (int S = 1; S <= 16 && S <= s.Wo; ++S) {
      size_t lds = 0;
      if (!set_geometry(s, L, S, &p, &lds)) continue;
      for (int TW : {6, 8, 12}) {
        // two channel groups, ten taps or moving offsets with 12 channels per
        // wave do not fit the registers.  6 channels per wave only for the
        // stride-phase layouts (they take no 12): a layer of 96 channels
        // (AlexNet conv1) then keeps all 16 waves gathering, where 8 per wave
        // left 4 of them idle (the cost below counts the reads of idle
        // channel slots, so it is not asked to weigh 6 against 8 elsewhere).
        if (TW == 12 && (s.Csp > 4 || L.gen)) continue;
        if (TW == 6 && (s.Csp > 4 || !L.gen || s.stride == 1)) continue;
        const int tc = kWaves * TW;
        const int tblocks = ceil_div(s.Ct, tc);
        for (int splits = 1; splits <= 16 && splits <= p.V; ++splits) {
          FlatParams q = p;
          q.tc = tc;
          q.tblocks = tblocks;
          q.v_per_split = ceil_div(p.V, splits);
          q.splits = ceil_div(p.V, q.v_per_split);
          if (q.splits != splits) continue;
          const long long work = (long long)p.tiles * tblocks * q.splits;
          if (work > (1LL << 30)) continue;
          q.work = (int)work;
          q.per_xcd = ceil_div(q.work, 8);
          q.ct_pad = tblocks * tc;
          if ((long long)p.V * q.ct_pad * code_stride(TW, taps) + 4 > (1LL << 31)) continue;
          const double c = plan_cost(q, taps, TW);
          if (!found || c < best) {
            found = true;
            best = c;
            *out = {q, L.rows, L.cols, L.gen, TW, lds};
          }
        }
      }
    }
  }
  return found;
}

template <int ROWS, int COLS, int WG4, int NC, int TW, bool GEN, bool PRIO>
hipError_t launch_kernel(const FlatPlan& pl, const float* x, const float* D, const uint8_t* codes8,
                         const float* bias, float* y, float* partial, hipStream_t stream, LaunchTimer* timer) {
  auto k = conv_flat_kernel<ROWS, COLS, WG4, NC, TW, GEN, PRIO, false>;
  if constexpr (!GEN) {
    if (pl.valu) k = conv_flat_kernel<ROWS, COLS, WG4, NC, TW, GEN, PRIO, true>;
  }
  hipError_t e = allow_max_lds((const void*)k);
  if (e != hipSuccess) return e;
  return timed_launch(timer, k, dim3(8 * pl.p.per_xcd), dim3(kThreads), (uint32_t)pl.lds, stream, x, D, codes8, bias, y,
                      partial, pl.p);
}

template <int ROWS, int COLS, int WG4, int NC, int TW, bool GEN>
hipError_t launch_main(const FlatPlan& pl, const float* x, const float* D, const uint8_t* codes8, const float* bias,
                       float* y, float* partial, hipStream_t stream, LaunchTimer* timer) {
  if (pl.prio)
    return launch_kernel<ROWS, COLS, WG4, NC, TW, GEN, true>(pl, x, D, codes8, bias, y, partial, stream, timer);
  return launch_kernel<ROWS, COLS, WG4, NC, TW, GEN, false>(pl, x, D, codes8, bias, y, partial, stream, timer);
}

struct LaunchArgs {
  const float* x;
  const float* D;
  const uint8_t* codes8;
  const float* bias;
  float* y;
  float* partial;
  hipStream_t stream;
  LaunchTimer* timer;
};

template <int ROWS, int COLS, int WG4, bool GEN>
hipError_t launch_nc(const FlatPlan& pl, const LaunchArgs& a) {
  if constexpr (GEN) {
    if (pl.TW == 6)  // the planner gives 6 channels per wave only with C's <= 4
      return launch_main<ROWS, COLS, WG4, 1, 6, GEN>(pl, a.x, a.D, a.codes8, a.bias, a.y, a.partial, a.stream, a.timer);
  }
  if (pl.p.Csp <= 4) {
    if constexpr (!GEN) {
      if (pl.TW == 12) return launch_main<ROWS, COLS, WG4, 1, 12, GEN>(pl, a.x, a.D, a.codes8, a.bias, a.y, a.partial,
                                                                       a.stream, a.timer);
    }
    return launch_main<ROWS, COLS, WG4, 1, 8, GEN>(pl, a.x, a.D, a.codes8, a.bias, a.y, a.partial, a.stream, a.timer);
  }
  return launch_main<ROWS, COLS, WG4, 2, 8, GEN>(pl, a.x, a.D, a.codes8, a.bias, a.y, a.partial, a.stream, a.timer);
}

template <int ROWS, int COLS, bool GEN>
hipError_t launch_wg(const FlatPlan& pl, const LaunchArgs& a) {
  if constexpr (ROWS == 1 && COLS == 1) {
    return launch_nc<1, 1, 0, GEN>(pl, a);  // one tap: no shift
  } else {
    switch (pl.p.Wg & 3) {
      case 0: return launch_nc<ROWS, COLS, 0, GEN>(pl, a);
      case 1: return launch_nc<ROWS, COLS, 1, GEN>(pl, a);
      case 2: return launch_nc<ROWS, COLS, 2, GEN>(pl, a);
      default: return launch_nc<ROWS, COLS, 3, GEN>(pl, a);
    }
  }
}

hipError_t launch_plan(const FlatPlan& pl, const LaunchArgs& a) {
  const int shape = pl.rows * 10 + pl.cols;
  if (!pl.gen) {
    if (shape == 11) return launch_wg<1, 1, false>(pl, a);
    if (shape == 33) return launch_wg<3, 3, false>(pl, a);
  } else {
    if (shape == 22) return launch_wg<2, 2, true>(pl, a);
    if (shape == 33) return launch_wg<3, 3, true>(pl, a);
    if (shape == 25) return launch_wg<2, 5, true>(pl, a);
  }
  return hipErrorInvalidConfiguration;
}

}  // namespace

bool conv_flat_supported(const ConvShape& s) {
  FlatPlan pl;
  return make_plan(s, &pl);
}

namespace {

// Workspace of a plan: the re-laid-out codes, then (split plans) the partials.
struct FlatWs {
  size_t n_codes, code_bytes, partial_elems, total;
};

FlatWs flat_ws(const FlatPlan& pl) {
  const FlatParams& p = pl.p;
  FlatWs w;
  w.n_codes = (size_t)p.V * p.ct_pad * code_stride(pl.TW, pl.rows * pl.cols);
  w.code_bytes = (w.n_codes + 4 + 255) & ~(size_t)255;  // + the tail of the last dword load
  w.partial_elems = (size_t)p.splits * p.tiles * p.ct_pad * 256;
  w.total = w.code_bytes + (p.splits > 1 ? w.partial_elems * sizeof(float) : 0);
  return w;
}

}  // namespace

size_t conv_flat_workspace(const ConvShape& s) {
  FlatPlan pl;
  return make_plan(s, &pl) ? flat_ws(pl).total : 0;
}

bool conv_flat_pools(const ConvShape& s) {
  FlatPlan pl;
  return make_plan(s, &pl) && pl.p.splits > 1 && s.Ho * s.Wo <= kPoolMapMax &&
         (long long)s.N * s.Ct <= 0x7ffffff0LL;
}

namespace {

// The plan of a call: make_plan's choice and the per-call switches.
bool flat_plan(const ConvShape& s, int relu, FlatPlan* pl) {
  if (!make_plan(s, pl)) return false;
  pl->p.relu = relu;
  // The priority steps only where no second workgroup can share the CU: by
  // LDS, or for the layouts with moving offsets by registers (their kernels
  // use 103-111 VGPRs per lane, so one 16-wave workgroup fills a CU's waves).
  pl->prio = pl->lds > kLdsBytes / 2 || pl->gen;
  // QCNN_TABLE_BUILD=valu: the vector-ALU table build, for comparison with
  // the MFMA build (read per call; the strided layouts keep MFMA).
  const char* tb = getenv("QCNN_TABLE_BUILD");
  pl->valu = !pl->gen && tb && strcmp(tb, "valu") == 0;
  static const bool trace = getenv("QCNN_TRACE_PLAN") && *getenv("QCNN_TRACE_PLAN") == '1';
  if (trace)
    fprintf(stderr, "qcnn conv_flat: taps %dx%d%s G=%d V=%d S=%d sw=%d Wg=%d Hg=%d tiles=%d TW=%d tc=%d tblocks=%d "
            "splits=%d work=%d PR=%d npb=%d zrow=%d lds=%zu\n", pl->rows, pl->cols, pl->gen ? " gen" : "", pl->p.G,
            pl->p.V, pl->p.S, pl->p.sw, pl->p.Wg, pl->p.Hg, pl->p.tiles, pl->TW, pl->p.tc, pl->p.tblocks, pl->p.splits,
            pl->p.work, pl->p.PR, pl->p.npb, pl->p.zrow, pl->lds);
  return true;
}

hipError_t launch_codes(const FlatPlan& pl, CodeStream codes, uint8_t* codes8, hipStream_t stream) {
  const FlatParams& p = pl.p;
  const size_t nwords = (flat_ws(pl).n_codes + 3) / 4;
  const CodeMap cm{p.Ct, p.dk, p.stride, p.M, p.G, pl.rows, pl.cols, p.K, p.ct_pad, p.zrow, p.V,
                   code_stride(pl.TW, pl.rows * pl.cols)};
  hipLaunchKernelGGL(flat_codes_kernel, dim3((unsigned)std::min<size_t>(2048, ceil_div_z(nwords, 256))), dim3(256), 0,
                     stream, codes, cm, reinterpret_cast<uint32_t*>(codes8));
  return hipGetLastError();
}

// The kernels of a call after the code re-layout: the main kernel, then (split
// plans) the split sum, which with `pool` takes the pooling maxima.
hipError_t run_flat(const FlatPlan& pl, const ConvShape& s, const float* x, const float* D, const uint8_t* codes8,
                    const float* bias, float* y, float* partial, hipStream_t stream, bool timed,
                    const PoolSpec* pool) {
  const FlatParams& p = pl.p;
  hipError_t e;
  {
    LaunchTimer timer(timed);
    e = launch_plan(pl, LaunchArgs{x, D, codes8, bias, y, partial, stream, &timer});
  }
  if (e == hipSuccess && partial && pool) {
    PoolGroups pg;
    pg.G = std::max(1, std::min(std::min(kPoolImages, p.N), kPoolMapMax / (s.Ho * s.Wo)));
    pg.groups = ceil_div(p.N, pg.G);
    const unsigned units = (unsigned)((size_t)p.Ct * pg.groups);
    hipLaunchKernelGGL(split_reduce_pool_kernel, dim3((units + 7) / 8 * 8), dim3(256),
                       (uint32_t)((size_t)pg.G * s.Ho * s.Wo * sizeof(float)), stream, partial, p, *pool, pg, bias,
                       y);
    e = hipGetLastError();
  } else if (e == hipSuccess && partial) {
    hipLaunchKernelGGL(split_reduce_kernel, dim3((unsigned)ceil_div_z(flat_ws(pl).partial_elems / p.splits, 256)),
                       dim3(256), 0, stream, partial, p, bias, y);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace

hipError_t launch_conv_flat(const ConvShape& s, const float* x, const float* D, CodeStream codes,
                            const float* bias, int relu, float* y, hipStream_t stream, const Workspace* ws,
                            const PoolSpec* pool) {
  FlatPlan pl;
  if (!flat_plan(s, relu, &pl)) return hipErrorInvalidConfiguration;
  if (pool && (pl.p.splits < 2 || s.Ho * s.Wo > kPoolMapMax)) return hipErrorInvalidConfiguration;
  const FlatWs w = flat_ws(pl);
  Scratch scratch;
  hipError_t e = scratch.take(stream, w.total, ws);
  if (e != hipSuccess) return e;
  char* base = scratch.get();
  uint8_t* codes8 = reinterpret_cast<uint8_t*>(base);
  float* partial = pl.p.splits > 1 ? reinterpret_cast<float*>(base + w.code_bytes) : nullptr;
  e = launch_codes(pl, codes, codes8, stream);
  if (e != hipSuccess) return e;
  return run_flat(pl, s, x, D, codes8, bias, y, partial, stream, ws == nullptr || ws->timed, pool);
}

size_t conv_flat_code_bytes(const ConvShape& s) {
  FlatPlan pl;
  return make_plan(s, &pl) ? flat_ws(pl).code_bytes : 0;
}

hipError_t launch_conv_flat_codes(const ConvShape& s, CodeStream codes, uint8_t* codes8, hipStream_t stream) {
  FlatPlan pl;
  if (!make_plan(s, &pl)) return hipErrorInvalidConfiguration;
  return launch_codes(pl, codes, codes8, stream);
}

hipError_t launch_conv_flat_relaid(const ConvShape& s, const float* x, const float* D, const uint8_t* codes8,
                                   const float* bias, int relu, float* y, hipStream_t stream, const PoolSpec* pool) {
  FlatPlan pl;
  if (!flat_plan(s, relu, &pl)) return hipErrorInvalidConfiguration;
  const FlatWs w = flat_ws(pl);
  // With a pooling that the split sum cannot take, the full map goes to the
  // workspace after the partial sums and a max-pool kernel reads it.
  const bool split_pools = pool && conv_flat_pools(s);
  const size_t part = pl.p.splits > 1 ? (w.partial_elems * sizeof(float) + 255) & ~(size_t)255 : 0;
  const size_t full = pool && !split_pools ? (size_t)s.N * s.Ct * s.Ho * s.Wo * sizeof(float) : 0;
  Scratch scratch;
  hipError_t e = scratch.take(stream, part + full, nullptr);
  if (e != hipSuccess) return e;
  float* partial = part ? reinterpret_cast<float*>(scratch.get()) : nullptr;
  float* ymap = full ? reinterpret_cast<float*>(scratch.get() + part) : y;
  e = run_flat(pl, s, x, D, codes8, bias, ymap, partial, stream, true, split_pools ? pool : nullptr);
  if (e != hipSuccess || !full) return e;
  return launch_maxpool(ymap, s.N, s.Ct, s.Ho, s.Wo, pool->k, pool->s, pool->Hp, pool->Wp, y, stream);
}

}  // namespace qcnn
