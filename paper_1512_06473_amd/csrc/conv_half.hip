// PQ convolution with two tables in LDS: the table of the next subspace is
// built while the current one is gathered.
//
// Paper: Sec. 3.2, Eq. (7): each response sums, over the receptive-field
// pairs (p_k, p_s) and the subspaces m, the table entry <D^(m)_k, S^(m)_{p_s}>
// selected by the code k = k_m(c_t, p_k); the table is pre-computed over the
// input positions (paragraph after Eq. (7); Table 1 term d_s^2 C_s K).
//
// Layout.  The output maps are stacked into one flat grid 14 slots wide, as
// in conv_flat.hip: grid slot s = ((n S + strip) Hg + yo) 14 + xl holds
// output (n, yo, strip sw + xl).  For maps with W + pad <= 14 the images
// share their zero halo (S = 1, Hg = H + pad); wider maps are cut into S
// column strips of sw = 15 - d_k outputs that keep their own margins.  A
// kernel tap (ty, tx) of a stride-1 layer is then the uniform shift
// ty 14 + tx of the flat slot, and the 3x3 taps reach 30 slots ahead.
//
// Work split.  A tile is 124 consecutive slots.  Each half of a wave (lanes
// 0-31 and 32-63) serves one output channel: lane l of the half owns slots
// 4l .. 4l+3 of the tile (lane 31 only supplies neighbour values), so one
// 128-bit table read per lane serves two channels at once, and one table of
// 156 positions x K codewords serves 2 x 16 x TWP channels.  The two halves
// read two different table rows: the row of lane l is a byte offset taken
// from a re-laid code stream (code x row stride, computed once per call),
// which the lane loads four at a time with vector loads (their wait counter
// is not the one the LDS reads use) a few groups ahead of use; a read's
// address is then one add, and the tap's shift is the read's immediate
// offset.  The 0..3 elements a tap shift moves past the lane's quad come from
// lane l+1 through a DPP wave shift.
//
// Pipelining.  Two table buffers: while the waves gather subspace v from one,
// the table of subspace v+1 is built into the other
// (v_mfma_f32_16x16x4_f32: 16 positions x 16 codewords x 4 input channels per
// instruction).  Either one wave of the workgroup builds every table while
// the other 15 gather (its operand loads then never delay the gathering
// waves' row-offset loads, which share their wait counter), synchronised by
// two LDS counters so that the gathering waves may drift up to one subspace
// apart; or every wave builds its share between its table reads, with one
// workgroup barrier per subspace.
//
// The subspaces may be split over workgroups (to fill the chip): each then
// stores its partial sums, 128 contiguous bytes per store, and a second
// kernel adds them in a fixed order.  Blocks are mapped XCD-major, so the
// workgroups of one tile share an XCD and its L2.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <utility>

#include "qcnn_internal.h"

namespace qcnn {

struct HalfParams {
  int N, Cs, H, W, M, K, Csp, Ct, dk, pad, Ho, Wo;
  int S, sw, Wg, Hg;     // strips per image, outputs per strip, grid width and rows per image
  int grid_pos;          // grid slots that may hold input (beyond: zero)
  int tiles;             // ceil(N S Hg Wg / 124)
  int PR, PT;            // table row stride in floats; table positions built
  int tbl_bytes;         // bytes of one table buffer
  int tc, tblocks, nwslots, ngp;  // channels per workgroup, channel blocks, waves x blocks, row-offset groups
  int splits, v_per_split, work, per_xcd, ct_pad;
  int relu;
};

namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;
constexpr int kTileSlots = 124;
constexpr int kGridW = 14;   // grid width of the tap kernels (1x1 layers use W)
constexpr int kMaxPB = 10;   // 16-position blocks of a table (156 positions + the last block's rest)
constexpr int kRing = 4;     // row-offset groups held per lane (loaded kRing - 1 groups ahead)
// Table reads kept in flight per wave: 6 when every wave builds; 4 with the
// builder wave (a shorter LDS queue lets the builder's table stores through).
template <bool BLD>
constexpr int kPDof = BLD ? 4 : 6;

typedef float f4v __attribute__((ext_vector_type(4)));
typedef uint32_t u4v __attribute__((ext_vector_type(4)));

template <int... Is, typename F>
__device__ __forceinline__ void static_for_impl(std::integer_sequence<int, Is...>, F&& f) {
  (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(std::make_integer_sequence<int, N>{}, f);
}

// acc[j] += element j + R of the lane's quad q, the elements past the quad
// from lane l+1's quad (DPP wave shift; lane 63 reads 0).
// (The elements are copied out of the vector first: a bit cast of a vector
// element reference reads element 0 whatever the index.)
template <int R>
__device__ __forceinline__ void tap_add(float (&a)[4], const f4v& q) {
  const float e[4] = {q[0], q[1], q[2], q[3]};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (j + R < 4) {
      a[j] += e[j + R];
    } else {
      const int nb = __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, e[j + R - 4]), 0x130 /* wave_shl:1 */,
                                                 0xf, 0xf, false);
      a[j] += __builtin_bit_cast(float, nb);
    }
  }
}

// Wait for this wave's LDS accesses, then the workgroup barrier.  (Vector
// loads stay in flight across it: the row offsets of the next subspace.)
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Spin until the LDS word at byte address `addr` is at least `target` (the
// producer is a wave of the same workgroup, resident with this one, so the
// wait ends); a bound on the polls (2^22) keeps every wave finite whatever
// happens.  The loop is one asm block: as compiler control flow inside the
// unrolled gather loop it made the register allocator spill.  It waits for
// all of the wave's LDS accesses, which is free where it is used (none are
// in flight there).
__device__ __forceinline__ void wait_at_least(uint32_t addr, int target) {
  int val;
  int sv;
  uint32_t cnt;
  asm volatile(
      "s_mov_b32 %[cnt], 0x400000\n"
      "1:\n\t"
      "ds_read_b32 %[val], %[addr]\n\t"
      "s_waitcnt lgkmcnt(0)\n\t"
      "v_readfirstlane_b32 %[sv], %[val]\n\t"
      "s_cmp_ge_i32 %[sv], %[tgt]\n\t"
      "s_cbranch_scc1 2f\n\t"
      "s_sleep 1\n\t"
      "s_sub_u32 %[cnt], %[cnt], 1\n\t"
      "s_cbranch_scc0 1b\n"
      "2:"
      : [val] "=&v"(val), [sv] "=&s"(sv), [cnt] "=&s"(cnt)
      : [addr] "v"(addr), [tgt] "s"(target)
      : "memory", "scc");
}

// After every LDS access of this wave has completed, add 1 to the LDS word
// at byte address `addr` from lane 0 only.  One asm block with the exec mask
// saved and restored: an `if (lane == 0)` here is a branch at the end of the
// gather stream, and the compiler sinks the stream's adds past it.
__device__ __forceinline__ void lds_count_done(uint32_t addr) {
  uint64_t saved;
  asm volatile(
      "s_waitcnt lgkmcnt(0)\n\t"
      "s_mov_b64 %[sv], exec\n\t"
      "s_mov_b64 exec, 1\n\t"
      "ds_add_u32 %[a], %[one]\n\t"
      "s_mov_b64 exec, %[sv]"
      : [sv] "=&s"(saved)
      : [a] "v"(addr), [one] "v"(1)
      : "memory");
}

// ROWS x COLS taps (3x3 or 1x1); NC: groups of 4 input channels per subspace
// (C'_s <= 4: 1, <= 8: 2); TWP: channels per half-wave; KBL: 16-codeword
// blocks of the table (1, 2, 4 or 8); BLD: the last wave builds every table
// after the first while the other waves gather (otherwise every wave
// builds its share of the next table between its table reads).
template <int ROWS, int COLS, int NC, int TWP, int KBL, bool BLD>
__global__ __launch_bounds__(kThreads, 1) void conv_half_kernel(const float* __restrict__ x,
                                                                const float* __restrict__ D,
                                                                const uint32_t* __restrict__ rowoff,
                                                                const float* __restrict__ bias,
                                                                float* __restrict__ y, float* __restrict__ partial,
                                                                HalfParams p) {
  extern __shared__ float4 lut4[];
  const char* lread = reinterpret_cast<const char*>(lut4);
  char* lwrite = reinterpret_cast<char*>(lut4);
  constexpr int TAPS = ROWS * COLS;
  constexpr int NQ = TWP * TAPS;                          // table reads per wave and subspace
  constexpr int NG = (NQ + 3) / 4;                        // row-offset groups (4 reads each)
  constexpr int NGP = (NG + kRing - 1) / kRing * kRing;   // groups per subspace in the stream
  constexpr int PBSTEP = kWaves / KBL;                    // position blocks between a wave's build tasks
  constexpr int TPW = (kMaxPB + PBSTEP - 1) / PBSTEP;     // build tasks per wave (first table; all of them without BLD)
  static_assert(kWaves % KBL == 0, "codeword blocks divide the waves");
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int hh = lane >> 5, ll = lane & 31;
  const int arow = lane & 15, acol = lane >> 4;

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
  const int wslot = tb * kWaves + wave;
  const int tw0 = tb * p.tc + (2 * wave + hh) * TWP;  // channel of acc[0] for this lane's half
  const int v0 = split * p.v_per_split;
  const int v1 = min(p.M, v0 + p.v_per_split);
  const int HW = p.H * p.W;

  // ---- table-build operands.  A operand of position block pb: lane supplies
  // position 16 pb + l % 16 and input channel 4 c + l / 16; B operand of
  // codeword block kb: input channel 4 c + l / 16 and codeword 16 kb + l % 16.
  // Raw buffer loads return 0 past a buffer's end, which is exactly the value
  // of a halo position, a channel beyond C'_s and a codeword beyond K.
  constexpr uint32_t kOOB = 0x80000000u;
  const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(x), 0, (int)((size_t)p.N * p.Cs * HW * 4), 0x00020000);
  auto x_offset = [&](int pb, int cc) -> uint32_t {
    const int f = s0 + 16 * pb + arow;
    const int row = f / p.Wg, c = f - row * p.Wg;
    const int g = row / p.Hg, n = g / p.S, strip = g - n * p.S;
    const int yy = row - g * p.Hg - p.pad, xx = strip * p.sw + c - p.pad;
    const int jc = 4 * cc + acol;
    const bool ok = 16 * pb < p.PT && f < p.grid_pos && n < p.N && yy >= 0 && yy < p.H && xx >= 0 && xx < p.W &&
                    jc < p.Csp;
    return ok ? (uint32_t)((n * p.Cs + jc) * HW + yy * p.W + xx) * 4u : kOOB;
  };
  auto d_offset = [&](int kbk, int cc) -> uint32_t {
    const int jc = 4 * cc + acol;
    return jc < p.Csp ? (uint32_t)((16 * kbk + arow) * p.Csp + jc) * 4u : kOOB;
  };
  auto d_rsrc = [&](int vv) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(D + (size_t)vv * p.K * p.Csp), 0, p.K * p.Csp * 4,
                                             0x00020000);
  };
  // Table store of (position block pb, codeword block kb): row 16 kb + l % 16,
  // positions 16 pb + 4 (l / 16) .. + 3; lanes whose positions lie past PT
  // (they would spill into the next row) write a spare slot after the two
  // tables instead, without a branch (a branch in the gather stream lets the
  // compiler sink the gather's adds past it and hold every read in registers).
  const uint32_t spare = 2u * (uint32_t)p.tbl_bytes;
  // With the builder wave, LDS words after the spare slot: [0] the last table
  // built (its subspace), [1 + b] how many (wave, table) gathers of buffer b
  // have finished.
  typedef __attribute__((address_space(3))) volatile int lds_int;
  lds_int* sync_words = (lds_int*)(lwrite + spare + 16);
  const uint32_t sync_addr = (uint32_t)(uintptr_t)sync_words;
  auto store_at = [&](int pb, int kbk, uint32_t bufoff, const f4v& d) {
    const int pos = 16 * pb + 4 * acol;
    const uint32_t a = pos < p.PT ? bufoff + (uint32_t)(((16 * kbk + arow) * p.PR + pos) * 4) : spare;
    *reinterpret_cast<f4v*>(lwrite + a) = d;
  };

  // Every wave's share of a table: codeword block kb of the position blocks
  // pb_j = wave / KBL + j PBSTEP.
  const int kb = wave % KBL, pbw = wave / KBL;
  uint32_t xoff[TPW][NC], dlane[NC];
#pragma unroll
  for (int j = 0; j < TPW; ++j)
#pragma unroll
    for (int cc = 0; cc < NC; ++cc) xoff[j][cc] = x_offset(pbw + j * PBSTEP, cc);
#pragma unroll
  for (int cc = 0; cc < NC; ++cc) dlane[cc] = d_offset(kb, cc);
  float av[TPW][NC], bv[NC];
  auto load_into = [&](int vv, float (&a)[TPW][NC], float (&bb)[NC]) {
    const __amdgpu_buffer_rsrc_t dres = d_rsrc(vv);
#pragma unroll
    for (int cc = 0; cc < NC; ++cc) bb[cc] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(dres, dlane[cc], 0, 0));
#pragma unroll
    for (int j = 0; j < TPW; ++j)
#pragma unroll
      for (int cc = 0; cc < NC; ++cc)
        a[j][cc] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(xres, xoff[j][cc], vv * p.Csp * HW * 4, 0));
  };
  auto load_build = [&](int vv) { load_into(vv, av, bv); };
  auto task_of = [&](int j, const float (&a)[TPW][NC], const float (&bb)[NC]) -> f4v {
    f4v d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int cc = 0; cc < NC; ++cc) d = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j][cc], bb[cc], d, 0, 0, 0);
    return d;
  };
  auto build_task = [&](int j) -> f4v { return task_of(j, av, bv); };

  // Prologue: the table of v0 into buffer 0, every wave its share (with the
  // builder wave also the table of v0 + 1 into buffer 1, so that the
  // builder's first own table has its operand loads' latency hidden).
  load_build(v0);
  if constexpr (BLD) {
    float av1[TPW][NC], bv1[NC];
    load_into(min(v0 + 1, v1 - 1), av1, bv1);
#pragma unroll
    for (int j = 0; j < TPW; ++j) store_at(pbw + j * PBSTEP, kb, 0u, build_task(j));
    if (v0 + 1 < v1) {
#pragma unroll
      for (int j = 0; j < TPW; ++j) store_at(pbw + j * PBSTEP, kb, (uint32_t)p.tbl_bytes, task_of(j, av1, bv1));
    }
    if (threadIdx.x == 0) {
      sync_words[0] = min(v0 + 1, v1 - 1);
      sync_words[1] = 0;
      sync_words[2] = 0;
    }
  } else {
#pragma unroll
    for (int j = 0; j < TPW; ++j) store_at(pbw + j * PBSTEP, kb, 0u, build_task(j));
  }

  if constexpr (BLD) {
    if (wave == kWaves - 1) {
      // ---- the builder wave: while the others gather subspace v, it builds
      // the table of v+1 into the other buffer (all position and codeword
      // blocks), its operands loaded one subspace ahead, so that their memory
      // latency hides behind a whole gather.  It holds no accumulators.
      uint32_t xo[kMaxPB][NC], dl[KBL][NC];
#pragma unroll
      for (int pb = 0; pb < kMaxPB; ++pb)
#pragma unroll
        for (int cc = 0; cc < NC; ++cc) xo[pb][cc] = x_offset(pb, cc);
#pragma unroll
      for (int k2 = 0; k2 < KBL; ++k2)
#pragma unroll
        for (int cc = 0; cc < NC; ++cc) dl[k2][cc] = d_offset(k2, cc);
      float A[kMaxPB][NC], B[KBL][NC];
      auto load_all = [&](int vv, float (&a)[kMaxPB][NC], float (&bb)[KBL][NC]) {
        const __amdgpu_buffer_rsrc_t dres = d_rsrc(vv);
#pragma unroll
        for (int k2 = 0; k2 < KBL; ++k2)
#pragma unroll
          for (int cc = 0; cc < NC; ++cc)
            bb[k2][cc] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(dres, dl[k2][cc], 0, 0));
#pragma unroll
        for (int pb = 0; pb < kMaxPB; ++pb)
#pragma unroll
          for (int cc = 0; cc < NC; ++cc)
            a[pb][cc] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(xres, xo[pb][cc], vv * p.Csp * HW * 4, 0));
      };
      // Store address of (pb, kb): row 16 kb + l % 16, position 16 pb + 4 (l / 16).
      const uint32_t sb0 = (uint32_t)((arow * p.PR + 4 * acol) * 4);
      const uint32_t kstep = (uint32_t)(16 * p.PR * 4);
      const int plim = p.PT - 4 * acol;
      // Table t goes into buffer (t - v0) & 1, the buffer of table t - 2: it
      // waits until every gathering wave is done with the tables that buffer
      // held before (the count of that buffer only; no wave can have gathered
      // t yet), then publishes t.  The gathering waves may therefore run up to
      // one subspace apart (no barrier per subspace).  Its operands are
      // loaded two tables ahead, in two register sets used in turn.
      auto build = [&](int t, const float (&a)[kMaxPB][NC], const float (&bb)[KBL][NC]) {
        const int nb = (t - v0) & 1;
        wait_at_least(sync_addr + 4u * (1u + nb), (kWaves - 1) * ((t - v0) >> 1));
        // Top issue priority while building: the gathering waves wait for
        // this table.  Masked stores go to the spare slot (no branch); the
        // codeword blocks of a position block go through the MFMA pipe back
        // to back before their stores.
        __builtin_amdgcn_s_setprio(3);
        uint32_t tb1 = (uint32_t)(nb * p.tbl_bytes) + sb0;
        uint32_t sp = spare;
        // (opaque here, so that the compiler forms the 80 store addresses
        // at their stores instead of holding them all across the loop)
        asm volatile("" : "+v"(tb1), "+v"(sp));
#pragma unroll
        for (int pb = 0; pb < kMaxPB; ++pb) {
          const bool in = 16 * pb < plim;
          f4v d[KBL];
#pragma unroll
          for (int k2 = 0; k2 < KBL; ++k2) {
            d[k2] = f4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int cc = 0; cc < NC; ++cc)
              d[k2] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[pb][cc], bb[k2][cc], d[k2], 0, 0, 0);
          }
#pragma unroll
          for (int k2 = 0; k2 < KBL; ++k2)
            *reinterpret_cast<f4v*>(lwrite + (in ? tb1 + k2 * kstep + pb * 64 : sp)) = d[k2];
        }
        __builtin_amdgcn_s_setprio(0);
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // the table is in LDS before it is published
        if (lane == 0) sync_words[0] = t;
      };
      float A2[kMaxPB][NC], B2[KBL][NC];
      load_all(min(v0 + 2, v1 - 1), A, B);
      load_all(min(v0 + 3, v1 - 1), A2, B2);
      lds_barrier();
      for (int t = v0 + 2; t < v1; t += 2) {
        build(t, A, B);
        load_all(min(t + 2, v1 - 1), A, B);
        if (t + 1 >= v1) break;
        build(t + 1, A2, B2);
        load_all(min(t + 3, v1 - 1), A2, B2);
      }
      return;
    }
  }

  // ---- row offsets: record (v, wslot) holds NGP groups x 2 halves x 4
  // dwords; this lane reads its half's 4 dwords of a group.
  const __amdgpu_buffer_rsrc_t rres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint32_t*>(rowoff), 0, (int)((size_t)p.M * p.nwslots * NGP * 32), 0x00020000);
  const uint32_t rlane = (uint32_t)hh * 16u;
  auto load_group = [&](int vv, int g) -> u4v {
    return __builtin_amdgcn_raw_buffer_load_b128(rres, rlane + (uint32_t)g * 32u, (vv * p.nwslots + wslot) * NGP * 32,
                                                 0);
  };
  u4v ring[kRing];
#pragma unroll
  for (int g = 0; g < kRing; ++g) ring[g] = load_group(v0, g);

  float acc[TWP][4];
#pragma unroll
  for (int i = 0; i < TWP; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
  lds_barrier();

  int buf = 0;
  for (int v = v0; v < v1; ++v) {
    const int vn = min(v + 1, v1 - 1);  // the last pass rebuilds v1 - 1 into the free buffer (no branch)
    if constexpr (!BLD) load_build(vn);
    if constexpr (BLD) wait_at_least(sync_addr, v);  // table v is complete
    const char* lrb = lread + (ll * 16 + buf * p.tbl_bytes);  // this lane's quad in the table of v
    const uint32_t nbuf = (uint32_t)(buf ^ 1) * (uint32_t)p.tbl_bytes;
    // read r of the stream: channel r / TAPS, tap r % TAPS
    auto read = [&](auto R) -> f4v {
      constexpr int r = decltype(R)::value;
      constexpr int tap = r % TAPS;
      constexpr int sh = (tap / COLS) * kGridW + tap % COLS;
      const uint32_t ro = ring[(r / 4) % kRing][r % 4];
      return *reinterpret_cast<const f4v*>(lrb + ro + (sh >> 2) * 16);
    };
    // After read r is issued: a group whose last read that was gets its ring
    // slot refilled with the group kRing ahead (of this subspace, or of the next).
    auto refill = [&](auto R) {
      constexpr int r = decltype(R)::value;
      static_for<NGP>([&](auto G) {
        constexpr int g = decltype(G)::value;
        constexpr int last = (4 * g + 3 < NQ) ? 4 * g + 3 : NQ - 1;
        if constexpr (last == r) {
          if constexpr (g + kRing < NGP)
            ring[g % kRing] = load_group(v, g + kRing);
          else
            ring[g % kRing] = load_group(vn, g + kRing - NGP);
        }
      });
    };
    f4v qb[kPDof<BLD>];
    static_for<(kPDof<BLD> < NQ ? kPDof<BLD> : NQ)>([&](auto R) {
      qb[decltype(R)::value] = read(R);
      refill(R);
    });
    __builtin_amdgcn_sched_barrier(0);
    // Without the builder wave: task j's MFMAs at stream step PM(j), its store a few reads later.
    f4v dt[TPW];
    static_for<NQ>([&](auto K) {
      constexpr int k = decltype(K)::value;
      const f4v q = qb[k % kPDof<BLD>];
      if constexpr (k + kPDof<BLD> < NQ) {
        qb[k % kPDof<BLD>] = read(std::integral_constant<int, k + kPDof<BLD>>{});
        refill(std::integral_constant<int, k + kPDof<BLD>>{});
      }
      if constexpr (!BLD) {
        static_for<TPW>([&](auto J) {
          constexpr int j = decltype(J)::value;
          constexpr int pm = (j + 1) * NQ / (TPW + 2);
          constexpr int ps = (pm + 6 < NQ) ? pm + 6 : NQ - 1;
          if constexpr (k == pm) dt[j] = build_task(j);
          if constexpr (k == ps) store_at(pbw + j * PBSTEP, kb, nbuf, dt[j]);
        });
      }
      // With the builder wave: the first three quarters of each wave's reads
      // at raised priority, the rest at the base level, so that waves ahead
      // yield the SIMD to the ones behind and the waves finish closer together.
      if constexpr (BLD && k == 0) __builtin_amdgcn_s_setprio(1);
      if constexpr (BLD && k == (3 * NQ) / 4) __builtin_amdgcn_s_setprio(0);
      constexpr int tap = k % TAPS;
      constexpr int sh = (tap / COLS) * kGridW + tap % COLS;
      tap_add<sh & 3>(acc[k / TAPS], q);
      // Keep the stream in this order: left free, the scheduler hoists every
      // row-offset load of the subspace to the top and runs out of registers.
      __builtin_amdgcn_sched_barrier(0);
    });
    if constexpr (BLD) {
      lds_count_done(sync_addr + 4u * (1u + buf));  // this wave's reads of table v are done
    } else {
      lds_barrier();
    }
    buf ^= 1;
  }

  // ---- epilogue
  if (ll == 31) return;  // its slots belong to the next tile
  if (partial) {
    // partial[split][tile][t][j][l]: slot 4 l + j of the tile; 124 contiguous bytes per store.
    float* dst = partial + (((size_t)split * p.tiles + tile) * p.ct_pad + tw0) * 128 + ll;
#pragma unroll
    for (int i = 0; i < TWP; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) dst[(size_t)i * 128 + 32 * j] = acc[i][j];
    return;
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int s = s0 + 4 * ll + j;
    const int row = s / p.Wg, xl = s - row * p.Wg;
    const int g = row / p.Hg, yo = row - g * p.Hg;
    const int n = g / p.S, xo = (g - n * p.S) * p.sw + xl;
    if (n >= p.N || yo >= p.Ho || xl >= p.sw || xo >= p.Wo) continue;
#pragma unroll
    for (int i = 0; i < TWP; ++i) {
      const int t = tw0 + i;
      if (t >= p.Ct) break;
      float v = acc[i][j] + (bias ? bias[t] : 0.f);
      if (p.relu) v = fmaxf(v, 0.f);
      y[(((size_t)n * p.Ct + t) * p.Ho + yo) * p.Wo + xo] = v;
    }
  }
}

// rowoff[v][wslot][g][h][e]: for read k = 4 g + e of wave slot wslot (channel
// block wslot / 16, wave wslot % 16) and half h, the table-row byte offset
// (code x row stride) of channel tc (wslot / 16) + (2 (wslot % 16) + h) TWP +
// k / taps at tap k % taps of subspace v, the code clamped to K-1; reads past
// the wave's stream, the builder wave's slot and channels past C_t give row
// 0.  One thread per dword.
struct HalfCodeMap {
  int Ct, dk, M, K, row_bytes, tc, twp, gw, nwslots, ngp;  // gw: gathering waves of a workgroup
};

__global__ __launch_bounds__(256) void half_rowoff_kernel(CodeStream codes, HalfCodeMap q, int total,
                                                          uint32_t* __restrict__ out) {
  const int taps = q.dk * q.dk;
  const int nq = q.twp * taps;
  for (int o = blockIdx.x * blockDim.x + threadIdx.x; o < total; o += gridDim.x * blockDim.x) {
    const int e = o & 3, h = (o >> 2) & 1;
    int r = o >> 3;
    const int g = r % q.ngp;
    r /= q.ngp;
    const int wslot = r % q.nwslots, v = r / q.nwslots;
    const int k = 4 * g + e;
    uint32_t val = 0;
    if (k < nq && wslot % kWaves < q.gw) {
      const int i = k / taps, tap = k - (k / taps) * taps;
      const int t = (wslot / kWaves) * q.tc + (2 * (wslot % kWaves) + h) * q.twp + i;
      if (t < q.Ct) {
        const int ky = tap / q.dk, kx = tap - ky * q.dk;
        uint32_t c = code_at(codes, (((size_t)t * q.dk + ky) * q.dk + kx) * q.M + v);
        c = c < (uint32_t)(q.K - 1) ? c : (uint32_t)(q.K - 1);
        val = c * (uint32_t)q.row_bytes;
      }
    }
    out[o] = val;
  }
}

// y = sum over splits in order + bias, then ReLU: one thread per stored
// partial value, in the partials' order [tile][t][j][l].
__global__ __launch_bounds__(256) void half_reduce_kernel(const float* __restrict__ partial, HalfParams p,
                                                          const float* __restrict__ bias, float* __restrict__ y) {
  const size_t per_split = (size_t)p.tiles * p.ct_pad * 128;
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= per_split) return;
  const int l = (int)(i & 31), j = (int)((i >> 5) & 3);
  if (l == 31) return;  // supply lane: not stored
  const size_t r = i >> 7;
  const int t = (int)(r % p.ct_pad);
  const int tile = (int)(r / p.ct_pad);
  const int slot = tile * kTileSlots + 4 * l + j;
  const int row = slot / p.Wg, xl = slot - row * p.Wg;
  const int g = row / p.Hg, yo = row - g * p.Hg;
  const int n = g / p.S, xo = (g - n * p.S) * p.sw + xl;
  if (t >= p.Ct || n >= p.N || yo >= p.Ho || xl >= p.sw || xo >= p.Wo) return;
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

struct HalfPlan {
  HalfParams p;
  int twp, kbl, nc;
  bool bld;
  size_t lds;
};

// Estimated cost in CU clocks of a plan (gather at ~190 B/clk of LDS, the
// build hidden in it, a fixed cost per subspace for the barrier, the partial
// sums written and read back at ~3 kB/clk chip-wide).
double half_cost(const HalfParams& p, int taps, int twp, int gw) {
  const double gather = (double)gw * twp * taps * 1024.0 / 190.0;
  const double per_wg = 3000.0 + (double)p.v_per_split * (gather + 700.0);
  const double rounds = (double)((p.work + 255) / 256);
  double cost = rounds * per_wg;
  if (p.splits > 1) cost += (double)p.splits * 2.0 * p.tiles * p.ct_pad * 128 * 4 / 3.0e3;
  return cost;
}

bool make_half_plan(const ConvShape& s, HalfPlan* out) {
  if (s.stride != 1 || !(s.dk == 1 || s.dk == 3) || s.pad > s.dk - 1) return false;
  if (s.Csp > 8 || s.K > 128) return false;
  const int kbl = (s.K + 15) / 16;
  if (kWaves % kbl != 0) return false;  // 1, 2, 4 or 8 codeword blocks
  if ((long long)s.N * s.Cs * s.H * s.W * 4 > (1LL << 31) - 1) return false;  // 32-bit buffer offsets
  HalfParams p{};
  p.N = s.N; p.Cs = s.Cs; p.H = s.H; p.W = s.W; p.M = s.M; p.K = s.K; p.Csp = s.Csp; p.Ct = s.Ct;
  p.dk = s.dk; p.pad = s.pad; p.Ho = s.Ho; p.Wo = s.Wo;
  bool shared;
  if (s.dk == 1) {  // no shifts: the grid is the map itself
    p.S = 1; p.sw = s.Wo; p.Wg = s.W; p.Hg = s.H;
    shared = true;
  } else if (s.W + s.pad <= kGridW) {  // neighbours share their zero halo
    p.S = 1; p.sw = s.Wo; p.Wg = kGridW; p.Hg = s.H + s.pad;
    shared = true;
  } else {  // column strips with their own margins
    const int swmax = kGridW - (s.dk - 1);
    p.S = ceil_div(s.Wo, swmax);
    p.sw = ceil_div(s.Wo, p.S);
    if ((p.S - 1) * p.sw >= s.Wo) return false;
    p.Wg = kGridW; p.Hg = s.Ho + s.dk - 1;
    shared = false;
  }
  const long long slots = (long long)s.N * p.S * p.Hg * p.Wg;
  const long long gpos = ((long long)s.N * p.S * p.Hg + (shared ? s.pad : 0)) * p.Wg;
  if (gpos + 4096 > (1LL << 31)) return false;
  p.grid_pos = (int)gpos;
  p.tiles = (int)((slots + kTileSlots - 1) / kTileSlots);
  const int dmax = (s.dk - 1) * kGridW + (s.dk - 1);
  p.PT = 4 * (32 + (dmax >> 2));
  p.PR = (p.PT / 4) % 2 == 1 ? p.PT : p.PT + 4;
  if ((p.PT + 15) / 16 > kMaxPB) return false;
  p.tbl_bytes = kbl * 16 * p.PR * 4;
  const size_t lds = (size_t)2 * p.tbl_bytes + 32;  // + the spare slot of masked table stores, the sync words
  if (lds > kLdsBytes) return false;
  const int taps = s.dk * s.dk;
  bool found = false;
  double best = 0;
  struct Opt { bool bld; int twp; };
  for (Opt o : {Opt{true, 6}, Opt{true, 9}, Opt{true, 13}}) {
    if (s.Csp > 4 && o.twp > 9) continue;  // two channel groups: registers
    const int gw = o.bld ? kWaves - 1 : kWaves;
    HalfParams q = p;
    q.tc = 2 * gw * o.twp;
    q.tblocks = ceil_div(s.Ct, q.tc);
    q.ct_pad = q.tblocks * q.tc;
    q.nwslots = q.tblocks * kWaves;
    const int ng = (o.twp * taps + 3) / 4;
    q.ngp = (ng + kRing - 1) / kRing * kRing;
    if ((long long)s.M * q.nwslots * q.ngp * 32 > (1LL << 31) - 1) continue;
    for (int splits = 1; splits <= 16 && splits <= s.M; ++splits) {
      HalfParams r = q;
      r.v_per_split = ceil_div(s.M, splits);
      r.splits = ceil_div(s.M, r.v_per_split);
      if (r.splits != splits) continue;
      const long long work = (long long)p.tiles * q.tblocks * r.splits;
      if (work > (1LL << 30)) continue;
      r.work = (int)work;
      r.per_xcd = ceil_div(r.work, 8);
      if ((long long)r.splits * p.tiles * q.ct_pad * 128 > (1LL << 40)) continue;
      const double c = half_cost(r, taps, o.twp, gw);
      if (!found || c < best) {
        found = true;
        best = c;
        *out = {r, o.twp, kbl, s.Csp <= 4 ? 1 : 2, o.bld, lds};
      }
    }
  }
  return found;
}

struct HalfArgs {
  const float* x;
  const float* D;
  const uint32_t* rowoff;
  const float* bias;
  float* y;
  float* partial;
  hipStream_t stream;
  LaunchTimer* timer;
};

template <int ROWS, int COLS, int NC, int TWP, int KBL, bool BLD>
hipError_t launch_k(const HalfPlan& pl, const HalfArgs& a) {
  auto k = conv_half_kernel<ROWS, COLS, NC, TWP, KBL, BLD>;
  hipError_t e = allow_max_lds((const void*)k);
  if (e != hipSuccess) return e;
  return timed_launch(a.timer, k, dim3(8 * pl.p.per_xcd), dim3(kThreads), (uint32_t)pl.lds, a.stream, a.x, a.D,
                      a.rowoff, a.bias, a.y, a.partial, pl.p);
}

template <int ROWS, int COLS, int NC, int TWP, bool BLD>
hipError_t launch_kbl(const HalfPlan& pl, const HalfArgs& a) {
  switch (pl.kbl) {
    case 1: return launch_k<ROWS, COLS, NC, TWP, 1, BLD>(pl, a);
    case 2: return launch_k<ROWS, COLS, NC, TWP, 2, BLD>(pl, a);
    case 4: return launch_k<ROWS, COLS, NC, TWP, 4, BLD>(pl, a);
    default: return launch_k<ROWS, COLS, NC, TWP, 8, BLD>(pl, a);
  }
}

// Only the builder-wave form is instantiated: on the layers measured (AlexNet
// conv3-conv5, VGG-16 conv3) the every-wave-builds form was slower.
template <int ROWS, int COLS>
hipError_t launch_taps(const HalfPlan& pl, const HalfArgs& a) {
  if (!pl.bld) return hipErrorInvalidConfiguration;
  if (pl.nc == 2) return pl.twp == 6 ? launch_kbl<ROWS, COLS, 2, 6, true>(pl, a) : launch_kbl<ROWS, COLS, 2, 9, true>(pl, a);
  switch (pl.twp) {
    case 6: return launch_kbl<ROWS, COLS, 1, 6, true>(pl, a);
    case 9: return launch_kbl<ROWS, COLS, 1, 9, true>(pl, a);
    default: return launch_kbl<ROWS, COLS, 1, 13, true>(pl, a);
  }
}

}  // namespace

bool conv_half_supported(const ConvShape& s) {
  HalfPlan pl;
  return make_half_plan(s, &pl);
}

namespace {

// Workspace of a plan: the row offsets, then (split plans) the partials.
struct HalfWs {
  size_t n_ro, ro_bytes, partial_elems, total;
};

HalfWs half_ws(const HalfPlan& pl) {
  const HalfParams& p = pl.p;
  HalfWs w;
  w.n_ro = (size_t)p.M * p.nwslots * p.ngp * 8;  // dwords
  w.ro_bytes = (w.n_ro * 4 + 255) & ~(size_t)255;
  w.partial_elems = (size_t)p.splits * p.tiles * p.ct_pad * 128;
  w.total = w.ro_bytes + (p.splits > 1 ? w.partial_elems * sizeof(float) : 0);
  return w;
}

}  // namespace

size_t conv_half_workspace(const ConvShape& s) {
  HalfPlan pl;
  return make_half_plan(s, &pl) ? half_ws(pl).total : 0;
}

hipError_t launch_conv_half(const ConvShape& s, const float* x, const float* D, CodeStream codes, const float* bias,
                            int relu, float* y, hipStream_t stream, const Workspace* ws) {
  HalfPlan pl;
  if (!make_half_plan(s, &pl)) return hipErrorInvalidConfiguration;
  pl.p.relu = relu;
  static const bool trace = getenv("QCNN_TRACE_PLAN") && *getenv("QCNN_TRACE_PLAN") == '1';
  const HalfParams& p = pl.p;
  if (trace)
    fprintf(stderr, "qcnn conv_half: taps %dx%d S=%d sw=%d Wg=%d Hg=%d tiles=%d %s TWP=%d tc=%d tblocks=%d "
            "splits=%d work=%d PR=%d PT=%d kbl=%d lds=%zu\n", s.dk, s.dk, p.S, p.sw, p.Wg, p.Hg, p.tiles,
            pl.bld ? "builder-wave" : "all-build", pl.twp, p.tc, p.tblocks, p.splits, p.work, p.PR, p.PT, pl.kbl,
            pl.lds);
  const HalfWs w = half_ws(pl);
  const size_t n_ro = w.n_ro, partial_elems = w.partial_elems;
  Scratch scratch;
  hipError_t e = scratch.take(stream, w.total, ws);
  if (e != hipSuccess) return e;
  char* base = scratch.get();
  uint32_t* rowoff = reinterpret_cast<uint32_t*>(base);
  float* partial = p.splits > 1 ? reinterpret_cast<float*>(base + w.ro_bytes) : nullptr;
  const HalfCodeMap cm{p.Ct, p.dk, p.M, p.K, p.PR * 4, p.tc, pl.twp, pl.bld ? kWaves - 1 : kWaves, p.nwslots, p.ngp};
  hipLaunchKernelGGL(half_rowoff_kernel, dim3((unsigned)std::min<size_t>(4096, ceil_div_z(n_ro, 256))), dim3(256), 0,
                     stream, codes, cm, (int)n_ro, rowoff);
  e = hipGetLastError();
  if (e == hipSuccess) {
    LaunchTimer timer(ws == nullptr || ws->timed);
    const HalfArgs a{x, D, rowoff, bias, y, partial, stream, &timer};
    e = s.dk == 1 ? launch_taps<1, 1>(pl, a) : launch_taps<3, 3>(pl, a);
  }
  if (e == hipSuccess && partial) {
    hipLaunchKernelGGL(half_reduce_kernel, dim3((unsigned)ceil_div_z(partial_elems / p.splits, 256)), dim3(256), 0,
                       stream, partial, p, bias, y);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace qcnn
