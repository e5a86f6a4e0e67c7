// Fused PQ convolution: table tile in LDS, gather-accumulate from it.
//
// Paper: Sec. 3.2, Eq. (7).  With the kernels quantized, the response at
// output position p_t of channel c_t is
//     T_{p_t}(c_t) = sum_{(p_k, p_s)} sum_m < D^(m)_{k_m(c_t, p_k)}, S^(m)_{p_s} >,
// and the inner products are read from a table pre-computed over the input
// positions (the paragraph after Eq. (7)).  Table 1: d_s^2 C_s K multiply-adds
// for the table plus d_t^2 C_t d_k^2 M additions for the responses.
//
// MI355X mapping (generic kernel, any stride / kernel / padding):
//   * a workgroup owns one image n, a toh x tow tile of output positions and
//     a block of TC = 4 * TW output channels;
//   * for each subspace m it builds, in LDS, the table over the input window
//     of its tile: lut[k][iy][ix], ih = (toh-1) s + d_k rows by
//     iw = (tow-1) s + d_k columns, with zeros where the window hangs over the
//     padding (<D_k, 0> = 0, so those reads add nothing);
//   * lanes own output positions (G per lane), waves own TW output channels.
//     A code depends only on (c_t, p_k, m), never on the position, so it is
//     wave-uniform: one scalar load serves 64 lanes, and the lanes read one
//     table row at consecutive positions;
//   * the table never leaves LDS.
#include <stdlib.h>
#include <string.h>

#include "qcnn_internal.h"

namespace qcnn {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr size_t kLdsLimit = 160 * 1024;

struct ConvParams {
  int N, Cs, H, W, M, K, Csp, Ct, dk, stride, pad, Ho, Wo;
  int toh, tow, tiles_x, ih, iw, tileP, tc;
  int relu;
};

template <int CSP, int G, int TW>
__global__ __launch_bounds__(kThreads) void conv_pq_generic(const float* __restrict__ x, const float* __restrict__ D,
                                                            CodeStream codes, const float* __restrict__ bias,
                                                            float* __restrict__ y, ConvParams p) {
  extern __shared__ float lut[];  // [K][ih * iw]
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int n = blockIdx.z;
  const int ty = blockIdx.x / p.tiles_x, tx = blockIdx.x - ty * p.tiles_x;
  const int oy0 = ty * p.toh, ox0 = tx * p.tow;
  const int iy0 = oy0 * p.stride - p.pad, ix0 = ox0 * p.stride - p.pad;
  const int csp = CSP > 0 ? CSP : p.Csp;
  const size_t HW = (size_t)p.H * p.W;
  const int tileP = p.tileP;

  // Output positions of this lane inside the tile.
  int off[G], oyl[G], oxl[G];
  bool valid[G];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const int q = lane + kWave * g;
    const int oy = q / p.tow, ox = q - (q / p.tow) * p.tow;
    valid[g] = q < p.toh * p.tow && oy0 + oy < p.Ho && ox0 + ox < p.Wo;
    oyl[g] = oy;
    oxl[g] = ox;
    off[g] = valid[g] ? (oy * p.stride) * p.iw + ox * p.stride : 0;
  }

  float acc[TW][G];
#pragma unroll
  for (int i = 0; i < TW; ++i)
#pragma unroll
    for (int g = 0; g < G; ++g) acc[i][g] = 0.f;

  const int tbase = blockIdx.y * p.tc + wave * TW;
  const int taps = p.dk * p.dk;
  const uint32_t kmax = (uint32_t)(p.K - 1);
  constexpr int XCAP = CSP > 0 ? CSP : 16;

  for (int m = 0; m < p.M; ++m) {
    __syncthreads();  // the previous subspace's gathers are done with the tile
    // ---- table tile for subspace m (Sec. 3.1 test phase, over input positions)
    const float* xm = x + ((size_t)n * p.Cs + (size_t)m * csp) * HW;
    const float* Dm = D + (size_t)m * p.K * csp;
    for (int q = tid; q < tileP; q += kThreads) {
      const int iy = q / p.iw, ix = q - (q / p.iw) * p.iw;
      const int gy = iy0 + iy, gx = ix0 + ix;
      const bool in = (unsigned)gy < (unsigned)p.H && (unsigned)gx < (unsigned)p.W;
      float xv[XCAP];
#pragma unroll
      for (int j = 0; j < XCAP; ++j)
        xv[j] = (j < csp && in) ? xm[(size_t)j * HW + (size_t)gy * p.W + gx] : 0.f;
      for (int k = 0; k < p.K; ++k) {
        const float* d = Dm + (size_t)k * csp;
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < XCAP; ++j)
          if (j < csp) s = fmaf(d[j], xv[j], s);
        lut[k * tileP + q] = s;
      }
    }
    __syncthreads();
    // ---- gather-accumulate, Eq. (7): one table read + one add per (c_t, p_k)
#pragma unroll
    for (int i = 0; i < TW; ++i) {
      const int t = tbase + i;
      if (t < p.Ct) {
        const size_t cbase = (size_t)t * taps * p.M + m;
        for (int ky = 0; ky < p.dk; ++ky)
          for (int kx = 0; kx < p.dk; ++kx) {
            uint32_t code = code_at(codes, cbase + (size_t)(ky * p.dk + kx) * p.M);
            code = code < kmax ? code : kmax;
            const float* row = lut + code * tileP + ky * p.iw + kx;
#pragma unroll
            for (int g = 0; g < G; ++g) acc[i][g] += row[off[g]];
          }
      }
    }
  }

  // ---- epilogue: bias, ReLU, store
#pragma unroll
  for (int i = 0; i < TW; ++i) {
    const int t = tbase + i;
    if (t >= p.Ct) continue;
    const float b = bias ? bias[t] : 0.f;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (!valid[g]) continue;
      float v = acc[i][g] + b;
      if (p.relu) v = fmaxf(v, 0.f);
      y[(((size_t)n * p.Ct + t) * p.Ho + oy0 + oyl[g]) * p.Wo + ox0 + oxl[g]] = v;
    }
  }
}

constexpr int kTW = 8;  // output channels per wave

struct Tiling {
  int G, toh, tow, ih, iw;
  size_t lds;
};

// Pick the output tile: at most 64 G positions, the table window must fit
// LDS; among those, the one with the lowest estimated VALU work (table build
// over the window + gathers over the lanes, idle lanes included).
bool choose_tiling(const ConvShape& s, Tiling* best) {
  double best_cost = 0;
  bool found = false;
  const int tc = kWaves * kTW;
  const int tblocks = ceil_div(s.Ct, tc);
  for (int G = 1; G <= 4; ++G) {
    for (int tow = 1; tow <= s.Wo && tow <= kWave * G; ++tow) {
      const int toh_max = (kWave * G) / tow;
      for (int toh = 1; toh <= toh_max && toh <= s.Ho; ++toh) {
        if (toh * tow <= kWave * (G - 1)) continue;  // a smaller G would do
        const int ih = (toh - 1) * s.stride + s.dk, iw = (tow - 1) * s.stride + s.dk;
        const size_t lds = (size_t)s.K * ih * iw * sizeof(float);
        if (lds > kLdsLimit) continue;
        const double tiles = (double)ceil_div(s.Ho, toh) * ceil_div(s.Wo, tow);
        const double build = ceil_div(ih * iw, kThreads) * (double)kWaves * s.K * (s.Csp + 1);
        const double gather = (double)kWaves * kTW * s.dk * s.dk * G * 2.0;
        const double cost = tiles * tblocks * s.N * s.M * (build + gather);
        if (!found || cost < best_cost) {
          found = true;
          best_cost = cost;
          *best = {G, toh, tow, ih, iw, lds};
        }
      }
    }
  }
  return found;
}

struct ConvPtrs {
  const float* x;
  const float* D;
  CodeStream codes;
  const float* bias;
  float* y;
  bool timed;  // false on the allocation-free path (no timing events)
};

template <int CSP, int G>
hipError_t launch_g(const ConvPtrs& a, const ConvParams& p, dim3 grid, size_t lds, hipStream_t stream) {
  auto k = conv_pq_generic<CSP, G, kTW>;
  hipError_t e = allow_max_lds((const void*)k);
  if (e != hipSuccess) return e;
  LaunchTimer timer(a.timed);
  return timed_launch(&timer, k, grid, dim3(kThreads), (uint32_t)lds, stream, a.x, a.D, a.codes, a.bias, a.y, p);
}

template <int CSP>
hipError_t launch_csp(const ConvPtrs& a, const ConvParams& p, int G, dim3 grid, size_t lds, hipStream_t stream) {
  switch (G) {
    case 1: return launch_g<CSP, 1>(a, p, grid, lds, stream);
    case 2: return launch_g<CSP, 2>(a, p, grid, lds, stream);
    case 3: return launch_g<CSP, 3>(a, p, grid, lds, stream);
    default: return launch_g<CSP, 4>(a, p, grid, lds, stream);
  }
}

}  // namespace

bool conv_supported(const ConvShape& s) {
  Tiling t;
  return conv_half_supported(s) || conv_flat_supported(s) || choose_tiling(s, &t);
}

namespace {

// Which conv kernel family serves a layer: the first of conv_flat,
// conv_half, conv_pq_generic that can tile it.  QCNN_CONV_KERNEL = half puts
// the two-table kernel first, = generic skips the first two (for comparisons
// and for tests of every kernel on shapes the default one also serves).
int conv_kernel_choice() {
  const char* v = getenv("QCNN_CONV_KERNEL");  // read per call: tests switch it within one process
  if (!v) return 0;
  if (strcmp(v, "half") == 0) return 1;
  if (strcmp(v, "generic") == 0) return 2;
  return 0;
}

enum class ConvKernel { kFlat, kHalf, kGeneric };

ConvKernel pick_conv_kernel(const ConvShape& s) {
  const int choice = conv_kernel_choice();
  if (choice == 1 && conv_half_supported(s)) return ConvKernel::kHalf;
  if (choice != 2 && conv_flat_supported(s)) return ConvKernel::kFlat;
  if (choice != 2 && conv_half_supported(s)) return ConvKernel::kHalf;
  return ConvKernel::kGeneric;
}

}  // namespace

int conv_kernel_pick(const ConvShape& s) { return static_cast<int>(pick_conv_kernel(s)); }

namespace {

ConvKernel kind_or_pick(const ConvShape& s, int kind) {
  return kind < 0 ? pick_conv_kernel(s) : static_cast<ConvKernel>(kind);
}

}  // namespace

size_t conv_forward_workspace(const ConvShape& s, int kind) {
  switch (kind_or_pick(s, kind)) {
    case ConvKernel::kFlat: return conv_flat_workspace(s);
    case ConvKernel::kHalf: return conv_half_workspace(s);
    default: return 0;  // the generic kernel reads the caller's codes directly
  }
}

hipError_t launch_conv_forward(const ConvShape& s, const float* x, const float* D, CodeStream codes,
                               const float* bias, int relu, float* y, hipStream_t stream, const Workspace* ws,
                               int kind) {
  const ConvKernel k = kind_or_pick(s, kind);
  if (k == ConvKernel::kFlat) return launch_conv_flat(s, x, D, codes, bias, relu, y, stream, ws);
  if (k == ConvKernel::kHalf) return launch_conv_half(s, x, D, codes, bias, relu, y, stream, ws);
  Tiling t;
  if (!choose_tiling(s, &t)) return hipErrorInvalidConfiguration;
  const ConvPtrs a{x, D, codes, bias, y, ws == nullptr || ws->timed};
  ConvParams p;
  p.N = s.N;
  p.Cs = s.Cs;
  p.H = s.H;
  p.W = s.W;
  p.M = s.M;
  p.K = s.K;
  p.Csp = s.Csp;
  p.Ct = s.Ct;
  p.dk = s.dk;
  p.stride = s.stride;
  p.pad = s.pad;
  p.Ho = s.Ho;
  p.Wo = s.Wo;
  p.toh = t.toh;
  p.tow = t.tow;
  p.tiles_x = ceil_div(s.Wo, t.tow);
  p.ih = t.ih;
  p.iw = t.iw;
  p.tileP = t.ih * t.iw;
  p.tc = kWaves * kTW;
  p.relu = relu;
  dim3 grid(ceil_div(s.Ho, t.toh) * p.tiles_x, ceil_div(s.Ct, p.tc), s.N);
  switch (s.Csp) {
    case 1: return launch_csp<1>(a, p, t.G, grid, t.lds, stream);
    case 2: return launch_csp<2>(a, p, t.G, grid, t.lds, stream);
    case 3: return launch_csp<3>(a, p, t.G, grid, t.lds, stream);
    case 4: return launch_csp<4>(a, p, t.G, grid, t.lds, stream);
    case 8: return launch_csp<8>(a, p, t.G, grid, t.lds, stream);
    default: return launch_csp<0>(a, p, t.G, grid, t.lds, stream);
  }
}

hipError_t launch_conv_pool_forward(const ConvShape& s, const float* x, const float* D, CodeStream codes,
                                    const float* bias, int relu, const PoolSpec& pool, float* y,
                                    hipStream_t stream, int kind) {
  const ConvKernel k = kind_or_pick(s, kind);
  if (k == ConvKernel::kFlat && conv_flat_pools(s))
    return launch_conv_flat(s, x, D, codes, bias, relu, y, stream, nullptr, &pool);
  // One library buffer holds the layer's own temporaries and, after them,
  // its full output map, which the max-pool kernel reads.
  const size_t conv_ws = (conv_forward_workspace(s, static_cast<int>(k)) + 255) & ~(size_t)255;
  const size_t full = (size_t)s.N * s.Ct * s.Ho * s.Wo * sizeof(float);
  Scratch scratch;
  hipError_t e = scratch.acquire(stream, conv_ws + full);
  if (e != hipSuccess) return e;
  float* ymap = reinterpret_cast<float*>(scratch.get() + conv_ws);
  const Workspace ws{scratch.get(), conv_ws, true};
  e = launch_conv_forward(s, x, D, codes, bias, relu, ymap, stream, &ws, static_cast<int>(k));
  if (e != hipSuccess) return e;
  return launch_maxpool(ymap, s.N, s.Ct, s.Ho, s.Wo, pool.k, pool.s, pool.Hp, pool.Wp, y, stream);
}

}  // namespace qcnn
