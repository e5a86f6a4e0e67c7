// Internal declarations shared by the HIP sources of libqcnn (not installed).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stddef.h>
#include <stdint.h>

#include <algorithm>

#include "qcnn.h"

namespace qcnn {

constexpr int kWave = 64;  // CDNA wavefront width

inline int ceil_div(int a, int b) { return (a + b - 1) / b; }
inline size_t ceil_div_z(size_t a, size_t b) { return (a + b - 1) / b; }

// The caller's codes as a stream of `bits` bits per code, base 4-byte
// aligned (the C ABI checks it): bits = 8 is one byte per code
// (qcnn_conv_forward, qcnn_fc_forward); otherwise the packed form of Table 1
// (qcnn_pack_codes): code i is stream bits i bits .. i bits + bits - 1, value
// bit j at stream bit i bits + j, stream bit q = bit q % 8 of byte q / 8;
// bits = 0 when K = 1 (every code is 0 and nothing is stored).
struct CodeStream {
  const uint8_t* p;
  int bits;
};

// Bits per packed code for K codewords: 0 for K = 1, else ceil(log2 K).
inline int code_bits(int K) {
  int b = 0;
  while ((1 << b) < K) ++b;
  return b;
}

// Code `idx` of a stream.  Whole aligned dwords are loaded, so a wave-uniform
// index becomes scalar loads; an aligned dword never straddles a page, and a
// dword that holds any bit of a code lies within the stream's last dword, so
// the bytes past the last code cannot fault.
__device__ __forceinline__ uint32_t code_at(const CodeStream& s, size_t idx) {
  const uint32_t* w = reinterpret_cast<const uint32_t*>(s.p);
  if (s.bits == 8) return (w[idx >> 2] >> ((uint32_t)(idx & 3) * 8u)) & 0xffu;
  if (s.bits == 0) return 0u;
  const size_t bit = idx * (size_t)s.bits;
  const uint32_t sh = (uint32_t)(bit & 31);
  uint32_t v = w[bit >> 5] >> sh;
  if (sh + (uint32_t)s.bits > 32u) v |= w[(bit >> 5) + 1] << (32u - sh);
  return v & ((1u << s.bits) - 1u);
}

// ---------------------------------------------------------------- launchers
// Each returns a hipError_t from the launch (hipGetLastError after it).

struct ConvShape {
  int N, Cs, H, W, M, K, Csp, Ct, dk, stride, pad, Ho, Wo;
};

hipError_t launch_lut_build(const float* x, int N, int Cs, int H, int W, const float* D, int M, int K,
                            int Csp, float* lut, hipStream_t stream);

// Device memory a call brings for its temporaries in place of the
// library's per-stream buffer (the allocation-free entry point's static
// array, or a region of a buffer the caller already holds): nothing is
// allocated, and a call that needs more than `bytes` fails with
// hipErrorOutOfMemory before it launches anything.  `timed`: the main kernel
// is timed as on the allocating path (the allocation-free path records no
// events).
struct Workspace {
  char* ptr;
  size_t bytes;
  bool timed = false;
};

// Max pooling of a conv layer's output, k x k windows with stride s and no
// padding, to an H_p x W_p map.
struct PoolSpec {
  int k, s, Hp, Wp;
};

// The conv kernel family for a layer: 0 the flat kernel, 1 the two-table
// kernel, 2 the generic one; conv_kernel_pick gives the one the launchers
// pick now (QCNN_CONV_KERNEL is read per call; host-side, no HIP call).  The
// launchers below take a `kind` from it, or -1 to pick at the call.
int conv_kernel_pick(const ConvShape& s);

// Returns hipErrorInvalidConfiguration when no tiling fits the device.
// With `ws` the temporaries live there (nothing allocated, no timing events).
hipError_t launch_conv_forward(const ConvShape& s, const float* x, const float* D, CodeStream codes,
                               const float* bias, int relu, float* y, hipStream_t stream,
                               const Workspace* ws = nullptr, int kind = -1);

// Bytes of temporaries launch_conv_forward needs for this layer with kernel
// `kind` (-1: the one it would pick now; host-side, no HIP call).
size_t conv_forward_workspace(const ConvShape& s, int kind = -1);

// The conv layer followed by max pooling, y: [N][C_t][H_p][W_p].  A layer
// whose subspaces the stride-1/strided flat kernel splits over workgroups
// takes the window maxima in its split-sum kernel; any other layer writes
// its full map to a temporary that the max-pool kernel reads.
hipError_t launch_conv_pool_forward(const ConvShape& s, const float* x, const float* D, CodeStream codes,
                                    const float* bias, int relu, const PoolSpec& pool, float* y,
                                    hipStream_t stream, int kind = -1);

hipError_t launch_fc_forward(int N, int Cs, int M, int K, int Csp, int Ct, const float* x, const float* D,
                             CodeStream codes, const float* bias, int relu, float* y, hipStream_t stream);

hipError_t launch_maxpool(const float* x, int N, int C, int H, int W, int k, int s, int Ho, int Wo, float* y,
                          hipStream_t stream);

// Zeroes *bad (a device int), then counts the codes >= K into it.
hipError_t launch_code_check(CodeStream codes, size_t n, int K, int* bad, hipStream_t stream);

// Packed codes (glue.hip): byte codes -> the stream of `bits` bits per code,
// written as ceil(n bits / 32) whole dwords (bits past the last code are 0);
// and back, one byte per code.
hipError_t launch_pack_codes(const uint8_t* codes, size_t n, int bits, uint32_t* packed, hipStream_t stream);
hipError_t launch_unpack_codes(CodeStream packed, size_t n, uint8_t* codes, hipStream_t stream);

// True when the conv kernels can tile this layer (host-side, no HIP call).
bool conv_supported(const ConvShape& s);

// Stride-1 kernel on the flattened padded grid (conv_flat.hip).
bool conv_flat_supported(const ConvShape& s);
size_t conv_flat_workspace(const ConvShape& s);
// True when the flat kernel's plan for this layer splits the subspaces over
// workgroups and an output map fits its pooled split-sum kernel (which then
// takes the pooling maxima).
bool conv_flat_pools(const ConvShape& s);
// With `pool`, y is the pooled map; only for a layer with conv_flat_pools.
hipError_t launch_conv_flat(const ConvShape& s, const float* x, const float* D, CodeStream codes,
                            const float* bias, int relu, float* y, hipStream_t stream, const Workspace* ws,
                            const PoolSpec* pool = nullptr);
// The same call in two parts, for a layer whose codes are re-laid once and
// then serve many calls: the re-laid codes' size (0 when the flat kernel
// cannot tile the layer), the re-layout into codes8, and the call on codes8
// (which must come from launch_conv_flat_codes for the same shape).  With
// `pool`, a plan the split sum cannot pool writes its full map to the
// library's workspace and a max-pool kernel reads it.
size_t conv_flat_code_bytes(const ConvShape& s);
hipError_t launch_conv_flat_codes(const ConvShape& s, CodeStream codes, uint8_t* codes8, hipStream_t stream);
hipError_t launch_conv_flat_relaid(const ConvShape& s, const float* x, const float* D, const uint8_t* codes8,
                                   const float* bias, int relu, float* y, hipStream_t stream,
                                   const PoolSpec* pool = nullptr);

// Stride-1 3x3 / 1x1 kernel with two tables in LDS and half-wave table rows
// (conv_half.hip): C'_s <= 8, K <= 128.
bool conv_half_supported(const ConvShape& s);
size_t conv_half_workspace(const ConvShape& s);
hipError_t launch_conv_half(const ConvShape& s, const float* x, const float* D, CodeStream codes,
                            const float* bias, int relu, float* y, hipStream_t stream, const Workspace* ws);

// Brackets the main kernel of a call with a pair of HIP events on its
// stream while kernel timing is switched on (qcnn_timing_enable); does
// nothing otherwise (or when `enabled` is false: the allocation-free path
// creates no events).  The pairs are read back by qcnn_timing_read.
class KernelTimer {
 public:
  explicit KernelTimer(hipStream_t stream, bool enabled = true);
  ~KernelTimer();
  KernelTimer(const KernelTimer&) = delete;
  KernelTimer& operator=(const KernelTimer&) = delete;

 private:
  hipStream_t stream_;
  hipEvent_t start_ = nullptr;
};

// Times one kernel launch exactly while kernel timing is on: its two events
// go to hipExtLaunchKernelGGL, which stamps them at the dispatch's start and
// end (an event recorded before the launch would also count the dispatch
// latency).  The pair is handed to qcnn_timing_read by the destructor once
// launched() was called; with timing off (or `enabled` false) both events are
// null and the launch is a plain one.
class LaunchTimer {
 public:
  explicit LaunchTimer(bool enabled = true);
  ~LaunchTimer();
  LaunchTimer(const LaunchTimer&) = delete;
  LaunchTimer& operator=(const LaunchTimer&) = delete;
  hipEvent_t start() const { return start_; }
  hipEvent_t stop() const { return stop_; }
  void launched() { launched_ = true; }

 private:
  hipEvent_t start_ = nullptr, stop_ = nullptr;
  bool launched_ = false;
};

// hipExtLaunchKernelGGL with the events of `t` (may be null: no timing).
template <typename... Args, typename F = void (*)(Args...)>
hipError_t timed_launch(LaunchTimer* t, F kernel, const dim3& grid, const dim3& block, uint32_t lds,
                        hipStream_t stream, Args... args) {
  hipExtLaunchKernelGGL(kernel, grid, block, lds, stream, t ? t->start() : nullptr, t ? t->stop() : nullptr, 0,
                        args...);
  const hipError_t e = hipGetLastError();
  if (e == hipSuccess && t) t->launched();
  return e;
}

// FC layer with tables of 4 subspaces per phase and 128-bit gathers over
// images (fc_tiled.hip): K <= 64, C's <= 8.
bool fc_tiled_supported(int N, int Cs, int M, int K, int Csp, int Ct);
hipError_t launch_fc_tiled(int N, int Cs, int M, int K, int Csp, int Ct, const float* x, const float* D,
                           CodeStream codes, const float* bias, int relu, float* y, hipStream_t stream);
// The same call in two parts (as for the flat conv kernel): the re-laid
// codes' size (0 when the kernel cannot tile the layer), the re-layout, and
// the call on codes re-laid for the same shape.
size_t fc_tiled_code_bytes(int N, int Cs, int M, int K, int Csp, int Ct);
hipError_t launch_fc_tiled_codes(int N, int Cs, int M, int K, int Csp, int Ct, CodeStream codes, uint32_t* codes4,
                                 hipStream_t stream);
hipError_t launch_fc_tiled_relaid(int N, int Cs, int M, int K, int Csp, int Ct, const float* x, const float* D,
                                  const uint32_t* codes4, const float* bias, int relu, float* y,
                                  hipStream_t stream);

// Parameter quantization (quantize.hip); objective arrays are device float64.
hipError_t launch_pq_assign(int Ct, int Cs, int dk, const float* W, const float* D, int M, int K, int Csp,
                            uint8_t* codes, double* objective, hipStream_t stream);
hipError_t launch_pq_update(int Ct, int Cs, int dk, const float* W, const uint8_t* codes, int M, int K, int Csp,
                            float* D, int* counts, hipStream_t stream);
hipError_t launch_pq_kmeans(int Ct, int Cs, int dk, const float* W, int M, int K, int Csp, int iters, float* D,
                            uint8_t* codes, double* objective, hipStream_t stream);

// Error correction (Sec. 3.3), the normal equations of one sub-codeword's
// least-squares fit: x with G x = b by elimination in channel order without
// row exchanges; a pivot <= 1e-12 x max diag(G) (or <= 0) drops that
// coordinate (x = 0).  A: N x N working storage of the calling lane
// (registers once the loops are unrolled, or LDS).
template <int N>
__device__ __forceinline__ void solve_normal(const double* __restrict__ Gm, const double (&bin)[N], double* A,
                                             double (&x)[N]) {
  double y[N];
  bool live[N];
  double scale = 0.0;
#pragma unroll
  for (int i = 0; i < N; ++i) {
#pragma unroll
    for (int j = 0; j < N; ++j) A[i * N + j] = Gm[i * N + j];
    y[i] = bin[i];
    scale = fmax(scale, Gm[i * N + i]);
  }
#pragma unroll
  for (int j = 0; j < N; ++j) {
    live[j] = A[j * N + j] > 1e-12 * scale && A[j * N + j] > 0.0;
    if (live[j]) {
#pragma unroll
      for (int i = j + 1; i < N; ++i) {
        const double f = A[i * N + j] / A[j * N + j];
#pragma unroll
        for (int q = j; q < N; ++q) A[i * N + q] -= f * A[j * N + q];
        y[i] -= f * y[j];
      }
    }
  }
#pragma unroll
  for (int j = N - 1; j >= 0; --j) {
    x[j] = 0.0;
    if (live[j]) {
      double s = y[j];
#pragma unroll
      for (int i = j + 1; i < N; ++i)
        if (live[i]) s -= A[j * N + i] * x[i];
      x[j] = s / A[j * N + j];
    }
  }
}

// Error-corrected quantization of a fully-connected layer (ec_fc.hip):
// S [N][C_s], T [N][C_t] fp32; D [M][K][C'_s] and codes [C_t][M] updated in
// place; objective (nullable) [1 + sweeps M] float64.
hipError_t launch_ec_fc(int N, int Cs, int Ct, int M, int K, int Csp, const float* S, const float* T, float* D,
                        uint8_t* codes, int sweeps, int inner, double* objective, hipStream_t stream);

// Error-corrected quantization of a conv layer (ec_conv.hip): S [N][C_s][H][W],
// T [N][C_t][H_o][W_o] fp32; D [M][K][C'_s] and codes [C_t][d_k][d_k][M]
// updated in place; objective (nullable) [1 + sweeps M] float64.
hipError_t launch_ec_conv(int N, int Cs, int H, int W, int Ct, int dk, int stride, int pad, int M, int K, int Csp,
                          const float* S, const float* T, float* D, uint8_t* codes, int sweeps, int inner,
                          double* objective, hipStream_t stream);

// The library's own stream-ordered memory pool on the current device
// (scratch.cpp): created on first use, it keeps freed memory for reuse (its
// release threshold is unlimited) and leaves the device's default pool, and
// every other user of it, untouched.
hipError_t library_pool(hipMemPool_t* pool);
// hipMallocFromPoolAsync from the library pool; free with hipFreeAsync.
hipError_t pool_alloc(void** ptr, size_t bytes, hipStream_t stream);

// LDS per workgroup on gfx950.
constexpr size_t kLdsBytes = 160 * 1024;

// The library's workspace for one call on `stream` (scratch.cpp): a buffer
// per (device, stream), grown in stream order and kept until the process
// ends.  The object holds that buffer's lock until it is destroyed, so it
// must live until every kernel of the call has been enqueued.
class Scratch {
 public:
  Scratch() = default;
  ~Scratch();
  Scratch(const Scratch&) = delete;
  Scratch& operator=(const Scratch&) = delete;
  hipError_t acquire(hipStream_t stream, size_t bytes);
  // `bytes` of the caller's workspace when `ws` is given (nothing is
  // allocated or locked; hipErrorOutOfMemory if it is too small), else
  // acquire(stream, bytes).
  hipError_t take(hipStream_t stream, size_t bytes, const Workspace* ws);
  char* get() const { return static_cast<char*>(ptr_); }

 private:
  void* slot_ = nullptr;
  void* ptr_ = nullptr;
};

// The allocation-free conv forward's device scratch (noalloc.hip): its size,
// and its address on the current device (looked up once per device).
size_t noalloc_scratch_bytes();
hipError_t noalloc_scratch(char** ptr);

// Peak probes (peaks.hip): LDS read bytes per clock per CU with the shader
// clock measured under that load, and HBM read / write / copy bytes per second.
hipError_t probe_lds(hipStream_t stream, double* bytes_per_clk_cu, double* clock_ghz, double* bytes_per_s);
hipError_t probe_hbm(const void* src, void* dst, size_t bytes, hipStream_t stream, double* read_bps,
                     double* write_bps, double* copy_bps);
hipError_t probe_valu(hipStream_t stream, double* add_clk, double* dpp_add_clk, double* mad_clk);

// Lets `kernel` take up to kLdsBytes of dynamic LDS (once per device).
hipError_t allow_max_lds(const void* kernel);

}  // namespace qcnn
