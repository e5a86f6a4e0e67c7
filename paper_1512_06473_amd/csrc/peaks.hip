// Peak probes: the denominators of the rooflines the benchmark reports,
// measured on the current device (not part of the paper's method).
//
// LDS: one 1024-thread workgroup per CU streams ds_read_b128 over 64 KB of
// its LDS: each wave reads blocks of eight 1 KB runs (lane l at offset 16 l
// of a run: conflict-free), the blocks sliding through the buffer, with the
// compiler free to keep reads of consecutive blocks in flight and to wait
// for them in order; four XOR chains keep all the data live.  The shader
// clock under that load is taken from the shader-clock counter (s_memtime)
// against the constant-rate counter (s_memrealtime) over each workgroup's
// loop.
//
// VALU: clocks per wave64 instruction per SIMD for the three instructions a
// gather read issues (plain add, DPP add, address multiply-add).
//
// HBM: streams of 16-byte loads over a caller buffer (read), of 16-byte
// stores to a second buffer (write), and of both (copy), one 16 KB chunk per
// 256-thread block over the whole buffer.
#include <algorithm>
#include <vector>

#include "qcnn_internal.h"

namespace qcnn {
namespace {

constexpr int kLdsProbeThreads = 1024;
constexpr int kLdsProbeBytes = 64 * 1024;
constexpr int kLdsProbeIters = 8192;  // of 8 reads per thread

__global__ __launch_bounds__(kLdsProbeThreads, 1) void lds_probe_kernel(uint32_t* __restrict__ sink,
                                                                        unsigned long long* __restrict__ stamps) {
  extern __shared__ uint4 buf[];  // kLdsProbeBytes
  const int tid = threadIdx.x;
  for (int i = tid; i < kLdsProbeBytes / 16; i += kLdsProbeThreads) buf[i] = make_uint4(i, i + 1, i + 2, i + 3);
  __syncthreads();
  const int lane = tid & 63, wave = tid >> 6;
  // Row r of wave w is (8 w + r) mod 64: 1 KB rows, so the largest byte read
  // is 63 * 1024 + 63 * 16 + 15 < 64 KB.
  const char* lb = reinterpret_cast<const char*>(buf);
  // A block is eight 1 KB runs at `off` + 0 .. 7 KB + 15, so `off` stays
  // below kWrap = 56 KB and every read stays inside the 64 KB; waves start
  // 3.5 KB apart (at most 15 * 3584 + 63 * 16 = 54768 < kWrap).
  constexpr uint32_t kWrap = kLdsProbeBytes - 8192;
  uint32_t off = (uint32_t)(wave * 3584 + lane * 16);
  uint4 acc = make_uint4(0, 0, 0, 0);
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  const unsigned long long r0 = __builtin_amdgcn_s_memrealtime();
  for (int it = 0; it < kLdsProbeIters; ++it) {
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const uint4 v = *reinterpret_cast<const uint4*>(lb + off + r * 1024);
      acc.x ^= v.x;
      acc.y ^= v.y;
      acc.z ^= v.z;
      acc.w ^= v.w;
    }
    off += 8192;  // next block, wrapped below kWrap
    if (off >= kWrap) off -= kWrap;
  }
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  const unsigned long long r1 = __builtin_amdgcn_s_memrealtime();
  sink[blockIdx.x * kLdsProbeThreads + tid] = acc.x ^ acc.y ^ acc.z ^ acc.w;
  if (tid == 0) {
    stamps[2 * blockIdx.x] = t1 - t0;
    stamps[2 * blockIdx.x + 1] = r1 - r0;
  }
}

// VALU issue probe: 16 waves per CU (4 per SIMD), each running kValuIters
// iterations of 8 independent instructions of one kind (chains 8 apart, so
// no dependency stalls), timed by wave 0 with s_memtime between two
// barriers.  MODE 0: v_add_f32; 1: v_add_f32 with a DPP wave_shl:1 operand
// (its source registers are not written in the loop); 2: v_mad_u32_u24.
constexpr int kValuIters = 4096;

template <int MODE>
__global__ __launch_bounds__(1024, 1) void valu_probe_kernel(uint32_t* __restrict__ sink,
                                                             unsigned long long* __restrict__ stamps) {
  const int tid = threadIdx.x;
  float f[8], g[8];
  uint32_t u[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    f[k] = (float)(tid + k);
    g[k] = 1.0f / (float)(k + 1 + (tid & 7));
    u[k] = (uint32_t)(tid * 8 + k);
  }
  const uint32_t cm = (uint32_t)(tid & 255) | 1u, ca = (uint32_t)tid >> 3;
  __syncthreads();
  const unsigned long long t0 = __builtin_amdgcn_s_memtime();
  for (int it = 0; it < kValuIters; ++it) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      if constexpr (MODE == 0) f[k] += g[k];
      // The instruction itself, written out so that the compiler neither
      // hoists the loop-invariant DPP move nor widens the 24-bit multiply;
      // the DPP source g[k] is written only before the loop (no VALU-write /
      // DPP-read hazard inside it).
      if constexpr (MODE == 1)
        asm volatile("v_add_f32_dpp %0, %1, %0 wave_shl:1 row_mask:0xf bank_mask:0xf" : "+v"(f[k]) : "v"(g[k]));
      if constexpr (MODE == 2) asm volatile("v_mad_u32_u24 %0, %0, %1, %2" : "+v"(u[k]) : "v"(cm), "v"(ca));
    }
  }
  __syncthreads();
  const unsigned long long t1 = __builtin_amdgcn_s_memtime();
  uint32_t acc = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) acc ^= __float_as_uint(f[k]) ^ u[k];
  sink[blockIdx.x * 1024 + tid] = acc;
  if (tid == 0) stamps[blockIdx.x] = t1 - t0;
}

// Each thread handles 4 consecutive-by-256 uint4 of a 1024-element chunk per
// block (coalesced 4 KB per wave), one chunk per block over the whole buffer.
__global__ __launch_bounds__(256) void hbm_read_kernel(const uint4* __restrict__ src, size_t n16,
                                                       uint32_t* __restrict__ sink) {
  const size_t base = (size_t)blockIdx.x * 1024 + threadIdx.x;
  uint32_t acc = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const size_t i = base + 256 * k;
    if (i < n16) {
      const uint4 v = src[i];
      acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
  }
  if (acc == 0x9e3779b9u) sink[threadIdx.x] = acc;  // practically never: keeps the loads live
}

__global__ __launch_bounds__(256) void hbm_write_kernel(uint4* __restrict__ dst, size_t n16) {
  const size_t base = (size_t)blockIdx.x * 1024 + threadIdx.x;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const size_t i = base + 256 * k;
    if (i < n16) dst[i] = make_uint4((uint32_t)i, 1u, 2u, 3u);
  }
}

__global__ __launch_bounds__(256) void hbm_copy_kernel(const uint4* __restrict__ src, size_t n16,
                                                       uint4* __restrict__ dst) {
  const size_t base = (size_t)blockIdx.x * 1024 + threadIdx.x;
  uint4 v[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const size_t i = base + 256 * k;
    if (i < n16) v[k] = src[i];
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const size_t i = base + 256 * k;
    if (i < n16) dst[i] = v[k];
  }
}

// Elapsed milliseconds of `launch` enqueued `reps` times between two events.
template <class F>
hipError_t time_ms(hipStream_t stream, int reps, F launch, float* ms) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipError_t e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  if (e == hipSuccess) e = hipEventRecord(e0, stream);
  for (int r = 0; r < reps && e == hipSuccess; ++r) e = launch();
  if (e == hipSuccess) e = hipEventRecord(e1, stream);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  if (e == hipSuccess) e = hipEventElapsedTime(ms, e0, e1);
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  return e;
}

}  // namespace

hipError_t probe_lds(hipStream_t stream, double* bytes_per_clk_cu, double* clock_ghz, double* bytes_per_s) {
  int dev = 0, cus = 0, wall_khz = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&wall_khz, hipDeviceAttributeWallClockRate, dev);
  if (e != hipSuccess) return e;
  if (cus < 1 || wall_khz < 1) return hipErrorInvalidValue;
  const int blocks = cus;
  uint32_t* sink = nullptr;
  unsigned long long* stamps = nullptr;
  e = hipMalloc((void**)&sink, (size_t)blocks * kLdsProbeThreads * sizeof(uint32_t));
  if (e == hipSuccess) e = hipMalloc((void**)&stamps, (size_t)blocks * 2 * sizeof(unsigned long long));
  float ms = 0.f;
  if (e == hipSuccess) e = allow_max_lds((const void*)lds_probe_kernel);
  auto launch = [&]() {
    hipLaunchKernelGGL(lds_probe_kernel, dim3(blocks), dim3(kLdsProbeThreads), kLdsProbeBytes, stream, sink, stamps);
    return hipGetLastError();
  };
  if (e == hipSuccess) e = time_ms(stream, 1, launch, &ms);  // warm-up (clock ramp)
  if (e == hipSuccess) e = time_ms(stream, 3, launch, &ms);
  std::vector<unsigned long long> host((size_t)blocks * 2);
  if (e == hipSuccess)
    e = hipMemcpy(host.data(), stamps, host.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost);
  if (sink) (void)hipFree(sink);
  if (stamps) (void)hipFree(stamps);
  if (e != hipSuccess) return e;
  // Shader clock: shader-clock ticks over constant-rate ticks, per workgroup
  // of the last launch, the median over workgroups.
  std::vector<double> ghz;
  for (int b = 0; b < blocks; ++b)
    if (host[2 * b + 1] > 0) ghz.push_back((double)host[2 * b] / ((double)host[2 * b + 1] / (wall_khz * 1e3)) / 1e9);
  if (ghz.empty()) return hipErrorInvalidValue;
  std::sort(ghz.begin(), ghz.end());
  const double clk = ghz[ghz.size() / 2];
  const double bytes = (double)blocks * kLdsProbeThreads * kLdsProbeIters * 8.0 * 16.0;
  const double sec = ms * 1e-3 / 3.0;
  *clock_ghz = clk;
  *bytes_per_s = bytes / sec;
  *bytes_per_clk_cu = bytes / (sec * clk * 1e9 * cus);
  return hipSuccess;
}

hipError_t probe_valu(hipStream_t stream, double* add_clk, double* dpp_add_clk, double* mad_clk) {
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  if (cus < 1) return hipErrorInvalidValue;
  uint32_t* sink = nullptr;
  unsigned long long* stamps = nullptr;
  e = hipMalloc((void**)&sink, (size_t)cus * 1024 * sizeof(uint32_t));
  if (e == hipSuccess) e = hipMalloc((void**)&stamps, (size_t)cus * sizeof(unsigned long long));
  double* out[3] = {add_clk, dpp_add_clk, mad_clk};
  std::vector<unsigned long long> host(cus);
  for (int mode = 0; mode < 3 && e == hipSuccess; ++mode) {
    for (int rep = 0; rep < 2 && e == hipSuccess; ++rep) {  // the first launch warms the clock up
      if (mode == 0) hipLaunchKernelGGL(valu_probe_kernel<0>, dim3(cus), dim3(1024), 0, stream, sink, stamps);
      if (mode == 1) hipLaunchKernelGGL(valu_probe_kernel<1>, dim3(cus), dim3(1024), 0, stream, sink, stamps);
      if (mode == 2) hipLaunchKernelGGL(valu_probe_kernel<2>, dim3(cus), dim3(1024), 0, stream, sink, stamps);
      e = hipGetLastError();
      if (e == hipSuccess) e = hipStreamSynchronize(stream);
    }
    if (e == hipSuccess) e = hipMemcpy(host.data(), stamps, host.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost);
    if (e == hipSuccess) {
      std::vector<unsigned long long> h(host);
      std::sort(h.begin(), h.end());
      // clocks per wave instruction on one SIMD: 4 waves per SIMD, 8 per iteration
      *out[mode] = (double)h[h.size() / 2] / (4.0 * 8.0 * kValuIters);
    }
  }
  if (sink) (void)hipFree(sink);
  if (stamps) (void)hipFree(stamps);
  return e;
}

hipError_t probe_hbm(const void* src, void* dst, size_t bytes, hipStream_t stream, double* read_bps,
                     double* write_bps, double* copy_bps) {
  const size_t n16 = bytes / 16;
  const size_t nblk = (n16 + 1023) / 1024;
  if (nblk > 0x7fffffffu) return hipErrorInvalidValue;
  const unsigned blocks = (unsigned)nblk;
  uint32_t* sink = nullptr;
  hipError_t e = hipMalloc((void**)&sink, 256 * sizeof(uint32_t));
  float ms = 0.f;
  const int reps = 5;
  auto rd = [&]() {
    hipLaunchKernelGGL(hbm_read_kernel, dim3(blocks), dim3(256), 0, stream, static_cast<const uint4*>(src), n16, sink);
    return hipGetLastError();
  };
  auto wr = [&]() {
    hipLaunchKernelGGL(hbm_write_kernel, dim3(blocks), dim3(256), 0, stream, static_cast<uint4*>(dst), n16);
    return hipGetLastError();
  };
  auto cp = [&]() {
    hipLaunchKernelGGL(hbm_copy_kernel, dim3(blocks), dim3(256), 0, stream, static_cast<const uint4*>(src), n16,
                       static_cast<uint4*>(dst));
    return hipGetLastError();
  };
  if (e == hipSuccess) e = time_ms(stream, 1, rd, &ms);
  if (e == hipSuccess) e = time_ms(stream, reps, rd, &ms);
  if (e == hipSuccess) *read_bps = (double)n16 * 16.0 * reps / (ms * 1e-3);
  if (e == hipSuccess) e = time_ms(stream, 1, wr, &ms);
  if (e == hipSuccess) e = time_ms(stream, reps, wr, &ms);
  if (e == hipSuccess) *write_bps = (double)n16 * 16.0 * reps / (ms * 1e-3);
  if (e == hipSuccess) e = time_ms(stream, 1, cp, &ms);
  if (e == hipSuccess) e = time_ms(stream, reps, cp, &ms);
  if (e == hipSuccess) *copy_bps = 2.0 * (double)n16 * 16.0 * reps / (ms * 1e-3);
  if (sink) (void)hipFree(sink);
  return e;
}

}  // namespace qcnn
