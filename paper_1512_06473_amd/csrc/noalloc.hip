// Device scratch of the allocation-free conv forward (qcnn_conv_forward_noalloc).
//
// The array below is the only memory that entry point uses besides the
// caller's inputs and outputs: the re-laid-out codes and the partial sums of
// split layers, and the counter of the optional code check.  It is part of
// the library's code object, so every device the library runs on holds its
// own copy, at its own address, from the module's load until the process
// ends.  In host code the array's name is not a device address: the address
// is looked up once per device with hipGetSymbolAddress and kept, and only
// that address is passed to kernels.
#include <mutex>

#include "qcnn_internal.h"

namespace {

constexpr size_t kNoAllocScratchBytes = (size_t)64 << 20;  // 64 MiB per device

static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
char* g_ptr[kMaxDevices] = {};

}  // namespace

namespace qcnn {

size_t noalloc_scratch_bytes() { return kNoAllocScratchBytes; }

hipError_t noalloc_scratch(char** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_ptr[dev] = static_cast<char*>(p);
  }
  *ptr = g_ptr[dev];
  return hipSuccess;
}

}  // namespace qcnn
