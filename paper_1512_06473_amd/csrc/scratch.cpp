// Library-owned device scratch and per-kernel launch attributes.
//
// A layer call needs a workspace for its re-laid-out codes and, when its
// subspaces are split over workgroups, for the partial sums.  Allocating it
// per call (hipMallocAsync / hipFreeAsync) cost tens of microseconds of host
// time per call, as much as the layer's kernels on the GPU, so the library
// keeps one buffer per (device, stream) instead:
//   * grown in stream order: the old buffer is released with hipFreeAsync on
//     the same stream (after the calls that used it) and a larger one is
//     taken from the library's own memory pool (hipMallocFromPoolAsync);
//   * held until the process ends (the library pool keeps freed memory;
//     the device's default pool is left as the application set it);
//   * locked for the whole enqueue of a call, so that two host threads that
//     share a stream cannot interleave their kernels over one buffer.
// Calls on different streams use different buffers and never wait for each
// other.
#include <map>
#include <memory>
#include <mutex>
#include <set>
#include <utility>

#include "qcnn_internal.h"

namespace qcnn {
namespace {

struct Slot {
  std::mutex mu;  // held by a Scratch for the enqueue of one call
  void* ptr = nullptr;
  size_t bytes = 0;
};

std::mutex g_mu;  // guards the maps (not the slots' contents)

std::map<std::pair<int, hipStream_t>, std::unique_ptr<Slot>>& slots() {
  static auto* m = new std::map<std::pair<int, hipStream_t>, std::unique_ptr<Slot>>();
  return *m;
}

}  // namespace

Scratch::~Scratch() {
  if (slot_) static_cast<Slot*>(slot_)->mu.unlock();
}

hipError_t Scratch::acquire(hipStream_t stream, size_t bytes) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  Slot* s;
  {
    std::lock_guard<std::mutex> lock(g_mu);
    auto& p = slots()[{dev, stream}];
    if (!p) p.reset(new Slot());
    s = p.get();
  }
  s->mu.lock();
  slot_ = s;
  if (s->bytes < bytes) {
    if (s->ptr) {
      e = hipFreeAsync(s->ptr, stream);
      s->ptr = nullptr;
      s->bytes = 0;
      if (e != hipSuccess) return e;
    }
    // Round up to 2 MiB and to 5/4 of the request, so that a few layers of
    // growing size do not each trigger a new allocation.
    const size_t want = ((bytes + bytes / 4) + ((size_t)2 << 20) - 1) & ~(((size_t)2 << 20) - 1);
    e = pool_alloc(&s->ptr, want, stream);
    if (e != hipSuccess) {
      s->ptr = nullptr;
      return e;
    }
    s->bytes = want;
  }
  ptr_ = s->ptr;
  return hipSuccess;
}

hipError_t library_pool(hipMemPool_t* pool) {
  static std::mutex mu;
  static auto* pools = new std::map<int, hipMemPool_t>();
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  auto it = pools->find(dev);
  if (it != pools->end()) {
    *pool = it->second;
    return hipSuccess;
  }
  hipMemPoolProps props = {};
  props.allocType = hipMemAllocationTypePinned;
  props.handleTypes = hipMemHandleTypeNone;
  props.location.type = hipMemLocationTypeDevice;
  props.location.id = dev;
  hipMemPool_t p = nullptr;
  e = hipMemPoolCreate(&p, &props);
  if (e != hipSuccess) return e;
  uint64_t threshold = UINT64_MAX;  // keep freed memory for the next call
  e = hipMemPoolSetAttribute(p, hipMemPoolAttrReleaseThreshold, &threshold);
  if (e != hipSuccess) {
    (void)hipMemPoolDestroy(p);
    return e;
  }
  (*pools)[dev] = p;  // kept until the process ends
  *pool = p;
  return hipSuccess;
}

hipError_t pool_alloc(void** ptr, size_t bytes, hipStream_t stream) {
  hipMemPool_t pool = nullptr;
  hipError_t e = library_pool(&pool);
  if (e != hipSuccess) return e;
  return hipMallocFromPoolAsync(ptr, bytes, pool, stream);
}

hipError_t Scratch::take(hipStream_t stream, size_t bytes, const Workspace* ws) {
  if (!ws) return acquire(stream, bytes);
  if (bytes > ws->bytes) return hipErrorOutOfMemory;
  ptr_ = ws->ptr;
  return hipSuccess;
}

hipError_t allow_max_lds(const void* kernel) {
  static std::mutex mu;
  static auto* done = new std::set<std::pair<int, const void*>>();
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(mu);
  if (done->count({dev, kernel})) return hipSuccess;
  e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsBytes);
  if (e == hipSuccess) done->insert({dev, kernel});
  return e;
}

}  // namespace qcnn
