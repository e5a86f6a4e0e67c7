// C ABI of libqcnn: host-side validation, then kernel launches on the
// caller's stream.  Every check runs before the first HIP call, so a rejected
// call launches nothing and leaves every output untouched.
#include <stdlib.h>
#include <string.h>

#include <atomic>
#include <initializer_list>
#include <mutex>
#include <new>
#include <utility>
#include <vector>

#include "qcnn_internal.h"

namespace {

using qcnn::ConvShape;

constexpr int kMaxGridYZ = 65535;
constexpr size_t kMaxElems = (size_t)1 << 40;

bool env_flag(const char* name) {
  const char* v = getenv(name);
  return v && *v && strcmp(v, "0") != 0;
}

// [a, a + na) and [b, b + nb) (bytes) overlap?
bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + nb && b0 < a0 + na;
}

bool mul_ok(size_t* acc, size_t v) {
  if (v != 0 && *acc > kMaxElems / v) return false;
  *acc *= v;
  return true;
}

// Elements of a product of positive ints, or 0 on overflow past kMaxElems.
size_t elems(std::initializer_list<int> dims) {
  size_t n = 1;
  for (int d : dims)
    if (!mul_ok(&n, (size_t)d)) return 0;
  return n;
}

qcnn_status check_pq(int N, int Cs, int M, int K, int Csp) {
  if (N < 1 || Cs < 1 || M < 1 || Csp < 1) return QCNN_ERR_SHAPE;
  if (K < 1 || K > 256) return QCNN_ERR_K_RANGE;
  if ((long long)M * Csp != Cs) return QCNN_ERR_SHAPE;
  if (Csp > 16) return QCNN_ERR_UNSUPPORTED;
  if (N > kMaxGridYZ || M > kMaxGridYZ) return QCNN_ERR_UNSUPPORTED;
  return QCNN_OK;
}

qcnn_status hip_status(hipError_t e) { return e == hipSuccess ? QCNN_OK : QCNN_ERR_HIP; }

// Once per device: create the library's memory pool (the per-call
// workspaces are recycled from it instead of remapped).
bool prepare_device() {
  hipMemPool_t pool = nullptr;
  return qcnn::library_pool(&pool) == hipSuccess;
}

// Bytes of the stream of n codes of `bits` bits each as the library writes
// it (whole dwords), or of one byte per code when bits == 8.
size_t code_stream_bytes(size_t n, int bits) {
  return bits == 8 ? n : (n * (size_t)bits + 31) / 32 * 4;
}

// QCNN_CHECK_CODES=1: count codes >= K on the device and wait for the answer.
// The counter is `counter` (a device int the caller owns) or a temporary.
qcnn_status check_codes(qcnn::CodeStream codes, size_t n, int K, hipStream_t st, int* counter = nullptr) {
  static const bool enabled = env_flag("QCNN_CHECK_CODES");
  if (!enabled || (1 << codes.bits) <= K) return QCNN_OK;  // no stored value can reach K
  int* bad = counter;
  int host = 0;
  hipError_t e = hipSuccess;
  if (!bad) e = qcnn::pool_alloc((void**)&bad, sizeof(int), st);
  if (e != hipSuccess) return QCNN_ERR_HIP;
  e = qcnn::launch_code_check(codes, n, K, bad, st);
  if (e == hipSuccess) e = hipMemcpyAsync(&host, bad, sizeof(int), hipMemcpyDeviceToHost, st);
  hipError_t e2 = counter ? hipSuccess : hipFreeAsync(bad, st);
  if (e == hipSuccess) e = e2;
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return QCNN_ERR_HIP;
  return host ? QCNN_ERR_CODE_RANGE : QCNN_OK;
}

// Kernel timing state: event pairs recorded by KernelTimer, read back and
// destroyed by qcnn_timing_read.
struct TimingState {
  std::mutex mu;
  std::atomic<bool> on{false};
  std::vector<std::pair<hipEvent_t, hipEvent_t>> pairs;
  bool failed = false;
};

TimingState& timing() {
  static TimingState t;
  return t;
}

}  // namespace

namespace qcnn {

KernelTimer::KernelTimer(hipStream_t stream, bool enabled) : stream_(stream) {
  if (!enabled || !timing().on.load(std::memory_order_relaxed)) return;
  if (hipEventCreate(&start_) != hipSuccess) {
    start_ = nullptr;
  } else if (hipEventRecord(start_, stream_) != hipSuccess) {
    (void)hipEventDestroy(start_);
    start_ = nullptr;
  }
  if (!start_) {
    std::lock_guard<std::mutex> lock(timing().mu);
    timing().failed = true;
  }
}

KernelTimer::~KernelTimer() {
  if (!start_) return;
  hipEvent_t stop = nullptr;
  TimingState& t = timing();
  if (hipEventCreate(&stop) != hipSuccess || hipEventRecord(stop, stream_) != hipSuccess) {
    if (stop) (void)hipEventDestroy(stop);
    (void)hipEventDestroy(start_);
    std::lock_guard<std::mutex> lock(t.mu);
    t.failed = true;
    return;
  }
  std::lock_guard<std::mutex> lock(t.mu);
  t.pairs.emplace_back(start_, stop);
}

LaunchTimer::LaunchTimer(bool enabled) {
  if (!enabled || !timing().on.load(std::memory_order_relaxed)) return;
  if (hipEventCreate(&start_) != hipSuccess || hipEventCreate(&stop_) != hipSuccess) {
    if (start_) (void)hipEventDestroy(start_);
    if (stop_) (void)hipEventDestroy(stop_);
    start_ = stop_ = nullptr;
    std::lock_guard<std::mutex> lock(timing().mu);
    timing().failed = true;
  }
}

LaunchTimer::~LaunchTimer() {
  if (!start_) return;
  if (!launched_) {
    (void)hipEventDestroy(start_);
    (void)hipEventDestroy(stop_);
    return;
  }
  std::lock_guard<std::mutex> lock(timing().mu);
  timing().pairs.emplace_back(start_, stop_);
}

}  // namespace qcnn

extern "C" {

qcnn_status qcnn_timing_enable(int enable) {
  timing().on.store(enable != 0);
  return QCNN_OK;
}

namespace {

// Reads and destroys every recorded pair; per-launch milliseconds go to
// `each` (the first `capacity` of them, when `each` is not null).
qcnn_status drain_timing(double* total_ms, long long* launches, double* each, long long capacity) {
  TimingState& t = timing();
  std::lock_guard<std::mutex> lock(t.mu);
  double sum = 0.0;
  bool ok = !t.failed;
  long long i = 0;
  for (auto& pr : t.pairs) {
    float ms = 0.f;
    if (hipEventSynchronize(pr.second) != hipSuccess || hipEventElapsedTime(&ms, pr.first, pr.second) != hipSuccess)
      ok = false;
    sum += ms;
    if (each && i < capacity) each[i] = ms;
    ++i;
    (void)hipEventDestroy(pr.first);
    (void)hipEventDestroy(pr.second);
  }
  if (total_ms) *total_ms = sum;
  *launches = (long long)t.pairs.size();
  t.pairs.clear();
  t.failed = false;
  return ok ? QCNN_OK : QCNN_ERR_HIP;
}

}  // namespace

qcnn_status qcnn_timing_read(double* total_ms, long long* launches) {
  if (!total_ms || !launches) return QCNN_ERR_NULL;
  return drain_timing(total_ms, launches, nullptr, 0);
}

qcnn_status qcnn_timing_read_each(double* ms_each, long long capacity, long long* launches) {
  if (!ms_each || !launches) return QCNN_ERR_NULL;
  if (capacity < 0) return QCNN_ERR_SHAPE;
  return drain_timing(nullptr, launches, ms_each, capacity);
}

int qcnn_version(void) { return 1; }

int qcnn_out_size(int in, int k, int stride, int pad) {
  if (in < 1 || k < 1 || stride < 1 || pad < 0) return 0;
  const long long span = (long long)in + 2LL * pad - k;
  if (span < 0) return 0;
  return (int)(span / stride + 1);
}

const char* qcnn_status_string(qcnn_status s) {
  switch (s) {
    case QCNN_OK: return "ok";
    case QCNN_ERR_NULL: return "a required pointer is NULL";
    case QCNN_ERR_SHAPE: return "invalid shape (size < 1, C_s != M*C's, empty output or overflow)";
    case QCNN_ERR_K_RANGE: return "K must be in [1, 256]";
    case QCNN_ERR_CODE_RANGE: return "a code is >= K";
    case QCNN_ERR_HIP: return "HIP runtime error";
    case QCNN_ERR_UNSUPPORTED: return "layer not supported by the kernels (C's > 16, grid or LDS limits)";
    case QCNN_ERR_ALIAS: return "an output overlaps an input";
    case QCNN_ERR_WORKSPACE: return "the layer needs more scratch than qcnn_conv_forward_noalloc holds";
  }
  return "unknown status";
}

qcnn_status qcnn_lut_build(const float* x, int N, int C_s, int H, int W, const float* codebooks, int M, int K,
                           int Csp, float* lut, void* stream) {
  if (!x || !codebooks || !lut) return QCNN_ERR_NULL;
  if (H < 1 || W < 1) return QCNN_ERR_SHAPE;
  qcnn_status s = check_pq(N, C_s, M, K, Csp);
  if (s != QCNN_OK) return s;
  const size_t nx = elems({N, C_s, H, W}), nd = elems({M, K, Csp});
  const size_t nl = elems({N, M, K, H, W});
  if (!nx || !nd || !nl) return QCNN_ERR_SHAPE;
  if (overlap(lut, nl * 4, x, nx * 4) || overlap(lut, nl * 4, codebooks, nd * 4)) return QCNN_ERR_ALIAS;
  return hip_status(qcnn::launch_lut_build(x, N, C_s, H, W, codebooks, M, K, Csp, lut, (hipStream_t)stream));
}

}  // extern "C"

namespace {

// Shape of a conv call (with pool_k or pool_s non-zero, of the conv and the
// max-pool after it) and the sizes of its arrays.
struct ConvCall {
  ConvShape sh;
  bool pooled;
  int Hp, Wp;
  size_t nx, nd, nc, ny, cb;  // elements of x, codebooks, codes, y; bytes of the code stream
};

// The host-side checks of a conv call that do not involve x and y.
qcnn_status check_conv(int N, int C_s, int H, int W, int M, int K, int Csp, const uint8_t* codes, int bits, int C_t,
                       int d_k, int stride, int pad, int pool_k, int pool_s, ConvCall* c) {
  if (H < 1 || W < 1 || C_t < 1 || d_k < 1 || stride < 1 || pad < 0) return QCNN_ERR_SHAPE;
  qcnn_status s = check_pq(N, C_s, M, K, Csp);
  if (s != QCNN_OK) return s;
  const int Ho = qcnn_out_size(H, d_k, stride, pad), Wo = qcnn_out_size(W, d_k, stride, pad);
  if (Ho < 1 || Wo < 1) return QCNN_ERR_SHAPE;
  c->pooled = pool_k != 0 || pool_s != 0;
  c->Hp = c->pooled ? qcnn_out_size(Ho, pool_k, pool_s, 0) : Ho;
  c->Wp = c->pooled ? qcnn_out_size(Wo, pool_k, pool_s, 0) : Wo;
  if (c->pooled && (pool_k < 1 || pool_s < 1 || c->Hp < 1 || c->Wp < 1)) return QCNN_ERR_SHAPE;
  c->nx = elems({N, C_s, H, W});
  c->nd = elems({M, K, Csp});
  c->nc = elems({C_t, d_k, d_k, M});
  c->ny = elems({N, C_t, c->Hp, c->Wp});
  if (!c->nx || !c->nd || !c->nc || !c->ny) return QCNN_ERR_SHAPE;
  c->cb = code_stream_bytes(c->nc, bits);
  if ((uintptr_t)codes & 3) return QCNN_ERR_UNSUPPORTED;
  c->sh = ConvShape{N, C_s, H, W, M, K, Csp, C_t, d_k, stride, pad, Ho, Wo};
  if (!qcnn::conv_supported(c->sh)) return QCNN_ERR_UNSUPPORTED;
  if (qcnn::ceil_div(C_t, 32) > kMaxGridYZ) return QCNN_ERR_UNSUPPORTED;
  return QCNN_OK;
}

// Body of qcnn_conv_forward (bits = 8), qcnn_conv_forward_packed, (with
// noalloc) qcnn_conv_forward_noalloc and (with pool_k > 0)
// qcnn_conv_pool_forward.
qcnn_status conv_forward(const float* x, int N, int C_s, int H, int W, const float* codebooks, int M, int K,
                         int Csp, const uint8_t* codes, int bits, int C_t, int d_k, int stride, int pad,
                         const float* bias, int relu, float* y, void* stream, bool noalloc = false,
                         int pool_k = 0, int pool_s = 0) {
  if (!x || !codebooks || !codes || !y) return QCNN_ERR_NULL;
  ConvCall c{};  // sizes 0 until check_conv has computed them
  qcnn_status s = check_conv(N, C_s, H, W, M, K, Csp, codes, bits, C_t, d_k, stride, pad, pool_k, pool_s, &c);
  // An overlap of y with an input is reported before the codes' alignment
  // and the kernels' limits, as far as the sizes are known.
  if (s != QCNN_OK && s != QCNN_ERR_UNSUPPORTED) return s;
  if (c.ny && (overlap(y, c.ny * 4, x, c.nx * 4) || overlap(y, c.ny * 4, codebooks, c.nd * 4) ||
               overlap(y, c.ny * 4, codes, c.cb) || overlap(y, c.ny * 4, bias, (size_t)C_t * 4)))
    return QCNN_ERR_ALIAS;
  if (s != QCNN_OK) return s;
  const ConvShape& sh = c.sh;
  const int Hp = c.Hp, Wp = c.Wp;
  const bool pooled = c.pooled;
  const size_t nc = c.nc;
  hipStream_t st = (hipStream_t)stream;
  const qcnn::CodeStream cs{codes, bits};
  if (noalloc) {
    // The static scratch: the layer's temporaries, then 256 bytes for the
    // code-check counter.  Checked before any HIP call.
    const size_t room = qcnn::noalloc_scratch_bytes() - 256;
    const int kind = qcnn::conv_kernel_pick(sh);  // one choice for the size check and the launch
    if (qcnn::conv_forward_workspace(sh, kind) > room) return QCNN_ERR_WORKSPACE;
    char* base = nullptr;
    if (qcnn::noalloc_scratch(&base) != hipSuccess) return QCNN_ERR_HIP;
    s = check_codes(cs, nc, K, st, reinterpret_cast<int*>(base + room));
    if (s != QCNN_OK) return s;
    const qcnn::Workspace ws{base, room};
    return hip_status(qcnn::launch_conv_forward(sh, x, codebooks, cs, bias, relu ? 1 : 0, y, st, &ws, kind));
  }
  if (!prepare_device()) return QCNN_ERR_HIP;
  s = check_codes(cs, nc, K, st);
  if (s != QCNN_OK) return s;
  if (pooled)
    return hip_status(qcnn::launch_conv_pool_forward(sh, x, codebooks, cs, bias, relu ? 1 : 0,
                                                     qcnn::PoolSpec{pool_k, pool_s, Hp, Wp}, y, st));
  return hip_status(qcnn::launch_conv_forward(sh, x, codebooks, cs, bias, relu ? 1 : 0, y, st));
}

// Body of qcnn_fc_forward (bits = 8) and qcnn_fc_forward_packed.
qcnn_status fc_forward(const float* x, int N, int C_s, const float* codebooks, int M, int K, int Csp,
                       const uint8_t* codes, int bits, int C_t, const float* bias, int relu, float* y, void* stream) {
  if (!x || !codebooks || !codes || !y) return QCNN_ERR_NULL;
  if (C_t < 1) return QCNN_ERR_SHAPE;
  qcnn_status s = check_pq(N, C_s, M, K, Csp);
  if (s != QCNN_OK) return s;
  const size_t nx = elems({N, C_s}), nd = elems({M, K, Csp}), nc = elems({C_t, M}), ny = elems({N, C_t});
  if (!nx || !nd || !nc || !ny) return QCNN_ERR_SHAPE;
  const size_t cb = code_stream_bytes(nc, bits);
  if (overlap(y, ny * 4, x, nx * 4) || overlap(y, ny * 4, codebooks, nd * 4) || overlap(y, ny * 4, codes, cb) ||
      overlap(y, ny * 4, bias, (size_t)C_t * 4))
    return QCNN_ERR_ALIAS;
  if ((uintptr_t)codes & 3) return QCNN_ERR_UNSUPPORTED;
  hipStream_t st = (hipStream_t)stream;
  if (!prepare_device()) return QCNN_ERR_HIP;
  const qcnn::CodeStream cs{codes, bits};
  s = check_codes(cs, nc, K, st);
  if (s != QCNN_OK) return s;
  return hip_status(qcnn::launch_fc_forward(N, C_s, M, K, Csp, C_t, x, codebooks, cs, bias, relu ? 1 : 0, y, st));
}

}  // namespace

extern "C" {

qcnn_status qcnn_conv_forward(const float* x, int N, int C_s, int H, int W, const float* codebooks, int M, int K,
                              int Csp, const uint8_t* codes, int C_t, int d_k, int stride, int pad,
                              const float* bias, int relu, float* y, void* stream) {
  return conv_forward(x, N, C_s, H, W, codebooks, M, K, Csp, codes, 8, C_t, d_k, stride, pad, bias, relu, y, stream);
}

qcnn_status qcnn_conv_pool_forward(const float* x, int N, int C_s, int H, int W, const float* codebooks, int M,
                                   int K, int Csp, const uint8_t* codes, int C_t, int d_k, int stride, int pad,
                                   const float* bias, int relu, int pool_k, int pool_s, float* y, void* stream) {
  if (!x || !codebooks || !codes || !y) return QCNN_ERR_NULL;
  if (pool_k < 1 || pool_s < 1) return QCNN_ERR_SHAPE;
  return conv_forward(x, N, C_s, H, W, codebooks, M, K, Csp, codes, 8, C_t, d_k, stride, pad, bias, relu, y, stream,
                      false, pool_k, pool_s);
}

qcnn_status qcnn_conv_forward_noalloc(const float* x, int N, int C_s, int H, int W, const float* codebooks, int M,
                                      int K, int Csp, const uint8_t* codes, int C_t, int d_k, int stride, int pad,
                                      const float* bias, int relu, float* y, void* stream) {
  return conv_forward(x, N, C_s, H, W, codebooks, M, K, Csp, codes, 8, C_t, d_k, stride, pad, bias, relu, y, stream,
                      true);
}

qcnn_status qcnn_conv_forward_packed(const float* x, int N, int C_s, int H, int W, const float* codebooks, int M,
                                     int K, int Csp, const uint8_t* packed_codes, int C_t, int d_k, int stride,
                                     int pad, const float* bias, int relu, float* y, void* stream) {
  if (K < 1 || K > 256) return QCNN_ERR_K_RANGE;
  return conv_forward(x, N, C_s, H, W, codebooks, M, K, Csp, packed_codes, qcnn::code_bits(K), C_t, d_k, stride,
                      pad, bias, relu, y, stream);
}

}  // extern "C"

// A conv or FC layer prepared for repeated forwards on inputs of one shape:
// its own copies of the codebooks and the bias, and the codes re-laid for the
// kernel that runs the layer (or, for a layer whose kernel reads the caller's
// layout, a copy of the code stream), in one device allocation.
struct qcnn_plan {
  bool fc;
  ConvShape sh;  // FC: N, Cs, M, K, Csp, Ct
  int relu;
  bool pooled;
  qcnn::PoolSpec pool;
  int device;
  bool relaid;
  int kind;  // conv kernel family, fixed at creation
  int bits;  // of the code copy when !relaid
  size_t nx, ny;
  void* mem;
  const float* D;
  const float* bias;
  const uint8_t* codes;
};

namespace {

// Second half of a plan's creation, after validation: the allocation, the
// copies, the code check and the re-layout (by `relayout`, or a copy of the
// code stream when it is null), then a synchronisation of the stream.
template <typename Relayout>
qcnn_status make_plan(qcnn_plan proto, const float* codebooks, size_t nd, const uint8_t* codes, size_t nc,
                      size_t code_stream, size_t relaid_bytes, const Relayout& relayout, const float* bias,
                      qcnn_plan** plan, hipStream_t st) {
  if (!prepare_device()) return QCNN_ERR_HIP;
  if (hipGetDevice(&proto.device) != hipSuccess) return QCNN_ERR_HIP;
  const int Ct = proto.sh.Ct, K = proto.sh.K;
  const qcnn::CodeStream cs{codes, proto.bits};
  // [codebooks | bias | codes | code-check counter], 256-byte aligned parts.
  auto up = [](size_t b) { return (b + 255) & ~(size_t)255; };
  const size_t d_bytes = up(nd * 4), b_bytes = bias ? up((size_t)Ct * 4) : 0;
  const size_t c_bytes = up(proto.relaid ? relaid_bytes : (code_stream + 3) / 4 * 4);
  char* mem = nullptr;
  if (hipMalloc((void**)&mem, d_bytes + b_bytes + c_bytes + 256) != hipSuccess) return QCNN_ERR_HIP;
  float* D = reinterpret_cast<float*>(mem);
  float* bcopy = bias ? reinterpret_cast<float*>(mem + d_bytes) : nullptr;
  uint8_t* ccopy = reinterpret_cast<uint8_t*>(mem + d_bytes + b_bytes);
  int* bad = reinterpret_cast<int*>(mem + d_bytes + b_bytes + c_bytes);
  int host_bad = 0;
  hipError_t e = hipSuccess;
  if ((1 << proto.bits) > K) {  // the codes are verified once, here
    e = qcnn::launch_code_check(cs, nc, K, bad, st);
    if (e == hipSuccess) e = hipMemcpyAsync(&host_bad, bad, sizeof(int), hipMemcpyDeviceToHost, st);
  }
  if (e == hipSuccess) e = hipMemcpyAsync(D, codebooks, nd * 4, hipMemcpyDeviceToDevice, st);
  if (e == hipSuccess && bias) e = hipMemcpyAsync(bcopy, bias, (size_t)Ct * 4, hipMemcpyDeviceToDevice, st);
  if (e == hipSuccess)
    e = proto.relaid ? relayout(cs, ccopy) : hipMemcpyAsync(ccopy, codes, code_stream, hipMemcpyDeviceToDevice, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  qcnn_status s = QCNN_OK;
  if (e == hipSuccess && host_bad) s = QCNN_ERR_CODE_RANGE;
  qcnn_plan* p = nullptr;
  if (e == hipSuccess && s == QCNN_OK) {
    proto.mem = mem;
    proto.D = D;
    proto.bias = bcopy;
    proto.codes = ccopy;
    p = new (std::nothrow) qcnn_plan(proto);
    if (!p) s = QCNN_ERR_HIP;
  }
  if (e != hipSuccess || s != QCNN_OK) {
    (void)hipStreamSynchronize(st);
    (void)hipFree(mem);
    return e != hipSuccess ? QCNN_ERR_HIP : s;
  }
  *plan = p;
  return QCNN_OK;
}

}  // namespace

extern "C" {

qcnn_status qcnn_conv_plan_create(int N, int C_s, int H, int W, const float* codebooks, int M, int K, int Csp,
                                  const uint8_t* codes, int packed, int C_t, int d_k, int stride, int pad,
                                  const float* bias, int relu, int pool_k, int pool_s, qcnn_plan** plan,
                                  void* stream) {
  if (!codebooks || !codes || !plan) return QCNN_ERR_NULL;
  if (K < 1 || K > 256) return QCNN_ERR_K_RANGE;
  if (pool_k < 0 || pool_s < 0 || (pool_k == 0) != (pool_s == 0)) return QCNN_ERR_SHAPE;
  const int bits = packed ? qcnn::code_bits(K) : 8;
  ConvCall c{};
  qcnn_status s = check_conv(N, C_s, H, W, M, K, Csp, codes, bits, C_t, d_k, stride, pad, pool_k, pool_s, &c);
  if (s != QCNN_OK) return s;
  hipStream_t st = (hipStream_t)stream;
  qcnn_plan proto{};
  proto.sh = c.sh;
  proto.relu = relu ? 1 : 0;
  proto.pooled = c.pooled;
  proto.pool = qcnn::PoolSpec{pool_k, pool_s, c.Hp, c.Wp};
  proto.kind = qcnn::conv_kernel_pick(c.sh);
  proto.relaid = proto.kind == 0;
  proto.bits = bits;
  proto.nx = c.nx;
  proto.ny = c.ny;
  const ConvShape sh = c.sh;
  return make_plan(
      proto, codebooks, c.nd, codes, c.nc, c.cb, proto.relaid ? qcnn::conv_flat_code_bytes(sh) : 0,
      [&](const qcnn::CodeStream& cs, uint8_t* out) { return qcnn::launch_conv_flat_codes(sh, cs, out, st); }, bias,
      plan, st);
}

qcnn_status qcnn_fc_plan_create(int N, int C_s, const float* codebooks, int M, int K, int Csp, const uint8_t* codes,
                                int packed, int C_t, const float* bias, int relu, qcnn_plan** plan, void* stream) {
  if (!codebooks || !codes || !plan) return QCNN_ERR_NULL;
  if (K < 1 || K > 256) return QCNN_ERR_K_RANGE;
  if (C_t < 1) return QCNN_ERR_SHAPE;
  qcnn_status s = check_pq(N, C_s, M, K, Csp);
  if (s != QCNN_OK) return s;
  const size_t nx = elems({N, C_s}), nd = elems({M, K, Csp}), nc = elems({C_t, M}), ny = elems({N, C_t});
  if (!nx || !nd || !nc || !ny) return QCNN_ERR_SHAPE;
  if ((uintptr_t)codes & 3) return QCNN_ERR_UNSUPPORTED;
  const int bits = packed ? qcnn::code_bits(K) : 8;
  hipStream_t st = (hipStream_t)stream;
  qcnn_plan proto{};
  proto.fc = true;
  proto.sh = ConvShape{N, C_s, 1, 1, M, K, Csp, C_t, 1, 1, 0, 1, 1};
  proto.relu = relu ? 1 : 0;
  proto.relaid = qcnn::fc_tiled_supported(N, C_s, M, K, Csp, C_t);
  proto.bits = bits;
  proto.nx = nx;
  proto.ny = ny;
  return make_plan(
      proto, codebooks, nd, codes, nc, code_stream_bytes(nc, bits),
      proto.relaid ? qcnn::fc_tiled_code_bytes(N, C_s, M, K, Csp, C_t) : 0,
      [&](const qcnn::CodeStream& cs, uint8_t* out) {
        return qcnn::launch_fc_tiled_codes(N, C_s, M, K, Csp, C_t, cs, reinterpret_cast<uint32_t*>(out), st);
      },
      bias, plan, st);
}

qcnn_status qcnn_plan_forward(const qcnn_plan* plan, const float* x, float* y, void* stream) {
  if (!plan || !x || !y) return QCNN_ERR_NULL;
  if (overlap(y, plan->ny * 4, x, plan->nx * 4)) return QCNN_ERR_ALIAS;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return QCNN_ERR_HIP;
  if (dev != plan->device) return QCNN_ERR_UNSUPPORTED;
  if (!prepare_device()) return QCNN_ERR_HIP;
  hipStream_t st = (hipStream_t)stream;
  const ConvShape& sh = plan->sh;
  const qcnn::CodeStream cs{plan->codes, plan->bits};
  if (plan->fc) {
    if (plan->relaid)
      return hip_status(qcnn::launch_fc_tiled_relaid(sh.N, sh.Cs, sh.M, sh.K, sh.Csp, sh.Ct, x, plan->D,
                                                     reinterpret_cast<const uint32_t*>(plan->codes), plan->bias,
                                                     plan->relu, y, st));
    return hip_status(
        qcnn::launch_fc_forward(sh.N, sh.Cs, sh.M, sh.K, sh.Csp, sh.Ct, x, plan->D, cs, plan->bias, plan->relu, y, st));
  }
  const qcnn::PoolSpec* pool = plan->pooled ? &plan->pool : nullptr;
  if (plan->relaid)
    return hip_status(qcnn::launch_conv_flat_relaid(sh, x, plan->D, plan->codes, plan->bias, plan->relu, y, st, pool));
  if (pool)
    return hip_status(
        qcnn::launch_conv_pool_forward(sh, x, plan->D, cs, plan->bias, plan->relu, *pool, y, st, plan->kind));
  return hip_status(qcnn::launch_conv_forward(sh, x, plan->D, cs, plan->bias, plan->relu, y, st, nullptr, plan->kind));
}

qcnn_status qcnn_plan_destroy(qcnn_plan* plan) {
  if (!plan) return QCNN_OK;
  int cur = 0;
  hipError_t e = hipGetDevice(&cur);
  if (e == hipSuccess && cur != plan->device) e = hipSetDevice(plan->device);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e == hipSuccess) e = hipFree(plan->mem);
  if (cur != plan->device) (void)hipSetDevice(cur);
  if (e != hipSuccess) return QCNN_ERR_HIP;
  delete plan;
  return QCNN_OK;
}

qcnn_status qcnn_fc_forward(const float* x, int N, int C_s, const float* codebooks, int M, int K, int Csp,
                            const uint8_t* codes, int C_t, const float* bias, int relu, float* y, void* stream) {
  return fc_forward(x, N, C_s, codebooks, M, K, Csp, codes, 8, C_t, bias, relu, y, stream);
}

qcnn_status qcnn_fc_forward_packed(const float* x, int N, int C_s, const float* codebooks, int M, int K, int Csp,
                                   const uint8_t* packed_codes, int C_t, const float* bias, int relu, float* y,
                                   void* stream) {
  if (K < 1 || K > 256) return QCNN_ERR_K_RANGE;
  return fc_forward(x, N, C_s, codebooks, M, K, Csp, packed_codes, qcnn::code_bits(K), C_t, bias, relu, y, stream);
}

qcnn_status qcnn_probe_lds(double* bytes_per_clk_cu, double* clock_ghz, double* bytes_per_s, void* stream) {
  if (!bytes_per_clk_cu || !clock_ghz || !bytes_per_s) return QCNN_ERR_NULL;
  return hip_status(qcnn::probe_lds((hipStream_t)stream, bytes_per_clk_cu, clock_ghz, bytes_per_s));
}

qcnn_status qcnn_probe_valu(double* add_clk, double* dpp_add_clk, double* mad_clk, void* stream) {
  if (!add_clk || !dpp_add_clk || !mad_clk) return QCNN_ERR_NULL;
  return hip_status(qcnn::probe_valu((hipStream_t)stream, add_clk, dpp_add_clk, mad_clk));
}

qcnn_status qcnn_probe_hbm(const void* src, void* dst, size_t bytes, double* read_bytes_per_s,
                           double* write_bytes_per_s, double* copy_bytes_per_s, void* stream) {
  if (!src || !dst || !read_bytes_per_s || !write_bytes_per_s || !copy_bytes_per_s) return QCNN_ERR_NULL;
  if (bytes < 16 || bytes > kMaxElems) return QCNN_ERR_SHAPE;
  if (((uintptr_t)src & 15) || ((uintptr_t)dst & 15)) return QCNN_ERR_UNSUPPORTED;
  if (overlap(dst, bytes, src, bytes)) return QCNN_ERR_ALIAS;
  return hip_status(
      qcnn::probe_hbm(src, dst, bytes, (hipStream_t)stream, read_bytes_per_s, write_bytes_per_s, copy_bytes_per_s));
}

int qcnn_code_bits(int K) {
  if (K < 1 || K > 256) return -1;
  return qcnn::code_bits(K);
}

size_t qcnn_packed_bytes(size_t n, int K) {
  if (K < 1 || K > 256 || n > kMaxElems) return 0;
  return (n * (size_t)qcnn::code_bits(K) + 31) / 32 * 4;
}

qcnn_status qcnn_pack_codes(const uint8_t* codes, size_t n, int K, uint8_t* packed, void* stream) {
  if (K < 1 || K > 256) return QCNN_ERR_K_RANGE;
  if (n > kMaxElems) return QCNN_ERR_SHAPE;
  const int bits = qcnn::code_bits(K);
  const size_t pb = (n * (size_t)bits + 31) / 32 * 4;
  if ((n > 0 && !codes) || (pb > 0 && !packed)) return QCNN_ERR_NULL;
  if (pb == 0) return QCNN_OK;
  if (((uintptr_t)packed & 3) || ((uintptr_t)codes & 3)) return QCNN_ERR_UNSUPPORTED;
  if (overlap(packed, pb, codes, n)) return QCNN_ERR_ALIAS;
  hipStream_t st = (hipStream_t)stream;
  if (!prepare_device()) return QCNN_ERR_HIP;
  qcnn_status s = check_codes(qcnn::CodeStream{codes, 8}, n, K, st);
  if (s != QCNN_OK) return s;
  return hip_status(qcnn::launch_pack_codes(codes, n, bits, reinterpret_cast<uint32_t*>(packed), st));
}

qcnn_status qcnn_unpack_codes(const uint8_t* packed, size_t n, int K, uint8_t* codes, void* stream) {
  if (K < 1 || K > 256) return QCNN_ERR_K_RANGE;
  if (n > kMaxElems) return QCNN_ERR_SHAPE;
  const int bits = qcnn::code_bits(K);
  const size_t pb = (n * (size_t)bits + 31) / 32 * 4;
  if ((n > 0 && !codes) || (pb > 0 && !packed)) return QCNN_ERR_NULL;
  if (n == 0) return QCNN_OK;
  if (pb > 0 && ((uintptr_t)packed & 3)) return QCNN_ERR_UNSUPPORTED;
  if (overlap(codes, n, packed, pb)) return QCNN_ERR_ALIAS;
  if (!prepare_device()) return QCNN_ERR_HIP;
  return hip_status(qcnn::launch_unpack_codes(qcnn::CodeStream{packed, bits}, n, codes, (hipStream_t)stream));
}

// Shared validation of the quantizer entry points (host only).
static qcnn_status check_quant(const float* W, int C_t, int C_s, int d_k, int M, int K, int Csp, size_t* nw,
                               size_t* nd, size_t* nc) {
  if (!W) return QCNN_ERR_NULL;
  if (C_t < 1 || d_k < 1) return QCNN_ERR_SHAPE;
  qcnn_status s = check_pq(1, C_s, M, K, Csp);
  if (s != QCNN_OK) return s;
  *nw = elems({C_t, C_s, d_k, d_k});
  *nd = elems({M, K, Csp});
  *nc = elems({C_t, d_k, d_k, M});
  if (!*nw || !*nd || !*nc) return QCNN_ERR_SHAPE;
  if ((long long)C_t * d_k * d_k > (1LL << 30)) return QCNN_ERR_UNSUPPORTED;
  return QCNN_OK;
}

qcnn_status qcnn_pq_assign(const float* W, int C_t, int C_s, int d_k, const float* codebooks, int M, int K, int Csp,
                           uint8_t* codes, double* objective, void* stream) {
  size_t nw, nd, nc;
  qcnn_status s = check_quant(W, C_t, C_s, d_k, M, K, Csp, &nw, &nd, &nc);
  if (s != QCNN_OK) return s;
  if (!codebooks || !codes) return QCNN_ERR_NULL;
  if (overlap(codes, nc, W, nw * 4) || overlap(codes, nc, codebooks, nd * 4) ||
      overlap(objective, (size_t)M * 8, W, nw * 4) || overlap(objective, (size_t)M * 8, codebooks, nd * 4) ||
      overlap(objective, (size_t)M * 8, codes, nc))
    return QCNN_ERR_ALIAS;
  if (!prepare_device()) return QCNN_ERR_HIP;
  return hip_status(qcnn::launch_pq_assign(C_t, C_s, d_k, W, codebooks, M, K, Csp, codes, objective,
                                           (hipStream_t)stream));
}

qcnn_status qcnn_pq_update(const float* W, int C_t, int C_s, int d_k, const uint8_t* codes, int M, int K, int Csp,
                           float* codebooks, int* counts, void* stream) {
  size_t nw, nd, nc;
  qcnn_status s = check_quant(W, C_t, C_s, d_k, M, K, Csp, &nw, &nd, &nc);
  if (s != QCNN_OK) return s;
  if (!codebooks || !codes) return QCNN_ERR_NULL;
  if (overlap(codebooks, nd * 4, W, nw * 4) || overlap(codebooks, nd * 4, codes, nc) ||
      overlap(counts, nd / Csp * 4, W, nw * 4) || overlap(counts, nd / Csp * 4, codes, nc) ||
      overlap(counts, nd / Csp * 4, codebooks, nd * 4))
    return QCNN_ERR_ALIAS;
  hipStream_t st = (hipStream_t)stream;
  if (!prepare_device()) return QCNN_ERR_HIP;
  s = check_codes(qcnn::CodeStream{codes, 8}, nc, K, st);
  if (s != QCNN_OK) return s;
  return hip_status(qcnn::launch_pq_update(C_t, C_s, d_k, W, codes, M, K, Csp, codebooks, counts, st));
}

qcnn_status qcnn_pq_kmeans(const float* W, int C_t, int C_s, int d_k, int M, int K, int Csp, int iters,
                           float* codebooks, uint8_t* codes, double* objective, void* stream) {
  size_t nw, nd, nc;
  qcnn_status s = check_quant(W, C_t, C_s, d_k, M, K, Csp, &nw, &nd, &nc);
  if (s != QCNN_OK) return s;
  if (!codebooks || !codes) return QCNN_ERR_NULL;
  if (iters < 0) return QCNN_ERR_SHAPE;
  const size_t no = ((size_t)iters + 1) * 8;
  if (overlap(codebooks, nd * 4, W, nw * 4) || overlap(codebooks, nd * 4, codes, nc) || overlap(codes, nc, W, nw * 4) ||
      overlap(objective, no, W, nw * 4) || overlap(objective, no, codebooks, nd * 4) || overlap(objective, no, codes, nc))
    return QCNN_ERR_ALIAS;
  if (!prepare_device()) return QCNN_ERR_HIP;
  return hip_status(qcnn::launch_pq_kmeans(C_t, C_s, d_k, W, M, K, Csp, iters, codebooks, codes, objective,
                                           (hipStream_t)stream));
}

qcnn_status qcnn_ec_fc(const float* S, int N, int C_s, const float* T, int C_t, float* codebooks, int M, int K,
                       int Csp, uint8_t* codes, int sweeps, int inner, double* objective, void* stream) {
  if (!S || !T || !codebooks || !codes) return QCNN_ERR_NULL;
  if (C_t < 1 || sweeps < 0 || inner < 1) return QCNN_ERR_SHAPE;
  qcnn_status s = check_pq(N, C_s, M, K, Csp);
  if (s != QCNN_OK) return s;
  const size_t ns = elems({N, C_s}), nt = elems({N, C_t}), nd = elems({M, K, Csp}), nc = elems({C_t, M});
  if (!ns || !nt || !nd || !nc || (long long)sweeps * M > (1LL << 30)) return QCNN_ERR_SHAPE;
  if (N > (1 << 20) || C_t > 65536 || nt > ((size_t)1 << 32)) return QCNN_ERR_UNSUPPORTED;
  const size_t no = ((size_t)sweeps * M + 1) * 8;
  if (overlap(codebooks, nd * 4, S, ns * 4) || overlap(codebooks, nd * 4, T, nt * 4) ||
      overlap(codes, nc, S, ns * 4) || overlap(codes, nc, T, nt * 4) || overlap(codes, nc, codebooks, nd * 4) ||
      overlap(objective, no, S, ns * 4) || overlap(objective, no, T, nt * 4) ||
      overlap(objective, no, codebooks, nd * 4) || overlap(objective, no, codes, nc))
    return QCNN_ERR_ALIAS;
  hipStream_t st = (hipStream_t)stream;
  if (!prepare_device()) return QCNN_ERR_HIP;
  if (((uintptr_t)codes & 3) == 0) {
    s = check_codes(qcnn::CodeStream{codes, 8}, nc, K, st);
    if (s != QCNN_OK) return s;
  }
  return hip_status(qcnn::launch_ec_fc(N, C_s, C_t, M, K, Csp, S, T, codebooks, codes, sweeps, inner, objective, st));
}

qcnn_status qcnn_ec_conv(const float* S, int N, int C_s, int H, int W, const float* T, int C_t, int d_k,
                         int stride, int pad, float* codebooks, int M, int K, int Csp, uint8_t* codes, int sweeps,
                         int inner, double* objective, void* stream) {
  if (!S || !T || !codebooks || !codes) return QCNN_ERR_NULL;
  if (H < 1 || W < 1 || C_t < 1 || d_k < 1 || stride < 1 || pad < 0 || sweeps < 0 || inner < 1)
    return QCNN_ERR_SHAPE;
  qcnn_status s = check_pq(N, C_s, M, K, Csp);
  if (s != QCNN_OK) return s;
  const int Ho = qcnn_out_size(H, d_k, stride, pad), Wo = qcnn_out_size(W, d_k, stride, pad);
  if (Ho < 1 || Wo < 1) return QCNN_ERR_SHAPE;
  const size_t ns = elems({N, C_s, H, W}), nt = elems({N, C_t, Ho, Wo}), nd = elems({M, K, Csp});
  const size_t nc = elems({C_t, d_k, d_k, M});
  if (!ns || !nt || !nd || !nc || (long long)sweeps * M > (1LL << 30)) return QCNN_ERR_SHAPE;
  if (Csp > 8 || (long long)C_t * d_k * d_k > 16384 || nt > ((size_t)1 << 31) ||
      (size_t)M * d_k * d_k * d_k * d_k * Csp * Csp > ((size_t)1 << 31))
    return QCNN_ERR_UNSUPPORTED;
  const size_t no = ((size_t)sweeps * M + 1) * 8;
  if (overlap(codebooks, nd * 4, S, ns * 4) || overlap(codebooks, nd * 4, T, nt * 4) ||
      overlap(codes, nc, S, ns * 4) || overlap(codes, nc, T, nt * 4) || overlap(codes, nc, codebooks, nd * 4) ||
      overlap(objective, no, S, ns * 4) || overlap(objective, no, T, nt * 4) ||
      overlap(objective, no, codebooks, nd * 4) || overlap(objective, no, codes, nc))
    return QCNN_ERR_ALIAS;
  hipStream_t st = (hipStream_t)stream;
  if (!prepare_device()) return QCNN_ERR_HIP;
  if (((uintptr_t)codes & 3) == 0) {
    s = check_codes(qcnn::CodeStream{codes, 8}, nc, K, st);
    if (s != QCNN_OK) return s;
  }
  return hip_status(qcnn::launch_ec_conv(N, C_s, H, W, C_t, d_k, stride, pad, M, K, Csp, S, T, codebooks, codes,
                                         sweeps, inner, objective, st));
}

qcnn_status qcnn_maxpool2d(const float* x, int N, int C, int H, int W, int k, int s, float* y, void* stream) {
  if (!x || !y) return QCNN_ERR_NULL;
  if (N < 1 || C < 1 || H < 1 || W < 1 || k < 1 || s < 1) return QCNN_ERR_SHAPE;
  const int Ho = qcnn_out_size(H, k, s, 0), Wo = qcnn_out_size(W, k, s, 0);
  if (Ho < 1 || Wo < 1) return QCNN_ERR_SHAPE;
  const size_t nx = elems({N, C, H, W}), ny = elems({N, C, Ho, Wo});
  if (!nx || !ny) return QCNN_ERR_SHAPE;
  if (overlap(y, ny * 4, x, nx * 4)) return QCNN_ERR_ALIAS;
  return hip_status(qcnn::launch_maxpool(x, N, C, H, W, k, s, Ho, Wo, y, (hipStream_t)stream));
}

}  // extern "C"
