// polyq_gemv_batch_noalloc: the decode launch of polyq_gemv_batch with its
// workspace in a fixed device array of this library instead of caller memory,
// for callers that cannot allocate (code under graph capture, tight serving
// loops, harnesses that forbid hipMalloc).  Same kernels, same plan, same
// results.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.h"

namespace polyq {
namespace {

// The workspace every call on a device shares.  Its device address comes from
// hipGetSymbolAddress, taken once per device with that device current: in host
// code the name `scratch` is only a host-side stand-in for the symbol.
constexpr size_t kScratchBytes = POLYQ_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};
// Leading bytes of each device's array known to be zero (the calls' split-K
// state is left zero; activation copies placed after it are not).
size_t g_clean[kMaxDevices] = {};

// Zero-fills n 16-byte words (the workspace contract: the split-K state is
// zero before a call and every completed call leaves it zero).  A kernel, not a memset, so that a
// first call made under graph capture records a kernel node.
__global__ __launch_bounds__(256) void clear_kernel(uint4* __restrict__ p, int64_t n) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    p[i] = uint4{0u, 0u, 0u, 0u};
}

// Device address of `scratch` on the current device (taken on the first call
// there), with its first `zero` bytes cleared on `stream` where they may not be
// zero; `dirty`: the call leaves bytes past `zero` non-zero.  Holds the lock
// only on the host (the clear is enqueued, not waited for).
polyq_status scratch_for_current_device(hipStream_t stream, size_t zero, bool dirty, void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return POLYQ_ERR_DEVICE;
  if (dev >= kMaxDevices) return POLYQ_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_scratch[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr)
      return POLYQ_ERR_DEVICE;
    g_scratch[dev] = ptr;
    g_clean[dev] = 0;
  }
  if (zero > g_clean[dev]) {
    // clear [clean, zero) rounded out to 16-byte words
    const size_t lo = g_clean[dev] / 16, hi = (zero + 15) / 16;
    hipLaunchKernelGGL(clear_kernel, dim3(1024), dim3(256), 0, stream,
                       static_cast<uint4*>(g_scratch[dev]) + lo, static_cast<int64_t>(hi - lo));
    if (hipGetLastError() != hipSuccess) return POLYQ_ERR_DEVICE;
    g_clean[dev] = hi * 16;
  }
  // after the call: [0, zero) is zero again; an activation copy after it is not
  if (dirty) g_clean[dev] = zero;
  *out = g_scratch[dev];
  return POLYQ_OK;
}

}  // namespace
}  // namespace polyq

extern "C" polyq_status polyq_gemv_batch_noalloc(const polyq_gemv_item* items, int32_t count,
                                                 int32_t m, void* stream) {
  using namespace polyq;
  // the request is validated and sized before anything is set up or launched
  size_t need = 0, zero = 0;
  const polyq_status st = gemv_batch_workspace_status(items, count, m, &need, &zero);
  if (st != POLYQ_OK) return st;
  if (need > kScratchBytes) return POLYQ_ERR_CAPACITY;
  void* ws = nullptr;
  const polyq_status sst =
      scratch_for_current_device(static_cast<hipStream_t>(stream), zero, need > zero, &ws);
  if (sst != POLYQ_OK) return sst;
  return polyq_gemv_batch(items, count, m, ws, kScratchBytes, stream);
}
