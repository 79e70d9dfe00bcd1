// Streaming-read probe: reads a device buffer once and keeps nothing, the
// reference rate the decode GEMV's weight stream is compared against (the
// highest read rate a launch of that size reaches on this GPU).  Not part of
// the product computation.
#include <hip/hip_runtime.h>

#include "internal.h"

namespace polyq {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeDepth = 4;  // 16-byte loads per thread in flight
constexpr int64_t kProbeStep = static_cast<int64_t>(kProbeThreads) * 16;  // bytes per load of a work-group

typedef uint32_t u4v __attribute__((ext_vector_type(4)));

// Work-group w reads its contiguous share [w * per, min((w + 1) * per, bytes))
// through a buffer resource bounded at the share (reads past it return 0),
// kProbeDepth loads of 4 KB per work-group in flight.  The xor of everything
// read is stored only if it equals a value it almost never takes, so the loads
// cannot be dropped and nothing is written in practice.
__global__ __launch_bounds__(kProbeThreads) void read_probe_kernel(const uint8_t* __restrict__ buf,
                                                                   int64_t bytes, int64_t per,
                                                                   uint32_t* __restrict__ sink) {
  const int64_t lo = per * blockIdx.x;
  if (lo >= bytes) return;
  const int64_t len = min(bytes - lo, per);
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(buf + lo), static_cast<short>(0), static_cast<int>(len), 0x00020000);
  const int voff = threadIdx.x * 16;
  u4v acc = {0u, 0u, 0u, 0u};
  for (int64_t base = 0; base < len; base += kProbeDepth * kProbeStep) {
    u4v v[kProbeDepth];
#pragma unroll
    for (int j = 0; j < kProbeDepth; ++j)
      v[j] = __builtin_bit_cast(u4v, __builtin_amdgcn_raw_buffer_load_b128(
                                         r, voff, static_cast<int>(base + j * kProbeStep), 0));
#pragma unroll
    for (int j = 0; j < kProbeDepth; ++j) acc ^= v[j];
  }
  const uint32_t h = acc.x ^ acc.y ^ acc.z ^ acc.w;
  if (h == 0x9E3779B9u) sink[blockIdx.x] = h;
}

}  // namespace
}  // namespace polyq

extern "C" polyq_status polyq_read_probe(const void* buf, int64_t bytes, int32_t work_groups,
                                         uint32_t* sink, void* stream) {
  using namespace polyq;
  if (buf == nullptr || sink == nullptr || bytes < 16 || bytes % 16 != 0 || work_groups < 1)
    return POLYQ_ERR_ARG;
  if (reinterpret_cast<uintptr_t>(buf) % 16 != 0) return POLYQ_ERR_ARG;
  // share per work-group: a multiple of one load round of the work-group, and
  // below 2^30 bytes (every offset the loop forms stays inside an int)
  const int64_t per = ((bytes + work_groups - 1) / work_groups + kProbeStep - 1) / kProbeStep * kProbeStep;
  if (per >= (static_cast<int64_t>(1) << 30)) return POLYQ_ERR_CAPACITY;
  const int64_t grid = (bytes + per - 1) / per;
  hipLaunchKernelGGL(read_probe_kernel, dim3(static_cast<unsigned>(grid)), dim3(kProbeThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const uint8_t*>(buf), bytes, per,
                     sink);
  return hipGetLastError() == hipSuccess ? POLYQ_OK : POLYQ_ERR_DEVICE;
}
