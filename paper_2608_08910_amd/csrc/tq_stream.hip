// The benchmark's second ceiling: a plain streaming read of a given byte count, shaped
// like the dot-pass kernels' weight stream (nontemporal 16-byte loads, every byte read
// once, a single round of loads per thread) but with no arithmetic beyond an XOR of what
// was read. The dot pass's rate is reported as a fraction of this kernel's measured rate
// on the same number of bytes, beside the fraction of the 8 TB/s peak.
#include <hip/hip_ext.h>

#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

constexpr int kReadThreads = 256;
constexpr int kReadPerThread = 8;  // 16-byte loads per thread, all issued before any use

__global__ __launch_bounds__(kReadThreads) void k_stream_read(const uint8_t* __restrict__ src, uint64_t n16,
                                                             uint32_t* __restrict__ sink) {
  const uint64_t base = (uint64_t)blockIdx.x * (kReadThreads * kReadPerThread) + threadIdx.x;
  uint4 v[kReadPerThread];
#pragma unroll
  for (int j = 0; j < kReadPerThread; ++j) {
    const uint64_t i = min(base + (uint64_t)j * kReadThreads, n16 - 1);  // the tail rereads the last chunk
    v[j] = ldg16(src + i * 16);
  }
  uint32_t acc = 0;
#pragma unroll
  for (int j = 0; j < kReadPerThread; ++j) acc ^= v[j].x ^ v[j].y ^ v[j].z ^ v[j].w;
  // a store that depends on every load (so that none is dropped) but practically never
  // happens: the kernel's traffic is its reads
  if (acc == 0x9E3779B9u) sink[0] = acc;
}

}  // namespace tq

extern "C" tq_status tq_stream_read_timed(const void* src, size_t bytes, uint32_t* sink, void* stream,
                                          void* const* events) {
  using namespace tq;
  clear_error();
  if (!src || !sink || bytes < 16 || bytes % 16 != 0)
    return fail(TQ_ERR_INVALID, "tq_stream_read_timed: null pointer, or bytes = %zu not a positive multiple of 16",
                bytes);
  if (!aligned(src, 16) || !aligned(sink, 4)) return fail(TQ_ERR_ALIGN, "tq_stream_read_timed: src 16-byte aligned");
  if (!events || !events[0] || !events[1]) return fail(TQ_ERR_INVALID, "tq_stream_read_timed: null event");
  const uint64_t n16 = bytes / 16;
  const uint64_t per_wg = (uint64_t)kReadThreads * kReadPerThread;
  const uint64_t wgs = (n16 + per_wg - 1) / per_wg;
  if (wgs > 0x7fffffffu) return fail(TQ_ERR_INVALID, "tq_stream_read_timed: too many bytes");
  (void)hipGetLastError();
  hipExtLaunchKernelGGL(k_stream_read, dim3((unsigned)wgs), dim3(kReadThreads), 0, (hipStream_t)stream,
                        (hipEvent_t)events[0], (hipEvent_t)events[1], 0, static_cast<const uint8_t*>(src), n16, sink);
  return check_launch("tq_stream_read_timed");
}
