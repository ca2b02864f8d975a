// Device generator of synthetic tq matrices for benchmark and test workloads (the
// 43-layer stack holds ~246 GB of codes, far too much to draw on the host): trits and
// f16 scales from SplitMix64 used as a counter-based generator (Steele, Lea & Flood,
// OOPSLA 2014), then the fold c = 3*t1 + t2 (Sec. 2.1) and the pack of tq.h, fused, so
// the codes are written once. The recipe is stated in tq.h (tq_synth_weights).
#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

__device__ __forceinline__ uint64_t splitmix64(uint64_t key, uint64_t i) {
  uint64_t z = key + (i + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Nibble c & 15 of one element from its word: t1 from field (0 or 2), t2 from the next
// field; a 16-bit field f maps to the trit ((f * 3) >> 16) - 1.
__device__ __forceinline__ uint32_t nibble_of(uint64_t word, int odd) {
  const uint32_t half = (uint32_t)(word >> (odd ? 32 : 0));
  const int a = (int)(((half & 0xFFFFu) * 3u) >> 16) - 1;
  const int b = (int)(((half >> 16) * 3u) >> 16) - 1;
  return (uint32_t)(3 * a + b) & 0xFu;
}

// One thread per 16-byte chunk (32 weights), grid-stride over all chunks.
__global__ __launch_bounds__(256) void k_synth(uint64_t key, int64_t n, int64_t k, uint8_t* __restrict__ codes,
                                               uint16_t* __restrict__ scales) {
  const int64_t kb = k / 256, nchunks = n * kb * 8;
  const uint64_t scale_base = (uint64_t)(n * k / 2);
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < nchunks;
       c += (int64_t)gridDim.x * blockDim.x) {
    const int64_t blk = c >> 3;  // r * kb + b
    const int j = (int)(c & 7);
    const int64_t r = blk / kb, b = blk - r * kb;
    const uint64_t e0 = (uint64_t)(r * k + b * 256 + 32 * j);  // even
    uint32_t out[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      uint32_t v = 0;
#pragma unroll
      for (int h = 0; h < 2; ++h) {  // bytes 4m + 2h, 4m + 2h + 1 share one word per half
        const uint64_t wlo = splitmix64(key, (e0 >> 1) + 2 * m + h);
        const uint64_t whi = splitmix64(key, (e0 >> 1) + 8 + 2 * m + h);
        const uint32_t b0 = nibble_of(wlo, 0) | (nibble_of(whi, 0) << 4);
        const uint32_t b1 = nibble_of(wlo, 1) | (nibble_of(whi, 1) << 4);
        v |= (b0 | (b1 << 8)) << (16 * h);
      }
      out[m] = v;
    }
    *reinterpret_cast<uint4*>(codes + c * 16) = make_uint4(out[0], out[1], out[2], out[3]);
    if (j == 0) {
      const uint64_t wv = splitmix64(key, scale_base + (uint64_t)blk);
      scales[blk] = (uint16_t)(0x1419u + (uint32_t)(((wv >> 32) * 0x1A4Eull) >> 32));
    }
  }
}

}  // namespace tq

extern "C" tq_status tq_synth_weights(uint64_t key, int32_t n, int32_t k, uint8_t* codes, uint16_t* scales,
                                      void* stream) {
  using namespace tq;
  clear_error();
  if (n < 1 || k <= 0 || k % 256 != 0)
    return fail(TQ_ERR_INVALID, "tq_synth_weights: bad shape n=%d k=%d (k must be a multiple of 256)", n, k);
  if (!codes || !scales) return fail(TQ_ERR_INVALID, "tq_synth_weights: null pointer");
  if (!aligned(codes, 128) || !aligned(scales, 2)) return fail(TQ_ERR_ALIGN, "tq_synth_weights: codes must be 128-byte aligned");
  const int64_t nchunks = (int64_t)n * (k / 256) * 8;
  const int64_t wgs = std::min<int64_t>((nchunks + 255) / 256, 256 * 64);
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_synth, dim3((unsigned)wgs), dim3(256), 0, (hipStream_t)stream, key, (int64_t)n, (int64_t)k,
                     codes, scales);
  return check_launch("tq_synth_weights");
}
