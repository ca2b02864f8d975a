// Per-256 activation quantizer (Sec. 2.2: the codes meet int8 activations that carry one
// scale per block; the block/scale/rounding rule is this library's reading, stated in tq.h).
#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

// One wave quantizes 8 consecutive blocks of the flattened [t][kb] block grid; each
// 8-lane group owns one block and each lane 32 contiguous values (128 bytes).
__global__ __launch_bounds__(256) void k_quantize(const float* __restrict__ x, int64_t nblocks,
                                                  int8_t* __restrict__ q, float* __restrict__ d,
                                                  int32_t* __restrict__ bsum) {
  const int lane = threadIdx.x & 63;
  const int64_t blk = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * 8 + (lane >> 3);
  if (blk >= nblocks) return;  // uniform across the block's 8-lane group
  const int cp = lane & 7;
  const float4* xp = reinterpret_cast<const float4*>(x + blk * 256 + cp * 32);
  float v[32];
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    const float4 f = xp[m];
    v[4 * m + 0] = f.x;
    v[4 * m + 1] = f.y;
    v[4 * m + 2] = f.z;
    v[4 * m + 3] = f.w;
  }
  int qw[8], qs, bs;
  float dd;
  quantize_group32(v, qw, qs, dd, bs);
  int4* qp = reinterpret_cast<int4*>(q + blk * 256 + cp * 32);
  qp[0] = make_int4(qw[0], qw[1], qw[2], qw[3]);
  qp[1] = make_int4(qw[4], qw[5], qw[6], qw[7]);
  if (cp == 0) {
    d[blk] = dd;
    bsum[blk] = bs;
  }
}

hipError_t launch_quantize(const float* x, int64_t t, int32_t k, int8_t* q, float* d, int32_t* bsum,
                           hipStream_t st) {
  const int64_t nblocks = t * (k / 256);
  if (nblocks == 0) return hipSuccess;
  const int64_t wgs = (nblocks + 31) / 32;
  hipLaunchKernelGGL(k_quantize, dim3((unsigned)wgs), dim3(256), 0, st, x, nblocks, q, d, bsum);
  return hipSuccess;
}

}  // namespace tq

extern "C" tq_status tq_quantize_act(const float* x, int64_t t, int32_t k, int8_t* q, float* d,
                                     int32_t* bsum, void* stream) {
  using namespace tq;
  clear_error();
  if (t < 0) return fail(TQ_ERR_INVALID, "tq_quantize_act: t = %lld < 0", (long long)t);
  if (k <= 0 || k % 256 != 0 || k > kMaxK)
    return fail(TQ_ERR_INVALID, "tq_quantize_act: k = %d must be a positive multiple of 256 <= %d", k, kMaxK);
  if (t == 0) return TQ_OK;
  if (!x || !q || !d || !bsum) return fail(TQ_ERR_INVALID, "tq_quantize_act: null pointer");
  if (!aligned(x, 16) || !aligned(q, 16) || !aligned(d, 4) || !aligned(bsum, 4))
    return fail(TQ_ERR_ALIGN, "tq_quantize_act: x and q must be 16-byte aligned, d and bsum 4-byte aligned");
  if (t * (int64_t)(k / 256) > (int64_t)INT32_MAX * 32)
    return fail(TQ_ERR_INVALID, "tq_quantize_act: t too large");
  (void)hipGetLastError();
  launch_quantize(x, t, k, q, d, bsum, (hipStream_t)stream);
  return check_launch("tq_quantize_act");
}
