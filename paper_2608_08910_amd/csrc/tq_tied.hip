// Tied quantizer (Sec. 2.1): fp32 weights -> the persistent folded code plane and its f16
// scales, by alternating code and scale steps against one scale per 256-weight block
// (the tied fit W_hat = s * c, c in -4..4). The start, the stopping rule and the
// precision of each step are this library's reading, stated in tq.h; every integer
// decision is taken in a fixed precision and order, so the result is reproducible bit
// for bit.
#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

// A wave owns one block; lane l holds weights l, l + 64, l + 128, l + 192 of it, so the
// pairwise-halving sum adds within the lane for the first two levels (h = 128, 64) and
// across lanes (xor 32 .. 1) for the rest.

// The code step: c = clamp(rne(fl32(w / s)), -4, 4). The quotient is formed as
// w * fl32(1 / s), which lies within |q| * 2^-22 of both w / s and fl32(w / s); rne only
// changes value at half-integers, so unless one lies that close the product rounds like
// the correctly rounded quotient. The few elements that near a half-integer (exact ties
// among them) take the division.
__device__ __forceinline__ void tied_code_step(const float (&w)[4], float s, int (&c)[4]) {
  const float rs = 1.0f / s;
  float r[4];
  bool near = false;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float q = w[j] * rs;
    const float f = q - floorf(q);  // exact: the distance above the integer below
    near |= fabsf(f - 0.5f) <= fabsf(q) * 0x1p-21f;
    r[j] = rintf(q);
  }
  if (__any(near)) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float q = w[j] * rs;
      const float f = q - floorf(q);
      if (fabsf(f - 0.5f) <= fabsf(q) * 0x1p-21f) r[j] = rintf(w[j] / s);  // correctly rounded division
    }
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) c[j] = (int)fminf(fmaxf(r[j], -4.0f), 4.0f);
}

// a + (the same lane-pair partner's a), for a butterfly over lane bit M (both lanes of a
// pair add the same two values, so they hold the same sum)
template <int M>
__device__ __forceinline__ double xor_add(double a) {
  const int lo = __double2loint(a), hi = __double2hiint(a);
  return a + __hiloint2double(lane_xor_i<M>(hi), lane_xor_i<M>(lo));
}
template <int M>
__device__ __forceinline__ int xor_add(int a) {
  return a + lane_xor_i<M>(a);
}

__global__ __launch_bounds__(256) void k_tied_quantize(const float* __restrict__ w, int64_t nblocks, int max_iter,
                                                       uint8_t* __restrict__ codes, uint16_t* __restrict__ scales,
                                                       uint8_t* __restrict__ iters) {
  __shared__ uint8_t s_bytes[4][128];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t blk = (int64_t)blockIdx.x * 4 + wv;
  if (blk >= nblocks) return;  // uniform across the wave
  const float* wb = w + blk * 256;
  float v[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) v[j] = wb[lane + 64 * j];
  float amax = fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3])));
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) amax = fmaxf(amax, __shfl_xor(amax, m));
  int c[4] = {0, 0, 0, 0};
  uint16_t h16 = 0;
  int it = 0;
  if (amax >= 0x1p-100f) {
    float s = amax / 4.0f;
    int prev[4] = {0, 0, 0, 0};
    for (;;) {
      tied_code_step(v, s, c);
      ++it;
      const bool same = it > 1 && __all(c[0] == prev[0] && c[1] == prev[1] && c[2] == prev[2] && c[3] == prev[3]);
      if (same || it == max_iter) break;
      // <w, c> in fp64 (exact products), pairwise halving: v[i] += v[i + h], h = 128 .. 1
      double p0 = (double)v[0] * (double)c[0], p1 = (double)v[1] * (double)c[1];
      const double p2 = (double)v[2] * (double)c[2], p3 = (double)v[3] * (double)c[3];
      p0 = p0 + p2;  // h = 128
      p1 = p1 + p3;
      p0 = p0 + p1;  // h = 64
      p0 = xor_add<32>(p0);  // h = 32 .. 1
      p0 = xor_add<16>(p0);
      p0 = xor_add<8>(p0);
      p0 = xor_add<4>(p0);
      p0 = xor_add<2>(p0);
      p0 = xor_add<1>(p0);
      int cc = c[0] * c[0] + c[1] * c[1] + c[2] * c[2] + c[3] * c[3];
      cc = xor_add<32>(cc);
      cc = xor_add<16>(cc);
      cc = xor_add<8>(cc);
      cc = xor_add<4>(cc);
      cc = xor_add<2>(cc);
      cc = xor_add<1>(cc);
#pragma unroll
      for (int j = 0; j < 4; ++j) prev[j] = c[j];
      if (cc == 0) break;
      s = (float)(p0 / (double)cc);
    }
    // f16, nearest even, saturating at the largest finite value
    const _Float16 hs = s >= 65520.0f ? (_Float16)65504.0f : (_Float16)s;
    h16 = __builtin_bit_cast(uint16_t, hs);
    const float sd = (float)hs;
    if (sd == 0.0f) {
#pragma unroll
      for (int j = 0; j < 4; ++j) c[j] = 0;
    } else {
      tied_code_step(v, sd, c);
    }
  }
  // pack: element e = lane + 64j; byte 16(e/32) + e%32 (e%32 < 16) holds e in its low
  // nibble and e + 16 (lane + 16) in its high nibble
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int hi = __shfl_xor(c[j], 16);
    if ((lane & 31) < 16) s_bytes[wv][16 * (lane >> 5) + 32 * j + (lane & 31)] = (uint8_t)((c[j] & 15) | ((hi & 15) << 4));
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  if (lane < 8)
    reinterpret_cast<uint4*>(codes + blk * 128)[lane] = reinterpret_cast<const uint4*>(s_bytes[wv])[lane];
  if (lane == 0) {
    scales[blk] = h16;
    if (iters) iters[blk] = (uint8_t)it;
  }
}

}  // namespace tq

extern "C" tq_status tq_tied_quantize(const float* w, int32_t n, int32_t k, int32_t max_iter, uint8_t* codes,
                                      uint16_t* scales, uint8_t* iters, void* stream) {
  using namespace tq;
  clear_error();
  if (n < 0 || k <= 0 || k % 256 != 0)
    return fail(TQ_ERR_INVALID, "tq_tied_quantize: n = %d, k = %d (need n >= 0, k a positive multiple of 256)", n, k);
  if (max_iter < 1 || max_iter > 255)
    return fail(TQ_ERR_INVALID, "tq_tied_quantize: max_iter = %d outside [1, 255]", max_iter);
  if (n == 0) return TQ_OK;
  if (!w || !codes || !scales) return fail(TQ_ERR_INVALID, "tq_tied_quantize: null pointer");
  if (!aligned(w, 4) || !aligned(codes, 128) || !aligned(scales, 2))
    return fail(TQ_ERR_ALIGN, "tq_tied_quantize: w must be 4-byte, codes 128-byte and scales 2-byte aligned");
  const int64_t nblocks = (int64_t)n * (k / 256);
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_tied_quantize, dim3((unsigned)((nblocks + 3) / 4)), dim3(256), 0, (hipStream_t)stream, w,
                     nblocks, (int)max_iter, codes, scales, iters);
  return check_launch("tq_tied_quantize");
}
