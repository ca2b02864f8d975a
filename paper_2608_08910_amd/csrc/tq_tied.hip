// Tied quantizer (Sec. 2.1): fp32 weights -> the persistent folded code plane and its f16
// scales, by alternating code and scale steps against one scale per 256-weight block
// (the tied fit W_hat = s * c, c in -4..4). The start, the stopping rule and the
// precision of each step are this library's reading, stated in tq.h; every integer
// decision is taken in a fixed precision and order, so the result is reproducible bit
// for bit.
#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

// A 16-lane group of a wave owns one block (a wave four): lane u of the group holds
// weights u + 16j, j = 0..15, so the pairwise-halving sum runs within the lane for
// h = 128 .. 16 (j with j + 8, j + 4, j + 2, j + 1) and across the group's lanes for
// h = 8 .. 1 (u with u ^ 8, ^ 4, ^ 2, ^ 1).
constexpr int kTiedE = 16;  // weights per lane

// The code step: c = clamp(rne(fl32(w / s)), -4, 4). The quotient is formed as
// w * fl32(1 / s), within |q| * 2^-22 of both w / s and fl32(w / s); rne only changes
// value at half-integers, so unless one lies that close the product rounds like the
// correctly rounded quotient. Past |q| = 8 the clamp decides alone, so a fixed margin of
// 2^-18 covers every q that matters. The few elements that near a half-integer (exact
// ties among them) take the division.
__device__ __forceinline__ void tied_code_step(const float (&w)[kTiedE], float s, int (&c)[kTiedE]) {
  const float rs = 1.0f / s;
  float r[kTiedE];
  bool near = false;
#pragma unroll
  for (int j = 0; j < kTiedE; ++j) {
    const float q = w[j] * rs;
    r[j] = rintf(q);
    near |= fabsf(q - r[j]) >= 0.5f - 0x1p-18f;
  }
  if (__any(near)) {
#pragma unroll
    for (int j = 0; j < kTiedE; ++j) {
      const float q = w[j] * rs;
      if (fabsf(q - rintf(q)) >= 0.5f - 0x1p-18f) r[j] = rintf(w[j] / s);  // correctly rounded division
    }
  }
#pragma unroll
  for (int j = 0; j < kTiedE; ++j) c[j] = (int)__builtin_amdgcn_fmed3f(r[j], -4.0f, 4.0f);
}

// a + (the lane-pair partner's a), for a butterfly over lane bit M (both lanes of a pair
// add the same two values, so they hold the same sum)
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
  __shared__ __attribute__((aligned(16))) uint8_t s_bytes[16][128];
  const int lane = threadIdx.x & 63, grp = lane >> 4, u = lane & 15;
  const int lb = (threadIdx.x >> 6) * 4 + grp;  // the group's block in the workgroup
  const int64_t blk0 = (int64_t)blockIdx.x * 16, blk = min(blk0 + lb, nblocks - 1);
  const bool real = blk0 + lb < nblocks;  // a group past the last block repeats it, stores nothing
  const float* wb = w + blk * 256;
  float v[kTiedE];
#pragma unroll
  for (int j = 0; j < kTiedE; ++j) v[j] = wb[u + 16 * j];
  float amax = 0.0f;
#pragma unroll
  for (int j = 0; j < kTiedE; ++j) amax = fmaxf(amax, fabsf(v[j]));
  amax = fmaxf(amax, __int_as_float(lane_xor_i<8>(__float_as_int(amax))));
  amax = fmaxf(amax, __int_as_float(lane_xor_i<4>(__float_as_int(amax))));
  amax = fmaxf(amax, __int_as_float(lane_xor_i<2>(__float_as_int(amax))));
  amax = fmaxf(amax, __int_as_float(lane_xor_i<1>(__float_as_int(amax))));
  int c[kTiedE];
#pragma unroll
  for (int j = 0; j < kTiedE; ++j) c[j] = 0;
  const bool live = amax >= 0x1p-100f;  // uniform within the group
  float s = amax / 4.0f;
  int it = 0;
  bool done = !live;  // a group stops at its own stopping point; the wave runs until all do
  {
    int prev[kTiedE];
#pragma unroll
    for (int j = 0; j < kTiedE; ++j) prev[j] = 0;
    while (true) {
      int cn[kTiedE];
      tied_code_step(v, s, cn);
      int diff = 0;
#pragma unroll
      for (int j = 0; j < kTiedE; ++j) {
        diff |= cn[j] ^ prev[j];
        if (!done) c[j] = cn[j];
      }
      const uint64_t unchanged = __ballot(diff == 0);
      const bool same = ((unchanged >> (16 * grp)) & 0xFFFFu) == 0xFFFFu;
      if (!done) {
        ++it;
        done = (it > 1 && same) || it == max_iter;
      }
      if (__all(done)) break;
      // <w, c> in fp64 (exact products), pairwise halving: within the lane h = 128 .. 16,
      // across the group h = 8 .. 1; <c, c> exact
      double p[kTiedE];
#pragma unroll
      for (int j = 0; j < kTiedE; ++j) p[j] = (double)v[j] * (double)c[j];
#pragma unroll
      for (int h = kTiedE / 2; h >= 1; h >>= 1)
#pragma unroll
        for (int j = 0; j < h; ++j) p[j] = p[j] + p[j + h];
      double num = xor_add<8>(p[0]);
      num = xor_add<4>(num);
      num = xor_add<2>(num);
      num = xor_add<1>(num);
      int cc = 0;
#pragma unroll
      for (int j = 0; j < kTiedE; ++j) cc += c[j] * c[j];
      cc = xor_add<8>(cc);
      cc = xor_add<4>(cc);
      cc = xor_add<2>(cc);
      cc = xor_add<1>(cc);
#pragma unroll
      for (int j = 0; j < kTiedE; ++j) prev[j] = c[j];
      if (!done && cc != 0) s = (float)(num / (double)cc);
      if (!done && cc == 0) done = true;
    }
  }
  uint16_t h16 = 0;
  if (live) {
    // f16, nearest even, saturating at the largest finite value
    const _Float16 hs = s >= 65520.0f ? (_Float16)65504.0f : (_Float16)s;
    h16 = __builtin_bit_cast(uint16_t, hs);
    const float sd = (float)hs;
    if (sd == 0.0f) {
#pragma unroll
      for (int j = 0; j < kTiedE; ++j) c[j] = 0;
    } else {
      tied_code_step(v, sd, c);
    }
  } else {
#pragma unroll
    for (int j = 0; j < kTiedE; ++j) c[j] = 0;
  }
  // pack: weight u + 32m (j = 2m) takes the low nibble of byte 16m + u, weight u + 32m + 16
  // (j = 2m + 1) its high nibble
#pragma unroll
  for (int m = 0; m < kTiedE / 2; ++m)
    s_bytes[lb][16 * m + u] = (uint8_t)((c[2 * m] & 15) | ((c[2 * m + 1] & 15) << 4));
  __syncthreads();
  // 16 blocks x 128 bytes: lanes write 16 bytes each
  const int t = threadIdx.x;
  if (t < 128 && blk0 + (t >> 3) < nblocks)
    reinterpret_cast<uint4*>(codes + (blk0 + (t >> 3)) * 128)[t & 7] = reinterpret_cast<const uint4*>(s_bytes[t >> 3])[t & 7];
  if (u == 0 && real) {
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
  hipLaunchKernelGGL(k_tied_quantize, dim3((unsigned)((nblocks + 15) / 16)), dim3(256), 0, (hipStream_t)stream, w,
                     nblocks, (int)max_iter, codes, scales, iters);
  return check_launch("tq_tied_quantize");
}
