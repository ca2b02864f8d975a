// Free-scale solver (Sec. 2.1: PTQTP fits W ~ alpha1*T1 + alpha2*T2 per group by
// alternating plane and scale updates with two free scales; the tie alpha = (3s, s) is
// its constrained case). Started from a tied fit, it refines each 256-weight block into
// the free-scale two-plane layout: least-squares scale pairs and best-of-nine plane
// pairs in turn, every decision in a fixed precision and order (stated in tq.h), so the
// result is reproducible bit for bit.
#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

// A 16-lane group owns one block (four a wave), lane u holding weights u + 16j.
constexpr int kFreeE = 16;

template <int M>
__device__ __forceinline__ double xor_addd(double a) {
  const int lo = __double2loint(a), hi = __double2hiint(a);
  return a + __hiloint2double(lane_xor_i<M>(hi), lane_xor_i<M>(lo));
}
template <int M>
__device__ __forceinline__ int xor_addi(int a) {
  return a + lane_xor_i<M>(a);
}

// Sum over the block in the pairwise-halving order: within the lane for h = 128 .. 16,
// then across the group's lanes for h = 8 .. 1.
__device__ __forceinline__ double block_sum(double (&p)[kFreeE]) {
#pragma unroll
  for (int h = kFreeE / 2; h >= 1; h >>= 1)
#pragma unroll
    for (int j = 0; j < h; ++j) p[j] = p[j] + p[j + h];
  double s = xor_addd<8>(p[0]);
  s = xor_addd<4>(s);
  s = xor_addd<2>(s);
  return xor_addd<1>(s);
}
__device__ __forceinline__ int block_sum(int a) {
  a = xor_addi<8>(a);
  a = xor_addi<4>(a);
  a = xor_addi<2>(a);
  return xor_addi<1>(a);
}

// The plane step: each weight takes the first pair in the order 0, -1, +1 (t1 outer,
// t2 inner) with the least |w - (a1 t1 + a2 t2)| in fp64. The nine candidate values
// are the block's own (a1 t1 exact, one rounding in the sum).
__device__ __forceinline__ void free_plane_step(const float (&w)[kFreeE], float a1, float a2, int (&t1)[kFreeE],
                                                int (&t2)[kFreeE]) {
#pragma clang fp contract(off)
  constexpr int kOrd[3] = {0, -1, 1};
  double cand[9];
#pragma unroll
  for (int x = 0; x < 3; ++x)
#pragma unroll
    for (int y = 0; y < 3; ++y) cand[3 * x + y] = (double)a1 * kOrd[x] + (double)a2 * kOrd[y];
#pragma unroll
  for (int j = 0; j < kFreeE; ++j) {
    const double wd = (double)w[j];
    double best = fabs(wd - cand[0]);
    int bi = 0;
#pragma unroll
    for (int c = 1; c < 9; ++c) {
      const double e = fabs(wd - cand[c]);
      if (e < best) {
        best = e;
        bi = c;
      }
    }
    t1[j] = kOrd[bi / 3];
    t2[j] = kOrd[bi % 3];
  }
}

// f32 -> f16 bits, nearest even, saturating to +-65504.
__device__ __forceinline__ uint16_t f16_sat(float x) {
  const float c = fminf(fmaxf(x, -65504.0f), 65504.0f);
  // values in (65504, 65520) round to 65504 anyway; clamping first keeps 65520 and up
  // from rounding to infinity
  return __builtin_bit_cast(uint16_t, (_Float16)(fabsf(x) >= 65520.0f ? c : x));
}

__global__ __launch_bounds__(256) void k_free_quantize(const float* __restrict__ w, int64_t nblocks, int max_iter,
                                                       const uint8_t* __restrict__ tcodes,
                                                       const uint16_t* __restrict__ tscales,
                                                       uint8_t* __restrict__ codes2, uint32_t* __restrict__ scales2,
                                                       uint8_t* __restrict__ iters) {
#pragma clang fp contract(off)
  __shared__ uint32_t s_w[16][32];  // per block: the 128 two-plane bytes as dwords
  const int lane = threadIdx.x & 63, grp = lane >> 4, u = lane & 15;
  const int lb = (threadIdx.x >> 6) * 4 + grp;
  const int64_t blk0 = (int64_t)blockIdx.x * 16, blk = min(blk0 + lb, nblocks - 1);
  const bool real = blk0 + lb < nblocks;  // a group past the last block repeats it, stores nothing
  for (int i = threadIdx.x; i < 16 * 32; i += 256) (&s_w[0][0])[i] = 0u;
  const float* wb = w + blk * 256;
  float v[kFreeE];
#pragma unroll
  for (int j = 0; j < kFreeE; ++j) v[j] = wb[u + 16 * j];
  // the tied fit: weight u + 32m in the low nibble of byte 16m + u, u + 32m + 16 in the high
  int t1[kFreeE], t2[kFreeE];
  const uint8_t* cb = tcodes + blk * 128;
#pragma unroll
  for (int m = 0; m < kFreeE / 2; ++m) {
    const int byte = cb[16 * m + u];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int nib = (byte >> (4 * h)) & 15;
      const int c = nib >= 8 ? nib - 16 : nib;
      const int a = (c + 4) / 3 - 1;  // unfold: balanced-ternary digits of c
      t1[2 * m + h] = a;
      t2[2 * m + h] = c - 3 * a;
    }
  }
  const float s = f16_bits_to_f32(tscales[blk]);
  const bool live = s != 0.0f;  // uniform within the group
  float a1 = 3.0f * s, a2 = s;
  int it = 0;
  bool done = !live;  // a group stops at its own stopping point; the wave runs until all do
  while (!__all(done)) {
    // scale step: least squares for (a1, a2) given the planes
    double pu[kFreeE], pv[kFreeE];
    int sa = 0, sb = 0, sc = 0;
#pragma unroll
    for (int j = 0; j < kFreeE; ++j) {
      pu[j] = (double)v[j] * (double)t1[j];
      pv[j] = (double)v[j] * (double)t2[j];
      sa += t1[j] * t1[j];
      sb += t1[j] * t2[j];
      sc += t2[j] * t2[j];
    }
    const double su = block_sum(pu), sv = block_sum(pv);
    sa = block_sum(sa);
    sb = block_sum(sb);
    sc = block_sum(sc);
    const int det = sa * sc - sb * sb;  // |.| <= 256^2: exact in int
    if (!done && det > 0) {
      const double num1 = (double)sc * su - (double)sb * sv;
      const double num2 = (double)sa * sv - (double)sb * su;
      a1 = (float)(num1 / (double)det);
      a2 = (float)(num2 / (double)det);
    }
    // plane step
    int n1[kFreeE], n2[kFreeE];
    free_plane_step(v, a1, a2, n1, n2);
    int diff = 0;
#pragma unroll
    for (int j = 0; j < kFreeE; ++j) {
      diff |= (n1[j] ^ t1[j]) | (n2[j] ^ t2[j]);
      if (!done) {
        t1[j] = n1[j];
        t2[j] = n2[j];
      }
    }
    const uint64_t unchanged = __ballot(diff == 0);
    const bool same = ((unchanged >> (16 * grp)) & 0xFFFFu) == 0xFFFFu;
    if (!done) {
      ++it;
      done = same || it == max_iter;
    }
  }
  uint16_t h1 = 0, h2 = 0;
  if (live) {
    h1 = f16_sat(a1);
    h2 = f16_sat(a2);
    free_plane_step(v, f16_bits_to_f32(h1), f16_bits_to_f32(h2), t1, t2);
  } else {
#pragma unroll
    for (int j = 0; j < kFreeE; ++j) t1[j] = t2[j] = 0;
  }
  __syncthreads();  // s_w cleared
  // pack: weight u + 16j is column 32 (j / 2) + 16 (j % 2) + 4 (u / 4) + (u % 4) of its
  // block, i.e. plane p's dword 4 (j / 2) + 2p + (j % 2), bits 8 (u % 4) + 2 (u / 4)
  const int sh = 8 * (u & 3) + 2 * (u >> 2);
#pragma unroll
  for (int j = 0; j < kFreeE; ++j) {
    atomicOr(&s_w[lb][4 * (j >> 1) + (j & 1)], (uint32_t)(t1[j] & 3) << sh);
    atomicOr(&s_w[lb][4 * (j >> 1) + 2 + (j & 1)], (uint32_t)(t2[j] & 3) << sh);
  }
  __syncthreads();
  const int t = threadIdx.x;
  if (t < 128 && blk0 + (t >> 3) < nblocks)
    reinterpret_cast<uint4*>(codes2 + (blk0 + (t >> 3)) * 128)[t & 7] = reinterpret_cast<const uint4*>(s_w[t >> 3])[t & 7];
  if (u == 0 && real) {
    scales2[blk] = (uint32_t)h1 | ((uint32_t)h2 << 16);
    if (iters) iters[blk] = (uint8_t)it;
  }
}

}  // namespace tq

extern "C" tq_status tq_free_quantize(const float* w, int32_t n, int32_t k, int32_t max_iter,
                                      const uint8_t* tied_codes, const uint16_t* tied_scales, uint8_t* codes2,
                                      uint16_t* scales2, uint8_t* iters, void* stream) {
  using namespace tq;
  clear_error();
  if (n < 0 || k <= 0 || k % 256 != 0)
    return fail(TQ_ERR_INVALID, "tq_free_quantize: n = %d, k = %d (need n >= 0, k a positive multiple of 256)", n, k);
  if (max_iter < 1 || max_iter > 255)
    return fail(TQ_ERR_INVALID, "tq_free_quantize: max_iter = %d outside [1, 255]", max_iter);
  if (n == 0) return TQ_OK;
  if (!w || !tied_codes || !tied_scales || !codes2 || !scales2)
    return fail(TQ_ERR_INVALID, "tq_free_quantize: null pointer");
  if (!aligned(w, 4) || !aligned(tied_codes, 128) || !aligned(tied_scales, 2) || !aligned(codes2, 128) ||
      !aligned(scales2, 4))
    return fail(TQ_ERR_ALIGN,
                "tq_free_quantize: w 4-byte, codes 128-byte, tied scales 2-byte and scale pairs 4-byte aligned");
  const int64_t nblocks = (int64_t)n * (k / 256);
  (void)hipGetLastError();
  hipLaunchKernelGGL(k_free_quantize, dim3((unsigned)((nblocks + 15) / 16)), dim3(256), 0, (hipStream_t)stream, w,
                     nblocks, (int)max_iter, tied_codes, tied_scales, codes2, reinterpret_cast<uint32_t*>(scales2),
                     iters);
  return check_launch("tq_free_quantize");
}
