// The free-scale two-plane serving pass (Sec. 2.1: W ~ alpha1*T1 + alpha2*T2 with two
// free scales per group; Sec. 4.1: the pair does not fold, so it is served as its two
// trit planes stored apart (4.125 bits/weight), one integer pass per plane).
//
// Same memory plan as the folded pass: a 256-weight block is 128 bytes of trits (two
// planes x 2 bits), 8 lanes per block, a wave's 16-byte load covers 8 consecutive blocks
// (1 KB, coalesced), and each wave owns RPW whole rows whose loads are all issued up
// front. The two planes of a chunk share its 32 activations: per chunk a lane forms
// both planes' exact partials (64t bytes against q), the integer butterfly carries the
// pair per (row, token) item, and the lane that keeps an item applies the block's two
// scales, plane 1's multiply-add before plane 2's.
#include <hip/hip_ext.h>

#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

// Free-scale two-plane chunks: the 16 bytes of chunk j hold plane 1's 32 trits in bytes
// 0..7 and plane 2's in bytes 8..15; within a plane's two dwords, dword u, byte b, bit
// pair 2s..2s+1 is column 32j + 16u + 4s + b as a 2-bit two's-complement trit (00 = 0,
// 01 = +1, 11 = -1). Shifting the pair to a byte's top bits and masking leaves 64*t as a
// signed byte, so a plane decodes in one or two bitwise operations per activation dword
// and the byte dot's sum is exactly 64 times the trit dot.
constexpr uint32_t kTopPairs = 0xC0C0C0C0u;

// One plane's 32 trits (dwords w0, w1) as 64t bytes in the order of the activation
// dwords: t[4u + s] = columns 16u + 4s .. 16u + 4s + 3.
__device__ __forceinline__ void unpack64t(uint32_t w0, uint32_t w1, int (&t)[8]) {
  t[0] = int((w0 << 6) & kTopPairs); t[1] = int((w0 << 4) & kTopPairs);
  t[2] = int((w0 << 2) & kTopPairs); t[3] = int(w0 & kTopPairs);
  t[4] = int((w1 << 6) & kTopPairs); t[5] = int((w1 << 4) & kTopPairs);
  t[6] = int((w1 << 2) & kTopPairs); t[7] = int(w1 & kTopPairs);
}

// Both planes' partials of one 16-byte chunk against 32 int8 activations: exact
// multiples of 64 (|.| <= 32 * 64 * 127 per chunk; a whole block stays below 2^21, and
// >> 6 of it is the exact block sum of t * q).
__device__ __forceinline__ void dot2_chunk16(const uint4 w, const int (&a)[8], int& p1, int& p2) {
  int t[8];
  unpack64t(w.x, w.y, t);
  int s1 = 0;
#pragma unroll
  for (int m = 0; m < 8; ++m) s1 = __builtin_amdgcn_sdot4(t[m], a[m], s1, false);
  unpack64t(w.z, w.w, t);
  int s2 = 0;
#pragma unroll
  for (int m = 0; m < 8; ++m) s2 = __builtin_amdgcn_sdot4(t[m], a[m], s2, false);
  p1 = s1;
  p2 = s2;
}

// LOOP = false: one chunk of at most NT tokens (t <= NT), no token loop, so nothing
// loop-invariant (the unpacked planes) is hoisted and kept live across it.
template <int NL, int NT, int RPW, bool LOOP>
__global__ __launch_bounds__(256) void k_gemv2(const uint8_t* __restrict__ codes,
                                               const uint32_t* __restrict__ scales, int n, int kb,
                                               const int8_t* __restrict__ q, const float* __restrict__ d, int t,
                                               float* __restrict__ y, int32_t* __restrict__ isum_dbg) {
  static_assert(RPW <= 8 && (RPW & (RPW - 1)) == 0, "RPW: a power of two <= 8");
  using RI = RowReduce<RPW * NT, 2>;  // integer butterfly: items carry both planes
  using RF = RowReduce<RPW * NT, 1>;  // fp32 butterfly: one row total per item
  constexpr int KI = RI::KI;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 3, cp = lane & 7;
  const int row0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * RPW;
  if (row0 >= n) return;
  const int64_t k = (int64_t)kb * 256;

  // The activations and block scales of a chunk of NT tokens. The first chunk's are
  // requested before the weights: a compute unit returns loads in issue order, so these
  // small, cache-resident loads would otherwise wait behind every weight load in flight.
  int qa[NT][NL][8];
  float dk[KI][NL];
  auto load_acts = [&](int t0) {
#pragma unroll
    for (int tt = 0; tt < NT; ++tt)
#pragma unroll
      for (int i = 0; i < NL; ++i) {
        const int64_t tc = min(t0 + tt, t - 1);
        const int4* p = reinterpret_cast<const int4*>(q + tc * k + min(8 * i + g, kb - 1) * 256 + cp * 32);
        const int4 lo = p[0], hi = p[1];
        qa[tt][i][0] = lo.x; qa[tt][i][1] = lo.y; qa[tt][i][2] = lo.z; qa[tt][i][3] = lo.w;
        qa[tt][i][4] = hi.x; qa[tt][i][5] = hi.y; qa[tt][i][6] = hi.z; qa[tt][i][7] = hi.w;
      }
    // the lane's kept items: their tokens' block scales (masked at use: a select here
    // would make the compiler wait for these loads before issuing the weights)
#pragma unroll
    for (int kk = 0; kk < KI; ++kk) {
      const int tok = t0 + RI::kept(kk, lane) % NT;
#pragma unroll
      for (int i = 0; i < NL; ++i) {
        const int b = 8 * i + g;
        dk[kk][i] = d[(int64_t)min(tok, t - 1) * kb + min(b, kb - 1)];
      }
    }
  };
  load_acts(0);

  // Loads are unconditional from clamped addresses (a predicated load becomes a branch
  // that serializes the loads): rows past n are computed and not stored, blocks past kb
  // get d = 0 and add exactly nothing. Buffer loads relative to the wave's first row:
  // one 32-bit offset per load, no 64-bit address arithmetic per lane.
  const int wrow0 = __builtin_amdgcn_readfirstlane(row0);
  const int nrows = min(RPW, n - wrow0);
  const __amdgpu_buffer_rsrc_t cr = make_rsrc(codes + (int64_t)wrow0 * kb * 128, (uint32_t)(nrows * kb * 128));
  uint4 w[RPW][NL];
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    const int rr = min(r, nrows - 1);
#pragma unroll
    for (int i = 0; i < NL; ++i) w[r][i] = buf_load16(cr, (uint32_t)((rr * kb + min(8 * i + g, kb - 1)) * 128 + cp * 16), 0);
  }
  // after the block butterfly a lane keeps items of one row (RPW <= 8): its scale pairs
  const int lrow = min(row0 + rev_bits<clog2(RPW)>(lane & (RPW - 1)), n - 1);
  float a1[NL], a2[NL];
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const uint32_t pr = scales[(int64_t)lrow * kb + min(8 * i + g, kb - 1)];
    a1[i] = f16_bits_to_f32((uint16_t)(pr & 0xFFFF));
    a2[i] = f16_bits_to_f32((uint16_t)(pr >> 16));
  }

  __builtin_amdgcn_sched_barrier(0);  // every load above is issued before any math

  // t >= 1 (the launcher returns early for t == 0): a do-while keeps the loads above
  // in the kernel's entry block instead of sinking them under a loop guard
  int t0 = 0;
  do {
    if (t0 > 0) load_acts(t0);
    float acc[KI];
#pragma unroll
    for (int kk = 0; kk < KI; ++kk) acc[kk] = 0.0f;
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      int p[RPW * NT * 2];
#pragma unroll
      for (int r = 0; r < RPW; ++r)
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) dot2_chunk16(w[r][i], qa[tt][i], p[(r * NT + tt) * 2], p[(r * NT + tt) * 2 + 1]);
      RI::block_sums(p);
#pragma unroll
      for (int kk = 0; kk < KI; ++kk) {
        const int is1 = p[2 * kk] >> 6, is2 = p[2 * kk + 1] >> 6;  // exact block sums per plane
        const int tok = t0 + RI::kept(kk, lane) % NT, b = 8 * i + g;
        const float dv = (tok < t && b < kb) ? dk[kk][i] : 0.0f;
        acc[kk] = fmaf(a1[i] * dv, (float)is1, acc[kk]);
        acc[kk] = fmaf(a2[i] * dv, (float)is2, acc[kk]);
        if (isum_dbg != nullptr && RI::block_writer(lane)) {
          const int row = row0 + RI::kept(kk, lane) / NT;
          if (tok < t && row < n && b < kb) {
            int32_t* o = isum_dbg + (((int64_t)tok * n + row) * kb + b) * 2;
            o[0] = is1;
            o[1] = is2;
          }
        }
      }
    }
    RF::block_totals(acc);
    if (RF::writer(lane)) {
      const int it = RF::item(lane), tok = t0 + it % NT, row = row0 + it / NT;
      if (tok < t && row < n) y[(int64_t)tok * n + row] = acc[0];
    }
    t0 += NT;
  } while (LOOP && t0 < t);
}

using gemv2_fn = void (*)(const uint8_t*, const uint32_t*, int, int, const int8_t*, const float*, int, float*,
                          int32_t*);

// Register budget (the launcher's rules): four rows per wave only where a row is at
// most two loads, four tokens per chunk only where a row is at most four loads.
template <int NL>
static gemv2_fn pick_gemv2_nl(int nt, int rpw, bool one) {
  if constexpr (NL <= 2) {
    if (nt == 1) return rpw == 1 ? k_gemv2<NL, 1, 1, false> : k_gemv2<NL, 1, 4, false>;
    return rpw == 1 ? k_gemv2<NL, 4, 1, true> : k_gemv2<NL, 4, 4, true>;
  } else if constexpr (NL <= 4) {
    (void)rpw;
    return nt == 1 ? k_gemv2<NL, 1, 1, false> : k_gemv2<NL, 4, 1, true>;
  } else {
    (void)rpw;
    (void)nt;
    return one ? k_gemv2<NL, 1, 1, false> : k_gemv2<NL, 1, 1, true>;
  }
}

static gemv2_fn pick_gemv2(int nl, int nt, int rpw, bool one) {
  switch (nl) {
    case 1: return pick_gemv2_nl<1>(nt, rpw, one);
    case 2: return pick_gemv2_nl<2>(nt, rpw, one);
    case 3: return pick_gemv2_nl<3>(nt, rpw, one);
    case 4: return pick_gemv2_nl<4>(nt, rpw, one);
    case 5: return pick_gemv2_nl<5>(nt, rpw, one);
    case 6: return pick_gemv2_nl<6>(nt, rpw, one);
    case 7: return pick_gemv2_nl<7>(nt, rpw, one);
    default: return pick_gemv2_nl<8>(nt, rpw, one);
  }
}

// Rows per wave for large matrices when several tokens share a chunk (build-time knob).
#ifndef TQ_GEMV2_RPW_MULTI
#define TQ_GEMV2_RPW_MULTI 1
#endif

static tq_status gemv2_run(const tq_mat2* w, const int8_t* q, const float* d, int64_t t, float* y, int32_t* isum_dbg,
                           void* stream, void* const* events) {
  if (!w) return fail(TQ_ERR_INVALID, "tq_gemv2: null matrix descriptor");
  const int n = w->n, k = w->k;
  if (n < 1) return fail(TQ_ERR_INVALID, "tq_gemv2: n = %d < 1", n);
  if (k <= 0 || k % 256 != 0 || k > kMaxK)
    return fail(TQ_ERR_INVALID, "tq_gemv2: k = %d must be a positive multiple of 256 <= %d", k, kMaxK);
  if (t < 0 || t > INT32_MAX) return fail(TQ_ERR_INVALID, "tq_gemv2: t = %lld out of range", (long long)t);
  if (t == 0) return TQ_OK;
  if (!w->codes || !w->scales || !q || !d || !y) return fail(TQ_ERR_INVALID, "tq_gemv2: null pointer");
  if (!aligned(w->codes, 128)) return fail(TQ_ERR_ALIGN, "tq_gemv2: codes must be 128-byte aligned");
  if (!aligned(q, 16) || !aligned(w->scales, 4) || !aligned(d, 4) || !aligned(y, 4) ||
      (isum_dbg && !aligned(isum_dbg, 4)))
    return fail(TQ_ERR_ALIGN, "tq_gemv2: q must be 16-byte and scales 4-byte aligned, other buffers naturally aligned");
  if ((int64_t)t * n * (k / 256) > ((int64_t)1 << 39)) return fail(TQ_ERR_INVALID, "tq_gemv2: problem too large");
  const int kb = k / 256, nl = (kb + 7) / 8;
  const int nt = (t == 1 || nl > 4) ? 1 : 4;
  const int rpw = (n >= 16384 && nl <= 2) ? (nt == 1 ? 4 : TQ_GEMV2_RPW_MULTI) : 1;
  const int64_t waves = (n + rpw - 1) / rpw;
  const unsigned wgs = (unsigned)((waves + 3) / 4);
  const uint32_t* sc = reinterpret_cast<const uint32_t*>(w->scales);
  (void)hipGetLastError();
  if (events)
    hipExtLaunchKernelGGL(pick_gemv2(nl, nt, rpw, t == 1), dim3(wgs), dim3(256), 0, (hipStream_t)stream,
                          (hipEvent_t)events[0], (hipEvent_t)events[1], 0, w->codes, sc, n, kb, q, d, (int)t, y,
                          isum_dbg);
  else
    hipLaunchKernelGGL(pick_gemv2(nl, nt, rpw, t == 1), dim3(wgs), dim3(256), 0, (hipStream_t)stream, w->codes, sc, n, kb, q,
                       d, (int)t, y, isum_dbg);
  return check_launch("tq_gemv2");
}

}  // namespace tq

extern "C" tq_status tq_gemv2(const tq_mat2* w, const int8_t* q, const float* d, int64_t t, float* y,
                              int32_t* isum_dbg, void* stream) {
  tq::clear_error();
  return tq::gemv2_run(w, q, d, t, y, isum_dbg, stream, nullptr);
}

extern "C" tq_status tq_gemv2_timed(const tq_mat2* w, const int8_t* q, const float* d, int64_t t, float* y,
                                    int32_t* isum_dbg, void* stream, void* const* events) {
  tq::clear_error();
  if (!events || !events[0] || !events[1]) return tq::fail(TQ_ERR_INVALID, "tq_gemv2_timed: null event");
  return tq::gemv2_run(w, q, d, t, y, isum_dbg, stream, events);
}
