// The serving dot pass for one tq matrix (Sec. 2.2): exact int32 block sums of the
// folded codes against int8 block-quantized activations, then one fp32 multiply-add
// per block.
//
// Decode is HBM-bound (0.5 byte of codes per weight, a few integer ops per weight per
// token), so the kernel is shaped for the memory system: each wave owns RPW whole
// rows, issues all of their 16-byte code loads up front (a wave load = 8 consecutive
// blocks = 1 KB, fully coalesced), and keeps them in registers, unpacked, while it walks
// the tokens NT at a time. A lane always covers the same columns of every row it owns
// (block 8i + l/8, chunk l & 7 for load i), so its activations sit in registers too,
// loaded once per token chunk. Per load, the lanes' exact 32-code partials of all
// RPW x NT (row, token) items meet in one integer butterfly over the 8 lanes of each
// block (exact block sums, which the debug output stores), each kept block sum gets one
// fp32 multiply-add by f32(s) * d, and one fp32 butterfly over the blocks gives the row
// totals.
#include <hip/hip_ext.h>

#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

// LOOP = false: one chunk of at most NT tokens (t <= NT), no token loop, so nothing
// loop-invariant is hoisted and kept live across it.
template <int NL, int NT, int RPW, bool LOOP>
__global__ __launch_bounds__(256) void k_gemv(const uint8_t* __restrict__ codes,
                                              const uint16_t* __restrict__ scales, int n, int kb,
                                              const int8_t* __restrict__ q, const float* __restrict__ d, int t,
                                              float* __restrict__ y, int32_t* __restrict__ isum_dbg) {
  static_assert(RPW <= 8 && (RPW & (RPW - 1)) == 0, "RPW: a power of two <= 8");
  using RR = RowReduce<RPW * NT, 1>;
  constexpr int KI = RR::KI;
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
      const int tok = t0 + RR::kept(kk, lane) % NT;
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
  // after the block butterfly a lane keeps items of one row (RPW <= 8): its scales
  const int lrow = min(row0 + rev_bits<clog2(RPW)>(lane & (RPW - 1)), n - 1);
  float s[NL];
#pragma unroll
  for (int i = 0; i < NL; ++i) s[i] = f16_bits_to_f32(scales[(int64_t)lrow * kb + min(8 * i + g, kb - 1)]);

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
      int p[RPW * NT];
#pragma unroll
      for (int r = 0; r < RPW; ++r)
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) {
          int c[8];
          unpack16c(w[r][i], c);
          p[r * NT + tt] = dot32x16(c, qa[tt][i]);
        }
      RR::block_sums(p);
#pragma unroll
      for (int kk = 0; kk < KI; ++kk) {
        const int is = p[kk] >> 4;  // exact block sum of c * q
        const int tok = t0 + RR::kept(kk, lane) % NT, b = 8 * i + g;
        const float dv = (tok < t && b < kb) ? dk[kk][i] : 0.0f;
        acc[kk] = fmaf(s[i] * dv, (float)is, acc[kk]);
        if (isum_dbg != nullptr && RR::block_writer(lane)) {
          const int row = row0 + RR::kept(kk, lane) / NT;
          if (tok < t && row < n && b < kb) isum_dbg[((int64_t)tok * n + row) * kb + b] = is;
        }
      }
    }
    RR::block_totals(acc);
    if (RR::writer(lane)) {
      const int it = RR::item(lane), tok = t0 + it % NT, row = row0 + it / NT;
      if (tok < t && row < n) y[(int64_t)tok * n + row] = acc[0];
    }
    t0 += NT;
  } while (LOOP && t0 < t);
}

// One token with fp32 activations, quantization fused: each workgroup quantizes x into LDS
// (8-lane group gid owns block gid, further blocks strided over the groups; waves with no
// block skip the load), with its weight loads issued right behind the x loads so that
// both are in flight together; after one barrier the pass runs as k_gemv's at one token
// (same butterflies, same per-block fp32 multiply-add, so the same bits as quantizing
// first and running k_gemv with the same rows per wave). Workgroup 0 also stores the
// quantized activations for the caller. Rows past n load the last row and store nothing.
template <int NL, int RPW, int WAVES, bool RAGGED>
__global__ __launch_bounds__(WAVES * 64) void k_gemv_x(const uint8_t* __restrict__ codes,
                                                       const uint16_t* __restrict__ scales, int n, int kb,
                                                       const float* __restrict__ x, int8_t* __restrict__ q_out,
                                                       float* __restrict__ d_out, int32_t* __restrict__ b_out,
                                                       float* __restrict__ y, int32_t* __restrict__ isum_dbg) {
  static_assert(RPW <= 8 && (RPW & (RPW - 1)) == 0, "RPW: a power of two <= 8");
  __shared__ __attribute__((aligned(16))) int8_t s_q[kMaxK];
  __shared__ float s_d[kMaxK / 256];
  __shared__ int s_b[kMaxK / 256];
  using RR = RowReduce<RPW, 1>;
  static_assert(RR::KI == 1, "a lane keeps one row after the block butterfly");
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 3, cp = lane & 7, gid = wv * 8 + g;
  const int row0 = (blockIdx.x * WAVES + wv) * RPW;

  // x first (its wait must not queue behind the weights), then every weight load
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, (uint32_t)kb * 1024u);
  float v[32];
  const bool xw = wv * 8 < kb;  // wave-uniform: the wave has blocks of x to quantize
  if (xw) buf_load32f(xr, (uint32_t)min(gid, kb - 1), cp, v);
  __builtin_amdgcn_sched_barrier(0);
  const __amdgpu_buffer_rsrc_t cr = make_rsrc(codes, (uint32_t)n * (uint32_t)kb * 128u);
  const __amdgpu_buffer_rsrc_t sr = make_rsrc(scales, (uint32_t)n * (uint32_t)kb * 2u);
  uint4 w[RPW][NL];
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    const uint32_t srow = (uint32_t)min(row0 + r, n - 1) * (uint32_t)kb * 128u;
#pragma unroll
    for (int i = 0; i < NL; ++i)
      w[r][i] = buf_load16(cr, (uint32_t)min(8 * i + g, kb - 1) * 128u + (uint32_t)cp * 16u, srow);
  }
  // after the block butterfly a lane keeps the row rev(lane bits): its scales
  const uint32_t lrow = (uint32_t)min(row0 + rev_bits<clog2(RPW)>(lane & (RPW - 1)), n - 1) * (uint32_t)kb;
  uint16_t sh[NL];
#pragma unroll
  for (int i = 0; i < NL; ++i) sh[i] = buf_load_u16(sr, (lrow + (uint32_t)min(8 * i + g, kb - 1)) * 2u, 0);
  if (xw) quantize_to_lds(v, min(gid, kb - 1), cp, s_q, s_d, s_b, gid < kb);
  for (int blk = gid + WAVES * 8; blk < kb; blk += WAVES * 8) {
    buf_load32f(xr, (uint32_t)blk, cp, v);
    quantize_to_lds(v, blk, cp, s_q, s_d, s_b, true);
  }
  __syncthreads();
  if (blockIdx.x == 0) {  // the quantized activations, once per call
    for (int i = threadIdx.x; i < kb * 64; i += WAVES * 64)
      reinterpret_cast<int*>(q_out)[i] = reinterpret_cast<const int*>(s_q)[i];
    for (int i = threadIdx.x; i < kb; i += WAVES * 64) {
      d_out[i] = s_d[i];
      b_out[i] = s_b[i];
    }
  }
  if (row0 >= n) return;
  float acc[1] = {0.0f};
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const int b = 8 * i + g, bc = min(b, kb - 1);
    const int4* qp = reinterpret_cast<const int4*>(s_q + bc * 256 + cp * 32);
    const int4 lo = qp[0], hi = qp[1];
    const int qa[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    int p[RPW];
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      int c[8];
      unpack16c(w[r][i], c);
      p[r] = dot32x16(c, qa);
    }
    RR::block_sums(p);
    const int is = p[0] >> 4;  // exact block sum of c * q
    const float dv = (!RAGGED || b < kb) ? s_d[bc] : 0.0f;
    acc[0] = fmaf(f16_bits_to_f32(sh[i]) * dv, (float)is, acc[0]);
    if (isum_dbg != nullptr && RR::block_writer(lane) && b < kb) {
      const int row = row0 + RR::kept(0, lane);
      if (row < n) isum_dbg[(int64_t)row * kb + b] = is;
    }
  }
  RR::block_totals(acc);
  if (RR::writer(lane)) {
    const int row = row0 + RR::item(lane);
    if (row < n) y[row] = acc[0];
  }
}

using gemv_x_fn = void (*)(const uint8_t*, const uint16_t*, int, int, const float*, int8_t*, float*, int32_t*,
                           float*, int32_t*);
constexpr int kGemvXWaves = 4;

template <int RPW, bool R>
static gemv_x_fn pick_gemv_x_r(int nl) {
  switch (nl) {
    case 1: return k_gemv_x<1, RPW, kGemvXWaves, R>;
    case 2: return k_gemv_x<2, RPW, kGemvXWaves, R>;
    case 3: return k_gemv_x<3, RPW, kGemvXWaves, R>;
    case 4: return k_gemv_x<4, RPW, kGemvXWaves, R>;
    case 5: return k_gemv_x<5, RPW, kGemvXWaves, R>;
    case 6: return k_gemv_x<6, RPW, kGemvXWaves, R>;
    case 7: return k_gemv_x<7, RPW, kGemvXWaves, R>;
    default: return k_gemv_x<8, RPW, kGemvXWaves, R>;
  }
}

// The same rows per wave as k_gemv at one token (so both give the same bits).
static gemv_x_fn pick_gemv_x(int kb, int rpw) {
  const int nl = (kb + 7) / 8;
  const bool r = kb % 8 != 0;
  if (rpw == 4) return r ? pick_gemv_x_r<4, true>(nl) : pick_gemv_x_r<4, false>(nl);
  return r ? pick_gemv_x_r<1, true>(nl) : pick_gemv_x_r<1, false>(nl);
}

using gemv_fn = void (*)(const uint8_t*, const uint16_t*, int, int, const int8_t*, const float*, int, float*,
                         int32_t*);

// Four rows per wave only where a row is at most two loads (the launcher's rule).
template <int NL>
static gemv_fn pick_gemv_nl(int nt, int rpw) {
  // one token: a single pass; several: chunks of four
  if constexpr (NL <= 2) {
    if (nt == 1) return rpw == 1 ? k_gemv<NL, 1, 1, false> : k_gemv<NL, 1, 4, false>;
    return rpw == 1 ? k_gemv<NL, 4, 1, true> : k_gemv<NL, 4, 4, true>;
  } else {
    (void)rpw;
    return nt == 1 ? k_gemv<NL, 1, 1, false> : k_gemv<NL, 4, 1, true>;
  }
}

static gemv_fn pick_gemv(int nl, int nt, int rpw) {
  switch (nl) {
    case 1: return pick_gemv_nl<1>(nt, rpw);
    case 2: return pick_gemv_nl<2>(nt, rpw);
    case 3: return pick_gemv_nl<3>(nt, rpw);
    case 4: return pick_gemv_nl<4>(nt, rpw);
    case 5: return pick_gemv_nl<5>(nt, rpw);
    case 6: return pick_gemv_nl<6>(nt, rpw);
    case 7: return pick_gemv_nl<7>(nt, rpw);
    default: return pick_gemv_nl<8>(nt, rpw);
  }
}

}  // namespace tq

namespace tq {
// Rows per wave for large matrices when several tokens share a chunk (build-time knob).
#ifndef TQ_GEMV_RPW_MULTI
#define TQ_GEMV_RPW_MULTI 4
#endif

static tq_status gemv_run(const tq_mat* w, const int8_t* q, const float* d, const int32_t* bsum, int64_t t, float* y,
                          int32_t* isum_dbg, void* stream, void* const* events) {
  if (!w) return fail(TQ_ERR_INVALID, "tq_gemv: null matrix descriptor");
  const int n = w->n, k = w->k;
  if (n < 1) return fail(TQ_ERR_INVALID, "tq_gemv: n = %d < 1", n);
  if (k <= 0 || k % 256 != 0 || k > kMaxK)
    return fail(TQ_ERR_INVALID, "tq_gemv: k = %d must be a positive multiple of 256 <= %d", k, kMaxK);
  if (t < 0 || t > INT32_MAX) return fail(TQ_ERR_INVALID, "tq_gemv: t = %lld out of range", (long long)t);
  if (t == 0) return TQ_OK;
  if (!w->codes || !w->scales || !q || !d || !y) return fail(TQ_ERR_INVALID, "tq_gemv: null pointer");
  if (!aligned(w->codes, 128)) return fail(TQ_ERR_ALIGN, "tq_gemv: codes must be 128-byte aligned");
  (void)bsum;  // signed codes: no offset correction
  if (!aligned(q, 16) || !aligned(w->scales, 2) || !aligned(d, 4) || !aligned(y, 4) ||
      (isum_dbg && !aligned(isum_dbg, 4)))
    return fail(TQ_ERR_ALIGN, "tq_gemv: q must be 16-byte aligned, other buffers naturally aligned");
  if ((int64_t)t * n * (k / 256) > ((int64_t)1 << 40)) return fail(TQ_ERR_INVALID, "tq_gemv: problem too large");
  const int kb = k / 256, nl = (kb + 7) / 8;
  const int nt = t == 1 ? 1 : 4;
  // Few rows: one row per wave, to spread a small matrix over all CUs.
  const int rpw = (n >= 16384 && nl <= 2) ? (nt == 1 ? 4 : TQ_GEMV_RPW_MULTI) : 1;
  const int64_t waves = (n + rpw - 1) / rpw;
  const unsigned wgs = (unsigned)((waves + 3) / 4);
  (void)hipGetLastError();
  if (events)
    hipExtLaunchKernelGGL(pick_gemv(nl, nt, rpw), dim3(wgs), dim3(256), 0, (hipStream_t)stream, (hipEvent_t)events[0],
                          (hipEvent_t)events[1], 0, w->codes, w->scales, n, kb, q, d, (int)t, y, isum_dbg);
  else
    hipLaunchKernelGGL(pick_gemv(nl, nt, rpw), dim3(wgs), dim3(256), 0, (hipStream_t)stream, w->codes, w->scales, n,
                       kb, q, d, (int)t, y, isum_dbg);
  return check_launch("tq_gemv");
}
}  // namespace tq

namespace tq {
static tq_status gemv_f32_run(const tq_mat* w, const float* x, int64_t t, float* y, int8_t* q, float* d, int32_t* bsum,
                              int32_t* isum_dbg, void* stream, void* const* events) {
  const char* fn = events ? "tq_gemv_f32_timed" : "tq_gemv_f32";
  if (!w) return fail(TQ_ERR_INVALID, "%s: null matrix descriptor", fn);
  const int n = w->n, k = w->k;
  if (n < 1) return fail(TQ_ERR_INVALID, "%s: n = %d < 1", fn, n);
  if (k <= 0 || k % 256 != 0 || k > kMaxK)
    return fail(TQ_ERR_INVALID, "%s: k = %d must be a positive multiple of 256 <= %d", fn, k, kMaxK);
  if (t < 0 || t > INT32_MAX) return fail(TQ_ERR_INVALID, "%s: t = %lld out of range", fn, (long long)t);
  if (t == 0) return TQ_OK;
  if (!w->codes || !w->scales || !x || !y || !q || !d || !bsum) return fail(TQ_ERR_INVALID, "%s: null pointer", fn);
  if (!aligned(w->codes, 128)) return fail(TQ_ERR_ALIGN, "%s: codes must be 128-byte aligned", fn);
  if (!aligned(x, 16) || !aligned(q, 16) || !aligned(w->scales, 2) || !aligned(d, 4) || !aligned(bsum, 4) ||
      !aligned(y, 4) || (isum_dbg && !aligned(isum_dbg, 4)))
    return fail(TQ_ERR_ALIGN, "%s: x and q must be 16-byte aligned, other buffers naturally aligned", fn);
  const int kb = k / 256;
  if (t > 1 || (int64_t)n * kb * 128 >= ((int64_t)1 << 32)) {
    // several tokens (or a matrix beyond 32-bit offsets): quantize, then the dot pass
    if (events && hipEventRecord((hipEvent_t)events[0], (hipStream_t)stream) != hipSuccess)
      return fail(TQ_ERR_DEVICE, "%s: hipEventRecord failed", fn);
    tq_status st = tq_quantize_act(x, t, k, q, d, bsum, stream);
    if (st != TQ_OK) return st;
    if ((st = tq_gemv(w, q, d, bsum, t, y, isum_dbg, stream)) != TQ_OK) return st;
    if (events && hipEventRecord((hipEvent_t)events[1], (hipStream_t)stream) != hipSuccess)
      return fail(TQ_ERR_DEVICE, "%s: hipEventRecord failed", fn);
    return TQ_OK;
  }
  const int nl = (kb + 7) / 8;
  const int rpw = (n >= 16384 && nl <= 2) ? 4 : 1;
  const unsigned wgs = (unsigned)(((int64_t)n + kGemvXWaves * rpw - 1) / (kGemvXWaves * rpw));
  (void)hipGetLastError();
  if (events)
    hipExtLaunchKernelGGL(pick_gemv_x(kb, rpw), dim3(wgs), dim3(kGemvXWaves * 64), 0, (hipStream_t)stream,
                          (hipEvent_t)events[0], (hipEvent_t)events[1], 0, w->codes, w->scales, n, kb, x, q, d, bsum, y,
                          isum_dbg);
  else
    hipLaunchKernelGGL(pick_gemv_x(kb, rpw), dim3(wgs), dim3(kGemvXWaves * 64), 0, (hipStream_t)stream, w->codes,
                       w->scales, n, kb, x, q, d, bsum, y, isum_dbg);
  return check_launch(fn);
}
}  // namespace tq

extern "C" tq_status tq_gemv_f32(const tq_mat* w, const float* x, int64_t t, float* y, int8_t* q, float* d,
                                 int32_t* bsum, int32_t* isum_dbg, void* stream) {
  tq::clear_error();
  return tq::gemv_f32_run(w, x, t, y, q, d, bsum, isum_dbg, stream, nullptr);
}

extern "C" tq_status tq_gemv_f32_timed(const tq_mat* w, const float* x, int64_t t, float* y, int8_t* q, float* d,
                                       int32_t* bsum, int32_t* isum_dbg, void* stream, void* const* events) {
  tq::clear_error();
  if (!events || !events[0] || !events[1]) return tq::fail(TQ_ERR_INVALID, "tq_gemv_f32_timed: null event");
  return tq::gemv_f32_run(w, x, t, y, q, d, bsum, isum_dbg, stream, events);
}

extern "C" tq_status tq_gemv(const tq_mat* w, const int8_t* q, const float* d, const int32_t* bsum,
                             int64_t t, float* y, int32_t* isum_dbg, void* stream) {
  tq::clear_error();
  return tq::gemv_run(w, q, d, bsum, t, y, isum_dbg, stream, nullptr);
}

extern "C" tq_status tq_gemv_timed(const tq_mat* w, const int8_t* q, const float* d, const int32_t* bsum,
                                   int64_t t, float* y, int32_t* isum_dbg, void* stream, void* const* events) {
  tq::clear_error();
  if (!events || !events[0] || !events[1]) return tq::fail(TQ_ERR_INVALID, "tq_gemv_timed: null event");
  return tq::gemv_run(w, q, d, bsum, t, y, isum_dbg, stream, events);
}
