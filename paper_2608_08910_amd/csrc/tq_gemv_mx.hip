// The MXFP4 reference arm's integer pass (Sec. 2.3): e2m1 (fp4) codes whose groups of 32
// share an e8m0 scale (the released expert bytes), dotted against the int8 block-quantized
// activations through the doubled-e2m1 integers {0, 1, 2, 3, 4, 6, 8, 12} (signed), the
// e8m0 scale absorbing the /2: weight = 2^(E - 128) * doubled(code).
//
// Same memory plan as the folded pass: 128 code bytes per 256 weights (eight 16-byte
// blocks of 32), 8 lanes per 256 weights, a wave's 16-byte load covers 1 KB. A lane's
// 16 bytes are exactly one 32-element block, so its integer dot is the block's exact
// sum: no integer butterfly, one fp32 multiply-add by 2^(E - 128) * d per lane and
// block, then one fp32 butterfly over the wave per (row, token) item.
#include <hip/hip_ext.h>

#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

// Doubled e2m1 magnitudes by 3-bit index (exponent, mantissa) and their negatives, as
// byte tables for v_perm (bytes 0..3 in the low word, 4..7 in the high word).
constexpr uint32_t kMxPosLo = 0x03020100u, kMxPosHi = 0x0C080604u;  //  0  1  2  3 |  4  6  8  12
constexpr uint32_t kMxNegLo = 0xFDFEFF00u, kMxNegHi = 0xF4F8FAFCu;  // -0 -1 -2 -3 | -4 -6 -8 -12
// v_perm selectors 8, 10, 9, 11 replicate bit 7 of bytes 1, 5, 3, 7 of {src0, src1}.
constexpr uint32_t kSignSel = 0x0B090A08u;

// Four e2m1 codes as signed doubled integers: magnitude indices in bytes of `idx`
// (0..7), sign bits at bit 7 of the bytes of `sgn`.
__device__ __forceinline__ int mx_dec4(uint32_t idx, uint32_t sgn) {
  const uint32_t pos = __builtin_amdgcn_perm(kMxPosHi, kMxPosLo, idx);
  const uint32_t neg = __builtin_amdgcn_perm(kMxNegHi, kMxNegLo, idx);
  // sgn's bytes 0..3 sit at bytes 1, 5, 3, 7 of {sgn, sgn << 8}: 0xFF where negative
  const uint32_t m = __builtin_amdgcn_perm(sgn, sgn << 8, kSignSel);
  return (int)((neg & m) | (pos & ~m));
}

// The exact sum of doubled codes times activations over one 32-element block: byte i of
// the 16 holds element i (low nibble) and element 16 + i (high nibble), so dword m's low
// nibbles meet activation dword m and its high nibbles activation dword 4 + m.
__device__ __forceinline__ int mx_dot32(const uint4 w, const int (&a)[8]) {
  const uint32_t wv[4] = {w.x, w.y, w.z, w.w};
  int acc = 0;
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const int lo = mx_dec4(wv[m] & 0x07070707u, wv[m] << 4);
    const int hi = mx_dec4((wv[m] >> 4) & 0x07070707u, wv[m]);
    acc = __builtin_amdgcn_sdot4(lo, a[m], acc, false);
    acc = __builtin_amdgcn_sdot4(hi, a[4 + m], acc, false);
  }
  return acc;
}

// LOOP = false: one chunk of at most NT tokens (t <= NT), no token loop.
template <int NL, int NT, int RPW, bool LOOP>
__global__ __launch_bounds__(256) void k_gemv_mx(const uint8_t* __restrict__ codes, const uint8_t* __restrict__ scales,
                                                 int n, int kb, const int8_t* __restrict__ q,
                                                 const float* __restrict__ d, int t, float* __restrict__ y,
                                                 int32_t* __restrict__ isum_dbg) {
  static_assert(RPW <= 8 && (RPW & (RPW - 1)) == 0, "RPW: a power of two <= 8");
  constexpr int NI = RPW * NT;
  using RR = RowReduce<NI, 1>;
  constexpr int KI = RR::KI;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 3, cp = lane & 7;
  const int row0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * RPW;
  if (row0 >= n) return;
  const int64_t k = (int64_t)kb * 256;

  // The activations and block scales of a chunk of NT tokens, the first chunk's requested
  // before the weights (a compute unit returns loads in issue order).
  int qa[NT][NL][8];
  float dt[NT][NL];
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
        dt[tt][i] = d[tc * kb + min(8 * i + g, kb - 1)];  // masked at use
      }
  };
  load_acts(0);

  // Unconditional loads from clamped addresses (rows past n are computed and not
  // stored; blocks past kb get d = 0), buffer loads relative to the wave's first row.
  const int wrow0 = __builtin_amdgcn_readfirstlane(row0);
  const int nrows = min(RPW, n - wrow0);
  const __amdgpu_buffer_rsrc_t cr = make_rsrc(codes + (int64_t)wrow0 * kb * 128, (uint32_t)(nrows * kb * 128));
  uint4 w[RPW][NL];
  int ex[RPW][NL];  // e8m0 exponent of the lane's 32-element block
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    const int rr = min(r, nrows - 1);
#pragma unroll
    for (int i = 0; i < NL; ++i) w[r][i] = buf_load16(cr, (uint32_t)((rr * kb + min(8 * i + g, kb - 1)) * 128 + cp * 16), 0);
  }
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    const int64_t rc = min(row0 + r, n - 1);
#pragma unroll
    for (int i = 0; i < NL; ++i) ex[r][i] = scales[(rc * kb + min(8 * i + g, kb - 1)) * 8 + cp];
  }
  __builtin_amdgcn_sched_barrier(0);  // every load above is issued before any math

  int t0 = 0;  // t >= 1: the launcher returns early for t == 0
  do {
    if (t0 > 0) load_acts(t0);
    float acc[NI];
#pragma unroll
    for (int it = 0; it < NI; ++it) acc[it] = 0.0f;
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int b = 8 * i + g;
#pragma unroll
      for (int r = 0; r < RPW; ++r)
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) {
          const int is = mx_dot32(w[r][i], qa[tt][i]);  // the block's exact sum
          const float dv = (t0 + tt < t && b < kb) ? dt[tt][i] : 0.0f;
          acc[r * NT + tt] = fmaf(ldexpf(dv, ex[r][i] - 128), (float)is, acc[r * NT + tt]);
          if (isum_dbg != nullptr) {
            const int tok = t0 + tt, row = row0 + r;
            if (tok < t && row < n && b < kb) isum_dbg[((int64_t)tok * n + row) * (kb * 8) + b * 8 + cp] = is;
          }
        }
    }
    // fp32 sums over the 64 lanes: lane bits 0..2 (the 8 blocks of 32 in a 256-block),
    // then bits 3..5 (the 256-blocks of a load)
    if constexpr (RR::LI >= 1) bfly_step<NI, 1>(acc);
    if constexpr (RR::LI >= 2) bfly_step<NI / 2, 2>(acc);
    if constexpr (RR::LI >= 3) bfly_step<NI / 4, 4>(acc);
    float kept[KI];
#pragma unroll
    for (int kk = 0; kk < KI; ++kk) {
      float v = acc[kk];
      if constexpr (RR::LI < 1) v = xor_sum<1>(v);
      if constexpr (RR::LI < 2) v = xor_sum<2>(v);
      if constexpr (RR::LI < 3) v = xor_sum<4>(v);
      kept[kk] = v;
    }
    RR::block_totals(kept);
    if (RR::writer(lane)) {
      const int it = RR::item(lane), tok = t0 + it % NT, row = row0 + it / NT;
      if (tok < t && row < n) y[(int64_t)tok * n + row] = kept[0];
    }
    t0 += NT;
  } while (LOOP && t0 < t);
}

using gemv_mx_fn = void (*)(const uint8_t*, const uint8_t*, int, int, const int8_t*, const float*, int, float*,
                            int32_t*);

// Register budget: two or four rows per wave only where a row is at most two loads.
template <int NL>
static gemv_mx_fn pick_gemv_mx_nl(int nt, int rpw) {
  if constexpr (NL <= 2) {
    if (nt == 1) return rpw == 1 ? k_gemv_mx<NL, 1, 1, false> : (rpw == 2 ? k_gemv_mx<NL, 1, 2, false> : k_gemv_mx<NL, 1, 4, false>);
    return rpw == 1 ? k_gemv_mx<NL, 4, 1, true> : k_gemv_mx<NL, 4, 4, true>;
  } else {
    (void)rpw;
    return nt == 1 ? k_gemv_mx<NL, 1, 1, false> : k_gemv_mx<NL, 4, 1, true>;
  }
}

static gemv_mx_fn pick_gemv_mx(int nl, int nt, int rpw) {
  switch (nl) {
    case 1: return pick_gemv_mx_nl<1>(nt, rpw);
    case 2: return pick_gemv_mx_nl<2>(nt, rpw);
    case 3: return pick_gemv_mx_nl<3>(nt, rpw);
    case 4: return pick_gemv_mx_nl<4>(nt, rpw);
    case 5: return pick_gemv_mx_nl<5>(nt, rpw);
    case 6: return pick_gemv_mx_nl<6>(nt, rpw);
    case 7: return pick_gemv_mx_nl<7>(nt, rpw);
    default: return pick_gemv_mx_nl<8>(nt, rpw);
  }
}

// Rows per wave on large matrices for one token (build-time knob; 2 measured best: the
// table decode makes a wave's compute long enough that four rows lengthen the tail).
#ifndef TQ_GEMV_MX_RPW1
#define TQ_GEMV_MX_RPW1 2
#endif

static tq_status gemv_mx_run(const tq_mat_mx* w, const int8_t* q, const float* d, int64_t t, float* y,
                             int32_t* isum_dbg, void* stream, void* const* events) {
  if (!w) return fail(TQ_ERR_INVALID, "tq_gemv_mx: null matrix descriptor");
  const int n = w->n, k = w->k;
  if (n < 1) return fail(TQ_ERR_INVALID, "tq_gemv_mx: n = %d < 1", n);
  if (k <= 0 || k % 256 != 0 || k > kMaxK)
    return fail(TQ_ERR_INVALID, "tq_gemv_mx: k = %d must be a positive multiple of 256 <= %d", k, kMaxK);
  if (t < 0 || t > INT32_MAX) return fail(TQ_ERR_INVALID, "tq_gemv_mx: t = %lld out of range", (long long)t);
  if (t == 0) return TQ_OK;
  if (!w->codes || !w->scales || !q || !d || !y) return fail(TQ_ERR_INVALID, "tq_gemv_mx: null pointer");
  if (!aligned(w->codes, 128)) return fail(TQ_ERR_ALIGN, "tq_gemv_mx: codes must be 128-byte aligned");
  if (!aligned(q, 16) || !aligned(d, 4) || !aligned(y, 4) || (isum_dbg && !aligned(isum_dbg, 4)))
    return fail(TQ_ERR_ALIGN, "tq_gemv_mx: q must be 16-byte aligned, other buffers naturally aligned");
  if ((int64_t)t * n * (k / 32) > ((int64_t)1 << 40)) return fail(TQ_ERR_INVALID, "tq_gemv_mx: problem too large");
  const int kb = k / 256, nl = (kb + 7) / 8;
  const int nt = t == 1 ? 1 : 4;
  const int rpw = (n >= 16384 && nl <= 2) ? (nt == 1 ? TQ_GEMV_MX_RPW1 : 4) : 1;
  const int64_t waves = (n + rpw - 1) / rpw;
  const unsigned wgs = (unsigned)((waves + 3) / 4);
  (void)hipGetLastError();
  if (events)
    hipExtLaunchKernelGGL(pick_gemv_mx(nl, nt, rpw), dim3(wgs), dim3(256), 0, (hipStream_t)stream,
                          (hipEvent_t)events[0], (hipEvent_t)events[1], 0, w->codes, w->scales, n, kb, q, d, (int)t, y,
                          isum_dbg);
  else
    hipLaunchKernelGGL(pick_gemv_mx(nl, nt, rpw), dim3(wgs), dim3(256), 0, (hipStream_t)stream, w->codes, w->scales,
                       n, kb, q, d, (int)t, y, isum_dbg);
  return check_launch("tq_gemv_mx");
}

}  // namespace tq

extern "C" tq_status tq_gemv_mx(const tq_mat_mx* w, const int8_t* q, const float* d, int64_t t, float* y,
                                int32_t* isum_dbg, void* stream) {
  tq::clear_error();
  return tq::gemv_mx_run(w, q, d, t, y, isum_dbg, stream, nullptr);
}

extern "C" tq_status tq_gemv_mx_timed(const tq_mat_mx* w, const int8_t* q, const float* d, int64_t t, float* y,
                                      int32_t* isum_dbg, void* stream, void* const* events) {
  tq::clear_error();
  if (!events || !events[0] || !events[1]) return tq::fail(TQ_ERR_INVALID, "tq_gemv_mx_timed: null event");
  return tq::gemv_mx_run(w, q, d, t, y, isum_dbg, stream, events);
}
