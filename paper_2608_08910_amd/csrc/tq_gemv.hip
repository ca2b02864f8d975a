// The serving dot pass for one tq matrix (Sec. 2.2): exact int32 block sums of the
// folded codes against int8 block-quantized activations, then one fp32 multiply-add
// per block.
//
// Decode is HBM-bound (0.5 byte of codes per weight, a few integer ops per weight per
// token), so the kernel is shaped for the memory system: each wave owns RPW whole
// rows, issues all of their 16-byte code loads up front (a wave load = 8 consecutive
// blocks = 1 KB, fully coalesced), and keeps them in registers while it walks the
// tokens NT at a time. A lane always covers the same columns of every row it owns
// (block 8i + l/8, chunk l & 7 for load i), so its activations sit in registers too,
// loaded once per token chunk. The 8 lanes of a block reduce their partial dots with 3
// DPP adds (exact int32), subtract 4*bsum (codes are stored as u = c + 4), multiply by
// f32(s)*d, and the row total is one DPP/swizzle/readlane reduction.
#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

template <int NL, int NT, int RPW>
__global__ __launch_bounds__(256) void k_gemv(const uint8_t* __restrict__ codes,
                                              const uint16_t* __restrict__ scales, int n, int kb,
                                              const int8_t* __restrict__ q, const float* __restrict__ d,
                                              const int32_t* __restrict__ bsum, int t,
                                              float* __restrict__ y, int32_t* __restrict__ isum_dbg) {
  const int lane = threadIdx.x & 63;
  const int g = lane >> 3, cp = lane & 7;
  const int row0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * RPW;
  if (row0 >= n) return;
  const int64_t k = (int64_t)kb * 256;

  // Loads are unconditional from clamped addresses; invalid lanes are zeroed by a select
  // (a predicated load becomes a branch that serializes the loads).
  uint4 w[RPW][NL];
  float s[RPW][NL];
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    const int64_t rc = min(row0 + r, n - 1);
    const uint8_t* rowcodes = codes + rc * kb * 128;
    const uint16_t* rowscales = scales + rc * kb;
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int b = 8 * i + g;
      const bool ok = b < kb && row0 + r < n;
      const int bc = b < kb ? b : kb - 1;
      const uint4 raw = ldg16(rowcodes + bc * 128 + cp * 16);
      const float sv = f16_bits_to_f32(rowscales[bc]);
      w[r][i] = ok ? raw : make_uint4(0, 0, 0, 0);
      s[r][i] = ok ? sv : 0.0f;
    }
  }

  for (int t0 = 0; t0 < t; t0 += NT) {
    int qa[NT][NL][8];
    float dd[NT][NL];
    int bb[NT][NL];
#pragma unroll
    for (int tt = 0; tt < NT; ++tt)
#pragma unroll
      for (int i = 0; i < NL; ++i) {
        const int tok = t0 + tt, b = 8 * i + g;
        const bool ok = tok < t && b < kb;
        const int64_t tc = min(tok, t - 1);
        const int bc = b < kb ? b : kb - 1;
        const int4* p = reinterpret_cast<const int4*>(q + tc * k + bc * 256 + cp * 32);
        const int4 lo = p[0], hi = p[1];
        const float dv = d[tc * kb + bc];
        const int bv = bsum[tc * kb + bc];
        qa[tt][i][0] = ok ? lo.x : 0; qa[tt][i][1] = ok ? lo.y : 0; qa[tt][i][2] = ok ? lo.z : 0;
        qa[tt][i][3] = ok ? lo.w : 0; qa[tt][i][4] = ok ? hi.x : 0; qa[tt][i][5] = ok ? hi.y : 0;
        qa[tt][i][6] = ok ? hi.z : 0; qa[tt][i][7] = ok ? hi.w : 0;
        dd[tt][i] = ok ? dv : 0.0f;
        bb[tt][i] = ok ? bv : 0;
      }
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      const int row = row0 + r;
#pragma unroll
      for (int tt = 0; tt < NT; ++tt) {
        const int tok = t0 + tt;
        float acc = 0.0f;
#pragma unroll
        for (int i = 0; i < NL; ++i) {
          const int is = group_sum_i32(dot_chunk_u(w[r][i], qa[tt][i])) - 4 * bb[tt][i];
          if (isum_dbg != nullptr && cp == 0 && tok < t && row < n && 8 * i + g < kb)
            isum_dbg[((int64_t)tok * n + row) * kb + 8 * i + g] = is;
          acc = fmaf(s[r][i] * dd[tt][i], (float)is, acc);
        }
        const float tot = wave_sum_groups_f32(acc);
        if (lane == 0 && tok < t && row < n) y[(int64_t)tok * n + row] = tot;
      }
    }
  }
}

using gemv_fn = void (*)(const uint8_t*, const uint16_t*, int, int, const int8_t*, const float*,
                         const int32_t*, int, float*, int32_t*);

template <int NL>
static gemv_fn pick_gemv_nl(int nt, int rpw) {
  if (nt == 1) return rpw == 1 ? k_gemv<NL, 1, 1> : k_gemv<NL, 1, 4>;
  return rpw == 1 ? k_gemv<NL, 4, 1> : k_gemv<NL, 4, 4>;
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

extern "C" tq_status tq_gemv(const tq_mat* w, const int8_t* q, const float* d, const int32_t* bsum,
                             int64_t t, float* y, int32_t* isum_dbg, void* stream) {
  using namespace tq;
  clear_error();
  if (!w) return fail(TQ_ERR_INVALID, "tq_gemv: null matrix descriptor");
  const int n = w->n, k = w->k;
  if (n < 1) return fail(TQ_ERR_INVALID, "tq_gemv: n = %d < 1", n);
  if (k <= 0 || k % 256 != 0 || k > kMaxK)
    return fail(TQ_ERR_INVALID, "tq_gemv: k = %d must be a positive multiple of 256 <= %d", k, kMaxK);
  if (t < 0 || t > INT32_MAX) return fail(TQ_ERR_INVALID, "tq_gemv: t = %lld out of range", (long long)t);
  if (t == 0) return TQ_OK;
  if (!w->codes || !w->scales || !q || !d || !bsum || !y) return fail(TQ_ERR_INVALID, "tq_gemv: null pointer");
  if (!aligned(w->codes, 128)) return fail(TQ_ERR_ALIGN, "tq_gemv: codes must be 128-byte aligned");
  if (!aligned(q, 16) || !aligned(w->scales, 2) || !aligned(d, 4) || !aligned(bsum, 4) || !aligned(y, 4) ||
      (isum_dbg && !aligned(isum_dbg, 4)))
    return fail(TQ_ERR_ALIGN, "tq_gemv: q must be 16-byte aligned, other buffers naturally aligned");
  if ((int64_t)t * n * (k / 256) > ((int64_t)1 << 40)) return fail(TQ_ERR_INVALID, "tq_gemv: problem too large");
  const int kb = k / 256, nl = (kb + 7) / 8;
  const int nt = t == 1 ? 1 : 4;
  // Few rows: one row per wave, to spread a small matrix over all CUs.
  const int rpw = (n >= 16384 && nl <= 2) ? 4 : 1;
  const int64_t waves = (n + rpw - 1) / rpw;
  const unsigned wgs = (unsigned)((waves + 3) / 4);
  (void)hipGetLastError();
  hipLaunchKernelGGL(pick_gemv(nl, nt, rpw), dim3(wgs), dim3(256), 0, (hipStream_t)stream, w->codes, w->scales, n,
                     kb, q, d, bsum, (int)t, y, isum_dbg);
  return check_launch("tq_gemv");
}
