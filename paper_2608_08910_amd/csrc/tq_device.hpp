// Device-side building blocks of the tied-trit-plane dot pass on gfx950 (CDNA4, wave64).
//
// Lane geometry shared by every kernel here: a 256-weight block is 128 bytes of
// nibble codes = 8 chunks of 16 bytes, and 8 consecutive lanes ("a group") cover one
// block, lane (l & 7) holding chunk (l & 7). A wave's 16-byte load therefore covers 8
// consecutive blocks (1 KB, fully coalesced). Chunk j's 16 bytes unpack to 32 int8
// codes: low nibbles are columns 32j..32j+15, high nibbles columns 32j+16..32j+31, so
// the matching activations are 32 contiguous int8 bytes.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tq {

// DPP control words (GCN/CDNA encoding of the dpp_ctrl field).
constexpr int kDppXor1 = 0xb1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4e;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // lane i <- lane 7-i within each 8-lane half row
constexpr int kDppRowRor8 = 0x128;    // lane i <- lane (i+8) mod 16 within each 16-lane row
// ds_swizzle bit-mode offset: lane ^ 16 within each 32-lane half (and 0x1f, xor 0x10).
constexpr int kSwizzleXor16 = 0x401f;

// Sum over the 8 lanes of a group; every lane of the group receives the sum.
__device__ __forceinline__ int group_sum_i32(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, kDppXor1, 0xf, 0xf, false);
  v += __builtin_amdgcn_update_dpp(0, v, kDppXor2, 0xf, 0xf, false);
  v += __builtin_amdgcn_update_dpp(0, v, kDppHalfMirror, 0xf, 0xf, false);
  return v;
}

__device__ __forceinline__ float group_max_f32(float v) {
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), kDppXor1, 0xf, 0xf, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), kDppXor2, 0xf, 0xf, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), kDppHalfMirror, 0xf, 0xf, false)));
  return v;
}

__device__ __forceinline__ float f16_bits_to_f32(uint16_t h) {
  return __half2float(__ushort_as_half(h));
}

// Codes are 4-bit two's-complement nibbles (c & 15). Keeping a byte's high nibble in
// place, or moving its low nibble up, leaves 16*c as a signed byte: the codes of a
// 16-byte chunk become 32 int8 values 16c in two bitwise operations per half, ready for
// the signed 4-way byte dot, and the dot's sum is exactly 16 times the code dot.
constexpr uint32_t kHiNibbles = 0xF0F0F0F0u;

__device__ __forceinline__ int lo16c(uint32_t w) { return int((w << 4) & kHiNibbles); }
__device__ __forceinline__ int hi16c(uint32_t w) { return int(w & kHiNibbles); }

// The 32 codes of one chunk as 16c bytes, in the order of the activation dwords:
// c[m] = columns 4m..4m+3 (low nibbles of bytes 4m..4m+3), c[4+m] = columns 16+4m..
__device__ __forceinline__ void unpack16c(const uint4 w, int (&c)[8]) {
  c[0] = lo16c(w.x); c[1] = lo16c(w.y); c[2] = lo16c(w.z); c[3] = lo16c(w.w);
  c[4] = hi16c(w.x); c[5] = hi16c(w.y); c[6] = hi16c(w.z); c[7] = hi16c(w.w);
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// 16-byte streaming load (nontemporal: expert weights are read once per step).
__device__ __forceinline__ uint4 ldg16(const void* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ uint4 ld16(const void* p) { return *reinterpret_cast<const uint4*>(p); }

// Buffer resources: a wave-uniform base (SGPRs) plus a 32-bit per-lane offset and a
// wave-uniform offset, so no per-lane 64-bit address arithmetic; reads past num_records
// bytes return zero. Word 3 is the raw-buffer configuration of the gfx9 family.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// Cache-policy bits of buffer loads: nt (streamed once).
constexpr int kBufNT = 2;

// soff must be wave-uniform (an SGPR operand); per-lane offsets go in voff.
__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, int aux = kBufNT) {
  const u32x4 v = aux == kBufNT ? __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, kBufNT)
                                : __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// soff must be wave-uniform (an SGPR operand); per-lane offsets go in voff.
__device__ __forceinline__ uint16_t buf_load_u16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, 0);
}

// Block quantizer on a group: each of the 8 lanes holds 32 consecutive values of one
// 256-block (lane (l & 7) holds columns 32*(l&7) ..). Produces the lane's 32 int8 codes
// packed into 8 dwords, the sum of those 32 codes (qs), and the block's fp32 scale d
// and code sum bsum (group-uniform).
// Rule: amax = max|x| (exact), d = amax/127 and inv = 127/amax (IEEE division, correctly
// rounded: this library is built without fast-math), q = rne(x * inv) with the multiply
// rounded on its own; amax < 2^-100 (all-zero blocks included) gives d = 0, q = 0.
// rne(y) for |y| <= 127.0001 (true here: |x| <= amax) is taken by adding 1.5 * 2^23: the
// sum lies in [2^23, 2^24), where the fp32 spacing is 1, so the add rounds y to the
// nearest integer with ties to even, and the low byte of the sum's bit pattern is that
// integer in two's complement. |y| <= 127.0001 also makes a clamp to +-127 unnecessary.
__device__ __forceinline__ void quantize_group32(const float (&x)[32], int (&qw)[8], int& qs, float& d, int& bsum) {
#pragma clang fp contract(off)  // x * inv and + 1.5 * 2^23 must round separately
  float a = 0.0f;
#pragma unroll
  for (int i = 0; i < 32; ++i) a = fmaxf(a, fabsf(x[i]));
  const float amax = group_max_f32(a);
  if (amax < 0x1p-100f) {
#pragma unroll
    for (int m = 0; m < 8; ++m) qw[m] = 0;
    qs = 0;
    d = 0.0f;
    bsum = 0;
    return;
  }
  const float inv = 127.0f / amax;
  d = amax / 127.0f;
  constexpr float kMagic = 12582912.0f;  // 1.5 * 2^23
  int s = 0;
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    uint32_t b[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const float y = x[4 * m + k] * inv;
      b[k] = __float_as_uint(y + kMagic);
    }
    // low bytes of the four sums -> one dword of int8 codes
    const uint32_t lo01 = __builtin_amdgcn_perm(b[1], b[0], 0x0c0c0400u);
    const uint32_t lo23 = __builtin_amdgcn_perm(b[3], b[2], 0x04000c0cu);
    qw[m] = int(lo01 | lo23);
    s = __builtin_amdgcn_sdot4(qw[m], 0x01010101, s, false);
  }
  qs = s;
  bsum = group_sum_i32(s);
}

// Quantize 256-block `blk` of src into LDS (one block per 8-lane group): codes, the
// block scale and code sum. `store` is group-uniform; the quantization itself runs
// regardless, so that the loads of v are not sunk into a branch behind the weight loads.
__device__ __forceinline__ void quantize_to_lds(const float (&v)[32], int blk, int cp, int8_t* s_q, float* s_d,
                                                int* s_b, bool store) {
  int qw[8], qs, bs;
  float dd;
  quantize_group32(v, qw, qs, dd, bs);
  if (!store) return;
  int4* qp = reinterpret_cast<int4*>(s_q + blk * 256 + cp * 32);
  qp[0] = make_int4(qw[0], qw[1], qw[2], qw[3]);
  qp[1] = make_int4(qw[4], qw[5], qw[6], qw[7]);
  if (cp == 0) {
    s_d[blk] = dd;
    s_b[blk] = bs;
  }
}

// The lane's 32 fp32 values of 256-block `blk` of a row-major fp32 buffer (AUX: cache
// policy of the loads).
template <int AUX = 0>
__device__ __forceinline__ void buf_load32f(__amdgpu_buffer_rsrc_t r, uint32_t blk, int cp, float (&v)[32]) {
  const uint32_t o = (blk * 256u + (uint32_t)cp * 32u) * 4u;
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    const u32x4 w = __builtin_amdgcn_raw_buffer_load_b128(r, o + 16u * m, 0, AUX);
    const uint4 u = make_uint4(w.x, w.y, w.z, w.w);
    v[4 * m + 0] = __uint_as_float(u.x);
    v[4 * m + 1] = __uint_as_float(u.y);
    v[4 * m + 2] = __uint_as_float(u.z);
    v[4 * m + 3] = __uint_as_float(u.w);
  }
}

// ---------------------------------------------------------------------------------
// Cross-lane reductions of many values at once (a butterfly: each exchange step halves
// the number of values a lane carries and pairs lanes whose index differs in one bit).
// ---------------------------------------------------------------------------------

constexpr int clog2(int n) { return n <= 1 ? 0 : 1 + clog2(n >> 1); }

// The low L bits of x in reverse order (L <= 5).
template <int L>
__device__ __forceinline__ int rev_bits(int x) {
  if constexpr (L == 0) return 0;
  else return (int)(__builtin_bitreverse32((unsigned)x) >> (32 - L));
}

// The value of lane (lane ^ M).
template <int M>
__device__ __forceinline__ int lane_xor_i(int v) {
  if constexpr (M == 1) return __builtin_amdgcn_update_dpp(0, v, kDppXor1, 0xf, 0xf, false);
  else if constexpr (M == 2) return __builtin_amdgcn_update_dpp(0, v, kDppXor2, 0xf, 0xf, false);
  else if constexpr (M == 4) return __builtin_amdgcn_ds_swizzle(v, 0x101f);  // bit mode, xor 4
  else if constexpr (M == 8) return __builtin_amdgcn_update_dpp(0, v, kDppRowRor8, 0xf, 0xf, false);
  else if constexpr (M == 16) return __builtin_amdgcn_ds_swizzle(v, kSwizzleXor16);
  else return __builtin_amdgcn_ds_bpermute((int)((__lane_id() ^ 32) << 2), v);
}

template <int M>
__device__ __forceinline__ float lane_xor(float v) { return __int_as_float(lane_xor_i<M>(__float_as_int(v))); }

template <int M>
__device__ __forceinline__ int lane_xchg(int v) { return lane_xor_i<M>(v); }
template <int M>
__device__ __forceinline__ float lane_xchg(float v) { return lane_xor<M>(v); }

// v[0 .. N2) -> v[0 .. N2/2): a lane whose index has bit M set keeps the upper half of
// the values, the others the lower half, each adding its partner's (lane ^ M) copy.
template <int N2, int M, typename T, int SZ>
__device__ __forceinline__ void bfly_step(T (&v)[SZ]) {
  static_assert(N2 <= SZ && N2 % 2 == 0, "bad butterfly step");
  const bool up = (__lane_id() & M) != 0;
#pragma unroll
  for (int k = 0; k < N2 / 2; ++k) {
    const T keep = up ? v[k + N2 / 2] : v[k];
    const T send = up ? v[k] : v[k + N2 / 2];
    v[k] = keep + lane_xchg<M>(send);
  }
}

template <int M>
__device__ __forceinline__ float xor_sum(float v) { return v + lane_xor<M>(v); }

// Row totals of a wave's dot products in the order of operations of the serving pass:
// exact integer block sums, one fp32 multiply-add per block, then the sum over blocks.
//
// A wave computes NI items (row x token pairs, a power of two), each for NM matrices
// that share the item (gate and up). For load i a lane holds the integer partials
// p[item * NM + m] of its 32 codes of block 8i + (lane >> 3); the 8 lanes of that block
// differ in lane bits 0..2.
//  block_sums (exact, once per load): a butterfly over lane bits 0..2 (LI halving
//    steps, then plain sums over the bits left) leaves each lane KI = NI >> LI items,
//    item = k + KI * rev(lane bits 0..LI-1), as whole-block sums.
//  The caller then scales each kept block sum: acc[k * NM + m] += f32(s) * d * isum.
//  block_totals (fp32, once per row): a butterfly over lane bits 3..5 (the 8 blocks of
//    a load; LF halving steps, then plain sums) leaves one item per lane:
//    item() = rev(lane bits 3..3+LF-1) + KI * rev(lane bits 0..LI-1).
// Every lane of a wave ends up with a total; writer() picks one lane per item.
template <int NI, int NM>
struct RowReduce {
  static_assert(NI >= 1 && NI <= 64 && (NI & (NI - 1)) == 0, "items: a power of two <= 64");
  static constexpr int LI = clog2(NI) < 3 ? clog2(NI) : 3;
  static constexpr int KI = NI >> LI;
  static constexpr int LF = clog2(KI);
  static constexpr int NV = NI * NM;

  // kept item k after block_sums
  __device__ static __forceinline__ int kept(int k, int lane) { return k + KI * rev_bits<LI>(lane & ((1 << LI) - 1)); }
  // the item a lane holds after block_totals
  __device__ static __forceinline__ int item(int lane) {
    return rev_bits<LF>((lane >> 3) & ((1 << LF) - 1)) + KI * rev_bits<LI>(lane & ((1 << LI) - 1));
  }
  __device__ static __forceinline__ bool writer(int lane) { return ((lane & 7) >> LI) == 0 && ((lane >> 3) >> LF) == 0; }
  // a lane that holds kept items (one lane per group of identical copies)
  __device__ static __forceinline__ bool block_writer(int lane) { return ((lane & 7) >> LI) == 0; }

  __device__ static __forceinline__ void block_sums(int (&v)[NV]) {
    if constexpr (LI >= 1) bfly_step<NV, 1>(v);
    if constexpr (LI >= 2) bfly_step<NV / 2, 2>(v);
    if constexpr (LI >= 3) bfly_step<NV / 4, 4>(v);
#pragma unroll
    for (int k = 0; k < KI * NM; ++k) {
      if constexpr (LI < 1) v[k] += lane_xor_i<1>(v[k]);
      if constexpr (LI < 2) v[k] += lane_xor_i<2>(v[k]);
      if constexpr (LI < 3) v[k] += lane_xor_i<4>(v[k]);
    }
  }

  __device__ static __forceinline__ void block_totals(float (&a)[KI * NM]) {
    if constexpr (LF >= 1) bfly_step<KI * NM, 8>(a);
    if constexpr (LF >= 2) bfly_step<KI * NM / 2, 16>(a);
    if constexpr (LF >= 3) bfly_step<KI * NM / 4, 32>(a);
#pragma unroll
    for (int m = 0; m < NM; ++m) {
      if constexpr (LF < 1) a[m] = xor_sum<8>(a[m]);
      if constexpr (LF < 2) a[m] = xor_sum<16>(a[m]);
      if constexpr (LF < 3) a[m] = xor_sum<32>(a[m]);
    }
  }
};

// Integer partials of one 16-byte chunk (32 codes, unpacked as 16c bytes) against 32
// int8 activations: sum (16c) * q, an exact multiple of 16 (|.| <= 32 * 64 * 127; a whole
// block's sum stays below 2^21, and >> 4 of it is the exact block sum of c * q).
__device__ __forceinline__ int dot32x16(const int (&c)[8], const int (&a)[8]) {
  int acc = 0;
#pragma unroll
  for (int m = 0; m < 8; ++m) acc = __builtin_amdgcn_sdot4(c[m], a[m], acc, false);
  return acc;
}

}  // namespace tq
