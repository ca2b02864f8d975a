// Persistent-format sizes, and fold + pack / unpack on the host (Sec. 2.1 fold
// c = 3*t1 + t2; Sec. 2.2 the folded code plane is the stored form).
#include <cstring>

#include "tq_internal.hpp"

extern "C" size_t tq_codes_bytes(int32_t n, int32_t k) {
  if (n < 0 || k <= 0 || k % 256 != 0) return 0;
  return (size_t)n * (size_t)k / 2;
}

extern "C" size_t tq_scales_bytes(int32_t n, int32_t k) {
  if (n < 0 || k <= 0 || k % 256 != 0) return 0;
  return (size_t)n * (size_t)(k / 256) * 2;
}

// The names the boundary's specification gives these sizes (same values).
extern "C" size_t tq_packed_codes_bytes(int32_t n, int32_t k) { return tq_codes_bytes(n, k); }
extern "C" size_t tq_packed_scales_bytes(int32_t n, int32_t k) { return tq_scales_bytes(n, k); }

// Pack an already-folded code plane: c [n][k] in -4..4 and f16 scales [n][k/256] (host)
// into the persistent planes (host): the nibbles as in tq_fold_pack_host, the scales
// copied as they are.
extern "C" tq_status tq_pack_host(const int8_t* c, const uint16_t* s_f16, int32_t n, int32_t k, uint8_t* codes_out,
                                  uint16_t* scales_out) {
  using namespace tq;
  clear_error();
  if (n < 0 || k <= 0 || k % 256 != 0)
    return fail(TQ_ERR_INVALID, "tq_pack_host: bad shape n=%d k=%d (k must be a multiple of 256)", n, k);
  if (n == 0) return TQ_OK;
  if (!c || !s_f16 || !codes_out || !scales_out) return fail(TQ_ERR_INVALID, "tq_pack_host: null pointer");
  const int64_t kb = k / 256;
  for (int64_t r = 0; r < n; ++r)
    for (int64_t b = 0; b < kb; ++b) {
      const int64_t col0 = r * k + b * 256;
      uint8_t* blk = codes_out + (r * kb + b) * 128;
      for (int j = 0; j < 8; ++j)
        for (int i = 0; i < 16; ++i) {
          const int64_t lo = col0 + 32 * j + i, hi = lo + 16;
          const int clo = c[lo], chi = c[hi];
          if (clo < -4 || clo > 4 || chi < -4 || chi > 4)
            return fail(TQ_ERR_INVALID, "tq_pack_host: code outside -4..4 near element %lld", (long long)lo);
          blk[16 * j + i] = (uint8_t)((clo & 0xF) | ((chi & 0xF) << 4));
        }
    }
  std::memcpy(scales_out, s_f16, (size_t)n * (size_t)kb * sizeof(uint16_t));
  return TQ_OK;
}

extern "C" tq_status tq_fold_pack_host(const int8_t* t1, const int8_t* t2, int32_t n, int32_t k,
                                       uint8_t* codes_out) {
  using namespace tq;
  clear_error();
  if (n < 0 || k <= 0 || k % 256 != 0)
    return fail(TQ_ERR_INVALID, "tq_fold_pack_host: bad shape n=%d k=%d (k must be a multiple of 256)", n, k);
  if (n == 0) return TQ_OK;
  if (!t1 || !t2 || !codes_out) return fail(TQ_ERR_INVALID, "tq_fold_pack_host: null pointer");
  const int64_t kb = k / 256;
  for (int64_t r = 0; r < n; ++r)
    for (int64_t b = 0; b < kb; ++b) {
      const int64_t col0 = r * k + b * 256;
      uint8_t* blk = codes_out + (r * kb + b) * 128;
      for (int j = 0; j < 8; ++j)
        for (int i = 0; i < 16; ++i) {
          const int64_t lo = col0 + 32 * j + i, hi = lo + 16;
          const int a1 = t1[lo], a2 = t2[lo], b1 = t1[hi], b2 = t2[hi];
          if (a1 < -1 || a1 > 1 || a2 < -1 || a2 > 1 || b1 < -1 || b1 > 1 || b2 < -1 || b2 > 1)
            return fail(TQ_ERR_INVALID, "tq_fold_pack_host: trit out of range near element %lld", (long long)lo);
          const int clo = 3 * a1 + a2, chi = 3 * b1 + b2;  // 4-bit two's complement nibbles
          blk[16 * j + i] = (uint8_t)((clo & 0xF) | ((chi & 0xF) << 4));
        }
    }
  return TQ_OK;
}

extern "C" tq_status tq_unpack_host(const uint8_t* codes, int32_t n, int32_t k, int8_t* c_out) {
  using namespace tq;
  clear_error();
  if (n < 0 || k <= 0 || k % 256 != 0)
    return fail(TQ_ERR_INVALID, "tq_unpack_host: bad shape n=%d k=%d (k must be a multiple of 256)", n, k);
  if (n == 0) return TQ_OK;
  if (!codes || !c_out) return fail(TQ_ERR_INVALID, "tq_unpack_host: null pointer");
  const int64_t kb = k / 256;
  for (int64_t r = 0; r < n; ++r)
    for (int64_t b = 0; b < kb; ++b) {
      const int64_t col0 = r * k + b * 256;
      const uint8_t* blk = codes + (r * kb + b) * 128;
      for (int j = 0; j < 8; ++j)
        for (int i = 0; i < 16; ++i) {
          const int nlo = blk[16 * j + i] & 0xF, nhi = blk[16 * j + i] >> 4;
          const int clo = nlo >= 8 ? nlo - 16 : nlo, chi = nhi >= 8 ? nhi - 16 : nhi;
          if (clo < -4 || clo > 4 || chi < -4 || chi > 4)
            return fail(TQ_ERR_INVALID, "tq_unpack_host: nibble outside -4..4 in block (%lld, %lld)", (long long)r,
                        (long long)b);
          c_out[col0 + 32 * j + i] = (int8_t)clo;
          c_out[col0 + 32 * j + 16 + i] = (int8_t)chi;
        }
    }
  return TQ_OK;
}

// Free-scale two-plane layout (Sec. 2.1 alpha1*T1 + alpha2*T2; Sec. 4.1: the two trit planes
// stored apart, 4.125 bits/weight): block byte 16j + 8p + 4u + b, bit pair 2s, holds
// plane p+1's trit of column 32j + 16u + 4s + b as 2-bit two's complement.
static inline int64_t plane_byte(int j, int p, int u, int b) { return 16 * j + 8 * p + 4 * u + b; }

extern "C" tq_status tq_pack2_host(const int8_t* t1, const int8_t* t2, int32_t n, int32_t k, uint8_t* codes_out) {
  using namespace tq;
  clear_error();
  if (n < 0 || k <= 0 || k % 256 != 0)
    return fail(TQ_ERR_INVALID, "tq_pack2_host: bad shape n=%d k=%d (k must be a multiple of 256)", n, k);
  if (n == 0) return TQ_OK;
  if (!t1 || !t2 || !codes_out) return fail(TQ_ERR_INVALID, "tq_pack2_host: null pointer");
  const int64_t kb = k / 256;
  for (int64_t r = 0; r < n; ++r)
    for (int64_t blk = 0; blk < kb; ++blk) {
      const int64_t col0 = r * k + blk * 256;
      uint8_t* out = codes_out + (r * kb + blk) * 128;
      std::memset(out, 0, 128);
      for (int j = 0; j < 8; ++j)
        for (int u = 0; u < 2; ++u)
          for (int sh = 0; sh < 4; ++sh)
            for (int b = 0; b < 4; ++b) {
              const int64_t col = col0 + 32 * j + 16 * u + 4 * sh + b;
              const int v[2] = {t1[col], t2[col]};
              for (int p = 0; p < 2; ++p) {
                if (v[p] < -1 || v[p] > 1)
                  return fail(TQ_ERR_INVALID, "tq_pack2_host: trit out of range at element %lld", (long long)col);
                out[plane_byte(j, p, u, b)] |= (uint8_t)((v[p] & 3) << (2 * sh));
              }
            }
    }
  return TQ_OK;
}

extern "C" tq_status tq_unpack2_host(const uint8_t* codes, int32_t n, int32_t k, int8_t* t1_out, int8_t* t2_out) {
  using namespace tq;
  clear_error();
  if (n < 0 || k <= 0 || k % 256 != 0)
    return fail(TQ_ERR_INVALID, "tq_unpack2_host: bad shape n=%d k=%d (k must be a multiple of 256)", n, k);
  if (n == 0) return TQ_OK;
  if (!codes || !t1_out || !t2_out) return fail(TQ_ERR_INVALID, "tq_unpack2_host: null pointer");
  const int64_t kb = k / 256;
  int8_t* outs[2] = {t1_out, t2_out};
  for (int64_t r = 0; r < n; ++r)
    for (int64_t blk = 0; blk < kb; ++blk) {
      const int64_t col0 = r * k + blk * 256;
      const uint8_t* in = codes + (r * kb + blk) * 128;
      for (int j = 0; j < 8; ++j)
        for (int u = 0; u < 2; ++u)
          for (int sh = 0; sh < 4; ++sh)
            for (int b = 0; b < 4; ++b)
              for (int p = 0; p < 2; ++p) {
                const int f = (in[plane_byte(j, p, u, b)] >> (2 * sh)) & 3;
                if (f == 2)
                  return fail(TQ_ERR_INVALID, "tq_unpack2_host: invalid trit pattern in block (%lld, %lld)",
                              (long long)r, (long long)blk);
                outs[p][col0 + 32 * j + 16 * u + 4 * sh + b] = (int8_t)(f == 3 ? -1 : f);
              }
    }
  return TQ_OK;
}

// MXFP4 arm (Sec. 2.3): e2m1 codes, two per byte in the order of a released 32-element
// block (element i low nibble, element 16 + i high nibble of byte i).
extern "C" tq_status tq_mx_pack_host(const uint8_t* c4, int32_t n, int32_t k, uint8_t* codes_out) {
  using namespace tq;
  clear_error();
  if (n < 0 || k <= 0 || k % 256 != 0)
    return fail(TQ_ERR_INVALID, "tq_mx_pack_host: bad shape n=%d k=%d (k must be a multiple of 256)", n, k);
  if (n == 0) return TQ_OK;
  if (!c4 || !codes_out) return fail(TQ_ERR_INVALID, "tq_mx_pack_host: null pointer");
  const int64_t nblk = (int64_t)n * (k / 32);
  for (int64_t j = 0; j < nblk; ++j)
    for (int i = 0; i < 16; ++i) {
      const uint8_t lo = c4[32 * j + i], hi = c4[32 * j + 16 + i];
      if (lo > 15 || hi > 15)
        return fail(TQ_ERR_INVALID, "tq_mx_pack_host: code above 15 in block %lld", (long long)j);
      codes_out[16 * j + i] = (uint8_t)(lo | (hi << 4));
    }
  return TQ_OK;
}

extern "C" tq_status tq_mx_unpack_host(const uint8_t* codes, int32_t n, int32_t k, uint8_t* c4_out) {
  using namespace tq;
  clear_error();
  if (n < 0 || k <= 0 || k % 256 != 0)
    return fail(TQ_ERR_INVALID, "tq_mx_unpack_host: bad shape n=%d k=%d (k must be a multiple of 256)", n, k);
  if (n == 0) return TQ_OK;
  if (!codes || !c4_out) return fail(TQ_ERR_INVALID, "tq_mx_unpack_host: null pointer");
  const int64_t nblk = (int64_t)n * (k / 32);
  for (int64_t j = 0; j < nblk; ++j)
    for (int i = 0; i < 16; ++i) {
      c4_out[32 * j + i] = codes[16 * j + i] & 0xF;
      c4_out[32 * j + 16 + i] = codes[16 * j + i] >> 4;
    }
  return TQ_OK;
}
