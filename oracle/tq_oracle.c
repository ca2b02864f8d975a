/*
 * CPU oracle for the tied-trit-plane integer dot pass (Grella, "Tied Trit-Planes",
 * 2026). TEST INFRASTRUCTURE ONLY: this file exists so that tests, the smoke check and
 * the benchmark's CPU-baseline leg can check the HIP path against a plain, slow,
 * obviously correct definition. No product code may link or call it, and it shares no
 * code with the HIP library (no headers, helpers, tables or constants).
 *
 * Arithmetic rules:
 *  - integer work (fold, unfold, block dots) is exact, accumulated in int64;
 *  - the activation quantizer decides integer codes in IEEE fp32 (the precision the
 *    kernels decide them in; the paper fixes none): correctly rounded division and
 *    multiplication, round-half-to-even, no fused multiply-add (build with
 *    -ffp-contract=off);
 *  - the scale combine is evaluated in fp64;
 *  - built with OpenMP, orc_gemv hands whole output rows to threads (nothing else is
 *    parallel, and no row's arithmetic depends on the thread count): the benchmark
 *    times the oracle on one core and on all of them.
 *
 * Pins (tests/oracle_pins.py; every function below has at least one, none re-derives
 * the function's own formula, and tests/test_oracle_mutants.py checks that planted
 * mistakes in each function are caught):
 *   orc_fold/orc_unfold ..... the paper's fold table (golden fixture), bijection onto
 *                             -4..4, round trip, equality with the tied two-plane model
 *   orc_two_plane_dequant ... the paper's level sets for ratios 1, 2, 3, 1/3, -3, 1.7
 *   orc_f16_to_f64/dequant .. numpy's binary16 decode
 *   orc_quantize ............ closed forms (amax 127 -> rne(x), amax 254 -> rne(x/2)),
 *                             amax element -> +-127, error bound, odd symmetry, block
 *                             independence, pure-Python fp32 brute force
 *   orc_dot_i8 .............. exhaustive 9^4 four-element code vectors, bound extremes
 *   orc_gemv ................ trit-plane identity 3(T1.q)+(T2.q), offset form, exact
 *                             integer products at unit scales, power-of-two scaling,
 *                             dequantized-matmul error bound, exact rational brute force
 *   orc_e2m1_to_f64 ......... the OCP table of e2m1 magnitudes (the paper's doubled set
 *                             halved), sign symmetry, monotone magnitudes
 *   orc_e2m1_doubled ........ the paper's doubled set; 2x the float decode, all codes
 *   orc_e8m0_to_f64 ......... numpy's ldexp for every E, NaN at 255
 *   orc_gemv_mx ............. the /2 absorbed exactly (equal to the float-dequantized
 *                             dot in exact rational arithmetic), block-scale exponent
 *                             steps double y exactly, per-32 isum against numpy,
 *                             exact rational brute force
 *   orc_free_quantize ....... planes the best of the nine pairs at the stored scales
 *                             (exhaustive per element), scales the f16 of numpy's least
 *                             squares for the previous planes (one step), error below the
 *                             tied fit's, exact recovery of a tied grid, invariants
 *   orc_gemv2 ............... tied scales (3s, s) reproduce the folded pass (integer
 *                             identity 3(T1.q)+(T2.q)), one empty plane reduces to a
 *                             single ternary plane, plane exchange, sign symmetry,
 *                             dequantized-matmul error bound, exact rational brute force
 *   orc_splitmix64_word ..... SplitMix64's published seed-0 outputs
 *   orc_synth_matrix ........ the written recipe (pure-Python), trit/code/scale
 *                             distributions
 * No function here is "parity unpinned". The activation quantizer's block size, scale
 * rule and rounding are this oracle's reading of a passage that fixes none of them;
 * the pins fix the reading, not the paper.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_OK 0
#define ORC_BAD_INPUT (-1)

/* ------------------------------------------------------------------------------ */
/* Fold and unfold (Sec. 2.1, the tied composite equation; Sec. 2.2).              */
/* With scales tied at alpha = (3s, s), the two trit planes combine into a single    */
/* code c = 3*t1 + t2, which takes the nine values -4..4.                            */
/* ------------------------------------------------------------------------------ */

/* Threads for the row-parallel loops (the benchmark times the oracle on one core and on
   all of them); returns the count now in effect (1 without OpenMP). */
int orc_set_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
  return omp_get_max_threads();
#else
  (void)n;
  return 1;
#endif
}

int orc_fold(const int8_t* t1, const int8_t* t2, int64_t n, int8_t* c) {
  for (int64_t i = 0; i < n; ++i) {
    if (t1[i] < -1 || t1[i] > 1 || t2[i] < -1 || t2[i] > 1) return ORC_BAD_INPUT;
    c[i] = (int8_t)(3 * t1[i] + t2[i]);
  }
  return ORC_OK;
}

/* Inverse of the fold: balanced-ternary digits of c in -4..4.
 * t1 = floor((c + 4) / 3) - 1 and t2 = c - 3*t1. */
int orc_unfold(const int8_t* c, int64_t n, int8_t* t1, int8_t* t2) {
  for (int64_t i = 0; i < n; ++i) {
    int v = c[i];
    if (v < -4 || v > 4) return ORC_BAD_INPUT;
    int a = (v + 4) / 3 - 1; /* v + 4 >= 0, so C division is floor */
    t1[i] = (int8_t)a;
    t2[i] = (int8_t)(v - 3 * a);
  }
  return ORC_OK;
}

/* PTQTP's two-plane reconstruction alpha1*T1 + alpha2*T2 (Sec. 2.1, first
 * paragraph), in fp64, for the free-scale model the tie constrains. */
int orc_two_plane_dequant(const int8_t* t1, const int8_t* t2, int64_t n, double alpha1,
                          double alpha2, double* w) {
  for (int64_t i = 0; i < n; ++i) {
    if (t1[i] < -1 || t1[i] > 1 || t2[i] < -1 || t2[i] > 1) return ORC_BAD_INPUT;
    w[i] = alpha1 * (double)t1[i] + alpha2 * (double)t2[i];
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------------------ */
/* IEEE 754 binary16 decode. The tied scale s is serialized as f16 (Sec. 2.1,     */
/* the scales are stored as f16; Sec. 2.2, four f16 column scales per block).       */
/* 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits.                         */
/* ------------------------------------------------------------------------------ */

double orc_f16_to_f64(uint16_t h) {
  int sign = (h >> 15) & 1;
  int e = (h >> 10) & 0x1F;
  int f = h & 0x3FF;
  double v;
  if (e == 0) {
    v = ldexp((double)f, -24); /* subnormal: f * 2^-14 / 2^10 */
  } else if (e == 31) {
    v = (f == 0) ? INFINITY : NAN;
  } else {
    v = ldexp((double)(1024 + f), e - 25); /* (1 + f/1024) * 2^(e-15) */
  }
  return sign ? -v : v;
}

/* Dequantized tied weight W_hat = s * c (Sec. 2.1), row-major [n][k], one scale per
 * (row, 256-column block). */
int orc_dequant(const int8_t* c, const uint16_t* s, int64_t n, int64_t k, double* w) {
  if (k % 256 != 0) return ORC_BAD_INPUT;
  int64_t kb = k / 256;
  for (int64_t r = 0; r < n; ++r)
    for (int64_t i = 0; i < k; ++i)
      w[r * k + i] = orc_f16_to_f64(s[r * kb + i / 256]) * (double)c[r * k + i];
  return ORC_OK;
}

/* ------------------------------------------------------------------------------ */
/* Block activation quantization (Sec. 2.2: the codes meet activations that were    */
/* quantized block by block). The paper fixes neither block size, scale rule nor     */
/* rounding; the reading implemented here: blocks of 256 along k (the weight block), */
/* symmetric absmax scale d = amax/127, codes q = clamp(rne(x * (127/amax)), +-127)  */
/* in fp32, d kept in fp32, bsum = sum of the block's codes. A block whose amax is    */
/* below 2^-100 (an all-zero block in particular) gives d = 0 and q = 0: below that   */
/* 127/amax would overflow fp32 or amax/127 turn subnormal.                          */
/* ------------------------------------------------------------------------------ */

static int quantize_block(const float* x, int64_t len, int8_t* q, float* d, int32_t* bsum) {
  float amax = 0.0f;
  for (int64_t i = 0; i < len; ++i) {
    if (!isfinite(x[i])) return ORC_BAD_INPUT;
    float a = fabsf(x[i]);
    if (a > amax) amax = a;
  }
  if (amax < 0x1p-100f) {
    for (int64_t i = 0; i < len; ++i) q[i] = 0;
    *d = 0.0f;
    *bsum = 0;
    return ORC_OK;
  }
  float inv = 127.0f / amax;
  *d = amax / 127.0f;
  int32_t s = 0;
  for (int64_t i = 0; i < len; ++i) {
    float y = x[i] * inv;       /* one fp32 multiply, rounded to nearest even */
    float r = rintf(y);         /* round half to even (default rounding mode) */
    if (r > 127.0f) r = 127.0f;
    if (r < -127.0f) r = -127.0f;
    q[i] = (int8_t)r;
    s += (int32_t)r;
  }
  *bsum = s;
  return ORC_OK;
}

/* x [t][k] fp32 -> q [t][k] int8, d [t][k/blk] fp32, bsum [t][k/blk] int32. */
int orc_quantize(const float* x, int64_t t, int64_t k, int64_t blk, int8_t* q, float* d,
                 int32_t* bsum) {
  if (blk <= 0 || k % blk != 0) return ORC_BAD_INPUT;
  int64_t nb = k / blk;
  for (int64_t tt = 0; tt < t; ++tt)
    for (int64_t b = 0; b < nb; ++b) {
      int rc = quantize_block(x + tt * k + b * blk, blk, q + tt * k + b * blk, d + tt * nb + b,
                              bsum + tt * nb + b);
      if (rc != ORC_OK) return rc;
    }
  return ORC_OK;
}

/* ------------------------------------------------------------------------------ */
/* Integer dot (Sec. 2.2: codes dot against the int8 activations with integer SIMD). */
/* ------------------------------------------------------------------------------ */

int64_t orc_dot_i8(const int8_t* a, const int8_t* b, int64_t n) {
  int64_t s = 0;
  for (int64_t i = 0; i < n; ++i) s += (int64_t)a[i] * (int64_t)b[i];
  return s;
}

/* ------------------------------------------------------------------------------ */
/* The serving dot pass (Sec. 2.2): for every token t, output channel r and        */
/* 256-block b, the exact integer block sum isum = sum_i c[r][256b+i] * q[t][256b+i], */
/* then one scale multiply-add per block: y[t][r] = sum_b s[r][b] * d[t][b] * isum.  */
/* Evaluated in fp64 in ascending b; absref[t][r] = sum_b |term| bounds cancellation. */
/* c: logical codes [n][k] in -4..4; s: f16 bits [n][k/256]; q [t][k]; d [t][k/256].  */
/* isum (nullable): [t][n][k/256].                                                    */
/* ------------------------------------------------------------------------------ */

int orc_gemv(const int8_t* c, const uint16_t* s, int64_t n, int64_t k, const int8_t* q,
             const float* d, int64_t t, double* y, double* absref, int32_t* isum) {
  if (k % 256 != 0) return ORC_BAD_INPUT;
  int64_t kb = k / 256;
  int bad = 0;
  /* OpenMP (when built with it) only hands whole output rows to threads: each row's
     integer sums and its fp64 combine run in the same order whatever the thread count. */
#pragma omp parallel for collapse(2) schedule(static) reduction(| : bad)
  for (int64_t tt = 0; tt < t; ++tt)
    for (int64_t r = 0; r < n; ++r) {
      double acc = 0.0, aacc = 0.0;
      for (int64_t b = 0; b < kb; ++b) {
        int64_t v = orc_dot_i8(c + r * k + b * 256, q + tt * k + b * 256, 256);
        if (v > INT32_MAX || v < INT32_MIN) bad = 1;
        if (isum) isum[(tt * n + r) * kb + b] = (int32_t)v;
        double term = orc_f16_to_f64(s[r * kb + b]) * (double)d[tt * kb + b] * (double)v;
        acc += term;
        aacc += fabs(term);
      }
      y[tt * n + r] = acc;
      if (absref) absref[tt * n + r] = aacc;
    }
  return bad ? ORC_BAD_INPUT : ORC_OK;
}

/* ------------------------------------------------------------------------------ */
/* Free-scale two-plane serving pass (Sec. 2.1, first paragraph: W ~ alpha1*T1 +     */
/* alpha2*T2 with two free scales per group; Sec. 4.1, the quality table's note: the  */
/* free pair does not fold, so its serving format keeps the two trit planes apart,    */
/* at 4.125 bits per weight, and the dot takes one integer pass per plane). Groups    */
/* are 256-weight blocks with two f16 scales each (a[r][b][0] = alpha1,               */
/* a[r][b][1] = alpha2: 2 x 16 bits per 256 weights, the 0.125 of 4.125):            */
/*   isum_p[t][r][b] = sum_i Tp[r][256b+i] * q[t][256b+i]   (exact, p = 1, 2),        */
/*   y[t][r] = sum_b d[t][b] * (alpha1[r][b] * isum_1 + alpha2[r][b] * isum_2),       */
/* evaluated in fp64 in ascending b, plane 1's term before plane 2's; absref[t][r] is  */
/* the sum of the terms' magnitudes. isum (nullable): [t][n][k/256][2].               */
/* ------------------------------------------------------------------------------ */

int orc_gemv2(const int8_t* t1, const int8_t* t2, const uint16_t* a, int64_t n, int64_t k,
              const int8_t* q, const float* d, int64_t t, double* y, double* absref, int32_t* isum) {
  if (k % 256 != 0) return ORC_BAD_INPUT;
  int64_t kb = k / 256;
  for (int64_t i = 0; i < n * k; ++i)
    if (t1[i] < -1 || t1[i] > 1 || t2[i] < -1 || t2[i] > 1) return ORC_BAD_INPUT;
  for (int64_t tt = 0; tt < t; ++tt)
    for (int64_t r = 0; r < n; ++r) {
      double acc = 0.0, aacc = 0.0;
      for (int64_t b = 0; b < kb; ++b) {
        const int8_t* qb = q + tt * k + b * 256;
        int64_t v1 = orc_dot_i8(t1 + r * k + b * 256, qb, 256);
        int64_t v2 = orc_dot_i8(t2 + r * k + b * 256, qb, 256);
        if (isum) {
          isum[((tt * n + r) * kb + b) * 2 + 0] = (int32_t)v1;
          isum[((tt * n + r) * kb + b) * 2 + 1] = (int32_t)v2;
        }
        double db = (double)d[tt * kb + b];
        double term1 = orc_f16_to_f64(a[(r * kb + b) * 2 + 0]) * db * (double)v1;
        double term2 = orc_f16_to_f64(a[(r * kb + b) * 2 + 1]) * db * (double)v2;
        acc += term1;
        acc += term2;
        aacc += fabs(term1) + fabs(term2);
      }
      y[tt * n + r] = acc;
      if (absref) absref[tt * n + r] = aacc;
    }
  return ORC_OK;
}

/* ------------------------------------------------------------------------------ */
/* MXFP4 reference arm (Sec. 2.3; Sec. 2.1 for the format: e2m1 (fp4) codes, groups  */
/* of 32 sharing an e8m0 scale). e2m1 is 1 sign bit, 2 exponent bits (bias 1) and 1    */
/* mantissa bit; exponent 0 is subnormal. e8m0 is a biased power of two, 2^(E - 127), */
/* with E = 255 reserved for NaN. The integer arm dots the doubled magnitudes (the     */
/* e2m1 values times 2 are integers) against the int8 activations per 32-element      */
/* block and folds the /2 into the power-of-two scale: 2^(E - 127) / 2 = 2^(E - 128).  */
/* ------------------------------------------------------------------------------ */

/* Value of an e2m1 code (low 4 bits of `code`) from the format definition. */
double orc_e2m1_to_f64(uint8_t code) {
  int sign = (code >> 3) & 1, e = (code >> 1) & 3, m = code & 1;
  double v = (e == 0) ? 0.5 * m : ldexp(1.0 + 0.5 * m, e - 1);
  return sign ? -v : v;
}

/* 2 * value of an e2m1 code, an integer in {0, +-1, +-2, +-3, +-4, +-6, +-8, +-12}. */
int orc_e2m1_doubled(uint8_t code) {
  int sign = (code >> 3) & 1, e = (code >> 1) & 3, m = code & 1;
  int v = (e == 0) ? m : (2 + m) << (e - 1);
  return sign ? -v : v;
}

/* Value of an e8m0 scale: 2^(E - 127); NaN for E = 255. */
double orc_e8m0_to_f64(uint8_t e) { return e == 255 ? NAN : ldexp(1.0, (int)e - 127); }

/* The integer arm's pass: c4 [n][k] e2m1 codes (0..15), e8 [n][k/32] e8m0 scales,
 * q [t][k], d [t][k/256]. For every 32-element block j (within 256-block b = j / 8):
 *   isum[t][r][j] = sum_i doubled(c4[r][32j+i]) * q[t][32j+i]   (exact),
 *   y[t][r] = sum_j 2^(E[r][j] - 128) * d[t][b] * isum[t][r][j]  (fp64, ascending j);
 * absref[t][r] = sum of the terms' magnitudes. isum (nullable): [t][n][k/32]. */
int orc_gemv_mx(const uint8_t* c4, const uint8_t* e8, int64_t n, int64_t k, const int8_t* q,
                const float* d, int64_t t, double* y, double* absref, int32_t* isum) {
  if (k % 256 != 0) return ORC_BAD_INPUT;
  int64_t kb = k / 256, k32 = k / 32;
  for (int64_t i = 0; i < n * k; ++i)
    if (c4[i] > 15) return ORC_BAD_INPUT;
  for (int64_t i = 0; i < n * k32; ++i)
    if (e8[i] == 255) return ORC_BAD_INPUT;
  for (int64_t tt = 0; tt < t; ++tt)
    for (int64_t r = 0; r < n; ++r) {
      double acc = 0.0, aacc = 0.0;
      for (int64_t j = 0; j < k32; ++j) {
        int64_t v = 0;
        for (int i = 0; i < 32; ++i)
          v += (int64_t)orc_e2m1_doubled(c4[r * k + 32 * j + i]) * (int64_t)q[tt * k + 32 * j + i];
        if (isum) isum[(tt * n + r) * k32 + j] = (int32_t)v;
        double term = ldexp(1.0, (int)e8[r * k32 + j] - 128) * (double)d[tt * kb + j / 8] * (double)v;
        acc += term;
        aacc += fabs(term);
      }
      y[tt * n + r] = acc;
      if (absref) absref[tt * n + r] = aacc;
    }
  return ORC_OK;
}

/* ------------------------------------------------------------------------------ */
/* Synthetic weight stream (input generation, not the method): SplitMix64 as a     */
/* counter-based generator (Steele, Lea & Flood 2014), trits by 16-bit multiply-     */
/* shift, scales uniform over the fp16 patterns in [1e-3, 1e-1]. Written here from    */
/* the published definition; the HIP side carries its own implementation.            */
/* ------------------------------------------------------------------------------ */

static uint64_t sm64_word(uint64_t key, uint64_t i) {
  uint64_t z = key + (i + 1) * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

uint64_t orc_splitmix64_word(uint64_t key, uint64_t i) { return sm64_word(key, i); }

static int8_t trit16(uint64_t f) { return (int8_t)((int)((f * 3u) >> 16) - 1); }

/* Trit planes and f16 scales of rows [row0, row0 + rows) of an n x k matrix. */
int orc_synth_matrix(uint64_t key, int64_t n, int64_t k, int64_t row0, int64_t rows,
                     int8_t* t1, int8_t* t2, uint16_t* s) {
  if (k % 256 != 0 || row0 < 0 || row0 + rows > n) return ORC_BAD_INPUT;
  const uint64_t lo = 0x1419, span = 0x2E66 - 0x1419 + 1;
  int64_t kb = k / 256;
  for (int64_t r = 0; r < rows; ++r) {
    for (int64_t col = 0; col < k; ++col) {
      uint64_t e = (uint64_t)((row0 + r) * k + col);
      uint64_t w = sm64_word(key, e >> 1);
      int sh = (e & 1) ? 32 : 0;
      t1[r * k + col] = trit16((w >> sh) & 0xFFFF);
      t2[r * k + col] = trit16((w >> (sh + 16)) & 0xFFFF);
    }
    for (int64_t b = 0; b < kb; ++b) {
      uint64_t j = (uint64_t)((row0 + r) * kb + b);
      uint64_t w = sm64_word(key, (uint64_t)(n * k / 2) + j);
      s[r * kb + b] = (uint16_t)(lo + (((w >> 32) * span) >> 32));
    }
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------------------ */
/* Tied solver (Sec. 2.1, first paragraph): with the plane scales tied at           */
/* alpha = (3s, s), fitting W ~ alpha1*T1 + alpha2*T2 by alternating plane and scale */
/* updates is fitting the uniform nine-level quantizer W_hat = s*c, c in -4..4, per  */
/* group of weights. Groups here are the format's 256-weight blocks (one scale per   */
/* row and 256 columns, Sec. 2.2). The paper gives neither the start, the stopping   */
/* rule nor the precision; the reading implemented (each half-step is the exact      */
/* minimizer of the squared error given the other half):                           */
/*  - amax = max |w|; a block with amax < 2^-100 (all-zero included) gets s = 0, c = 0;*/
/*  - start s = amax / 4 (the largest weight on the outermost level);               */
/*  - code step:  c_i = clamp(rne(fl32(w_i / s)), -4, 4), IEEE fp32 division;        */
/*  - scale step: s = fl32(<w, c> / <c, c>), <c, c> an exact integer, <w, c> summed   */
/*    in fp64 (the products are exact) by pairwise halving: v[i] += v[i + h] for      */
/*    h = 128, 64, ..., 1, so that any implementation following the same order makes  */
/*    the same decisions;                                                            */
/*  - stop when a code step reproduces the previous codes (then the scale step would  */
/*    reproduce s), or after max_iter code steps;                                    */
/*  - the scale is stored as f16 (round to nearest even, saturating at 65504), and   */
/*    the codes are the code step at the stored scale (all zero if it is 0).         */
/* iters[block] = the number of code steps taken (0 for a zero block).                */
/* ------------------------------------------------------------------------------ */

/* fp32 -> binary16, round to nearest even, saturating to the largest finite value,
 * from the format's definition (sign, 5-bit exponent with bias 15, 10-bit fraction;
 * subnormals below 2^-14 in steps of 2^-24). Input finite. */
uint16_t orc_f32_to_f16(float x) {
  uint16_t sign = signbit(x) ? 0x8000 : 0;
  double a = fabs((double)x);
  if (a == 0.0) return sign;
  int e;
  frexp(a, &e); /* a = m * 2^e, 0.5 <= m < 1, so the leading bit has weight 2^(e-1) */
  int ue = e - 1;
  if (ue < -14) ue = -14; /* subnormal range: fixed step 2^-24 */
  double step = ldexp(1.0, ue - 10);
  double q = a / step;           /* exact: a power-of-two division */
  double r = nearbyint(q);       /* round half to even (default rounding mode) */
  double v = r * step;
  if (v > 65504.0) v = 65504.0;  /* saturate (covers rounding up past the top binade) */
  /* encode v (a representable value) */
  if (v < ldexp(1.0, -14)) return (uint16_t)(sign | (uint16_t)(v / ldexp(1.0, -24)));
  frexp(v, &e);
  int be = e - 1 + 15;
  uint16_t frac = (uint16_t)((v / ldexp(1.0, e - 1) - 1.0) * 1024.0);
  return (uint16_t)(sign | (uint16_t)(be << 10) | frac);
}

static double pairwise_sum256(double* v) {
  for (int h = 128; h >= 1; h /= 2)
    for (int i = 0; i < h; ++i) v[i] = v[i] + v[i + h];
  return v[0];
}

static void code_step(const float* w, float s, int8_t* c) {
  for (int i = 0; i < 256; ++i) {
    float t = w[i] / s;
    float r = nearbyintf(t);
    if (r > 4.0f) r = 4.0f;
    if (r < -4.0f) r = -4.0f;
    c[i] = (int8_t)r;
  }
}

int orc_tied_quantize(const float* w, int64_t n, int64_t k, int max_iter, int8_t* c, uint16_t* s16,
                      uint8_t* iters) {
  if (k % 256 != 0 || max_iter < 1 || max_iter > 255) return ORC_BAD_INPUT;
  const int64_t kb = k / 256;
  for (int64_t r = 0; r < n; ++r) {
    for (int64_t b = 0; b < kb; ++b) {
      const float* wb = w + r * k + b * 256;
      int8_t* cb = c + r * k + b * 256;
      float amax = 0.0f;
      for (int i = 0; i < 256; ++i) {
        if (!isfinite(wb[i])) return ORC_BAD_INPUT;
        if (fabsf(wb[i]) > amax) amax = fabsf(wb[i]);
      }
      if (!(amax >= 0x1p-100f)) {
        for (int i = 0; i < 256; ++i) cb[i] = 0;
        s16[r * kb + b] = 0;
        if (iters) iters[r * kb + b] = 0;
        continue;
      }
      float s = amax / 4.0f;
      int8_t prev[256];
      int it = 0;
      for (;;) {
        code_step(wb, s, cb);
        ++it;
        int same = it > 1;
        for (int i = 0; i < 256 && same; ++i) same = cb[i] == prev[i];
        if (same || it == max_iter) break;
        double v[256];
        int64_t cc = 0;
        for (int i = 0; i < 256; ++i) {
          v[i] = (double)wb[i] * (double)cb[i];
          cc += (int64_t)cb[i] * cb[i];
          prev[i] = cb[i];
        }
        if (cc == 0) break; /* not reached from the start above; kept as a guard */
        s = (float)(pairwise_sum256(v) / (double)cc);
      }
      uint16_t h = orc_f32_to_f16(s);
      s16[r * kb + b] = h;
      if (iters) iters[r * kb + b] = (uint8_t)it;
      float sd = (float)orc_f16_to_f64(h);
      if (sd == 0.0f) {
        for (int i = 0; i < 256; ++i) cb[i] = 0;
      } else {
        code_step(wb, sd, cb);
      }
    }
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------------------ */
/* Free-scale solver (Sec. 2.1, first paragraph: PTQTP fits W ~ alpha1*T1 + alpha2*T2 */
/* per group by alternating plane and scale updates with two free scales; the tie     */
/* alpha = (3s, s) is its constrained case, so the free fit is started from the tied  */
/* fit and refines it). The paper gives neither start, stop rule nor precision; the   */
/* reading implemented, per 256-weight block:                                         */
/*  - start: planes = unfold(tied codes), alpha = (3 f(s), f(s)), f(s) the tied f16    */
/*    scale; a zero tied scale gives a zero fit (alpha = 0, planes 0, 0 steps);         */
/*  - scale step: least squares for the two scales given the planes. With            */
/*    a = <T1,T1>, b = <T1,T2>, c = <T2,T2> (exact) and u = <w,T1>, v = <w,T2> (fp64,  */
/*    pairwise halving as in the tied solver), det = a c - b^2; if det > 0,            */
/*    alpha1 = fl32((c u - b v) / det) and alpha2 = fl32((a v - b u) / det), every fp64  */
/*    operation rounded on its own; if det = 0 the scales stay;                        */
/*  - plane step: each weight takes the first pair (t1, t2), in the order 0, -1, +1    */
/*    for t1 and within it for t2, with the least |w - (alpha1 t1 + alpha2 t2)| in fp64;*/
/*  - stop when a plane step reproduces the previous planes, or after max_iter steps;  */
/*  - store alpha1, alpha2 as f16 (nearest even, saturating) and the planes of a plane */
/*    step at the stored scales.                                                       */
/* iters[block] = the plane steps taken before the final one (0 for a zero block).     */
/* ------------------------------------------------------------------------------ */

static const int kFreeOrder[3] = {0, -1, 1};

static void free_plane_step(const float* w, float a1, float a2, int8_t* t1, int8_t* t2) {
  for (int i = 0; i < 256; ++i) {
    double best = INFINITY;
    int b1 = 0, b2 = 0;
    for (int x = 0; x < 3; ++x)
      for (int y = 0; y < 3; ++y) {
        int u1 = kFreeOrder[x], u2 = kFreeOrder[y];
        double e = fabs((double)w[i] - ((double)a1 * u1 + (double)a2 * u2));
        if (e < best) {
          best = e;
          b1 = u1;
          b2 = u2;
        }
      }
    t1[i] = (int8_t)b1;
    t2[i] = (int8_t)b2;
  }
}

int orc_free_quantize(const float* w, int64_t n, int64_t k, int max_iter, const int8_t* c_tied,
                      const uint16_t* s_tied, int8_t* t1, int8_t* t2, uint16_t* a16, uint8_t* iters) {
  if (k % 256 != 0 || max_iter < 1 || max_iter > 255) return ORC_BAD_INPUT;
  const int64_t kb = k / 256;
  for (int64_t r = 0; r < n; ++r)
    for (int64_t b = 0; b < kb; ++b) {
      const float* wb = w + r * k + b * 256;
      int8_t* p1 = t1 + r * k + b * 256;
      int8_t* p2 = t2 + r * k + b * 256;
      uint16_t* ab = a16 + (r * kb + b) * 2;
      for (int i = 0; i < 256; ++i)
        if (!isfinite(wb[i])) return ORC_BAD_INPUT;
      if (orc_unfold(c_tied + r * k + b * 256, 256, p1, p2) != ORC_OK) return ORC_BAD_INPUT;
      const float s = (float)orc_f16_to_f64(s_tied[r * kb + b]);
      if (s == 0.0f) {
        for (int i = 0; i < 256; ++i) p1[i] = p2[i] = 0;
        ab[0] = ab[1] = 0;
        if (iters) iters[r * kb + b] = 0;
        continue;
      }
      float a1 = 3.0f * s, a2 = s;
      int it = 0;
      for (;;) {
        double vu[256], vv[256];
        int64_t sa = 0, sb = 0, sc = 0;
        for (int i = 0; i < 256; ++i) {
          vu[i] = (double)wb[i] * (double)p1[i];
          vv[i] = (double)wb[i] * (double)p2[i];
          sa += p1[i] * p1[i];
          sb += p1[i] * p2[i];
          sc += p2[i] * p2[i];
        }
        const double u = pairwise_sum256(vu), v = pairwise_sum256(vv);
        const int64_t det = sa * sc - sb * sb;
        if (det > 0) {
          const double num1 = (double)sc * u - (double)sb * v;
          const double num2 = (double)sa * v - (double)sb * u;
          a1 = (float)(num1 / (double)det);
          a2 = (float)(num2 / (double)det);
        }
        int8_t q1[256], q2[256];
        free_plane_step(wb, a1, a2, q1, q2);
        ++it;
        int same = 1;
        for (int i = 0; i < 256; ++i) {
          same &= q1[i] == p1[i] && q2[i] == p2[i];
          p1[i] = q1[i];
          p2[i] = q2[i];
        }
        if (same || it == max_iter) break;
      }
      ab[0] = orc_f32_to_f16(a1);
      ab[1] = orc_f32_to_f16(a2);
      if (iters) iters[r * kb + b] = (uint8_t)it;
      free_plane_step(wb, (float)orc_f16_to_f64(ab[0]), (float)orc_f16_to_f64(ab[1]), p1, p2);
    }
  return ORC_OK;
}
