/*
 * tq.h - C ABI of the MI355X (gfx950) tied-trit-plane expert dot pass.
 *
 * The method (M. Grella, "Tied Trit-Planes", 2026):
 *  - Sec. 2.1: with the two PTQTP plane scales tied at alpha = (3s, s), the trit planes
 *    T1, T2 in {-1,0,1} fold into one code c = 3*t1 + t2 in {-4,...,4}; W_hat = s*c with
 *    one f16 scale s per group.
 *  - Sec. 2.2: the folded code plane is the persistent serving representation (4.0625
 *    bits/weight: 4-bit codes plus one f16 scale per 256 weights of an output channel).
 *    A matrix-vector product reads those bytes once: each nibble becomes an integer in
 *    -4..4 with two bitwise operations (no lookup), 256 of them meet int8 activations
 *    (one fp32 scale per 256 inputs) in an exact integer sum, and that sum enters the
 *    fp32 result through a single fused multiply-add with the two scales.
 *
 * Persistent layout of one matrix with n output channels (rows) and k inputs
 * (k % 256 == 0, kb = k/256 blocks per row):
 *   codes  [n][kb][128] bytes, 128-byte aligned. Block (r, b) holds the 256 codes of
 *          row r, columns 256b .. 256b+255, as 4-bit two's-complement nibbles c & 15
 *          (c = 0..4 -> 0..4, c = -4..-1 -> 12..15; 5..11 never occur). Byte 16j + i
 *          (j = 0..7, i = 0..15) holds column 256b + 32j + i in its low nibble and column
 *          256b + 32j + 16 + i in its high nibble, so that the 16 bytes of chunk j unpack
 *          to 32 int8 codes whose activations are 32 contiguous bytes. The sign sits in
 *          each nibble's top bit: masking a byte's high nibble in place (b & 0xF0), or
 *          shifting its low nibble up ((b << 4) & 0xF0), gives 16*c as a signed byte, so
 *          the codes decode by two bitwise operations with no offset to correct.
 *   scales [n][kb] IEEE binary16 bit patterns (s of row r, block b).
 *   Bytes: 128 + 2 per 256 weights = 4.0625 bits/weight, the paper's figure.
 * Quantized activations of t tokens over k inputs:
 *   q [t][k] int8 (-127..127), d [t][kb] fp32 block scale, bsum [t][kb] int32 = sum of the
 *   block's q. The codes and d are this library's reading of the block-wise activation
 *   quantization of Sec. 2.2 (which fixes no rule): blocks of 256, amax = max|x| over the block,
 *   d = amax/127 and q = rne(x * (127/amax)) in IEEE fp32 (correctly rounded division,
 *   round half to even); a block with amax < 2^-100 (an all-zero block in particular) has
 *   d = 0 and q = 0.
 * Block integer sum and combine (Sec. 2.2):
 *   isum[t][r][b] = sum_i c[r][256b+i] * q[t][256b+i] (exact int32; computed as
 *   (sum (16c)*q) >> 4), y[t][r] = sum_b f32(s[r][b]) * d[t][b] * isum[t][r][b] in fp32
 *   (block order unspecified).
 *
 * Conventions for every entry point:
 *  - Pointers are device pointers unless marked "host". The caller owns every buffer; the
 *    library allocates and frees no memory and never synchronizes a stream, except
 *    tq_moe_status, which synchronizes the stream it is given.
 *  - Device work is enqueued on the caller's HIP stream, passed as `void* stream`
 *    (a hipStream_t; NULL means the default stream). Calls are asynchronous.
 *  - Arguments are validated on the host before any launch. A failed check returns a
 *    negative status with no side effects; tq_last_error() then describes it (the
 *    message is thread-local and valid until the calling thread's next call).
 *  - TQ_ERR_DEVICE reports a launch failure (the HIP error string is in tq_last_error).
 *  - Preconditions not checked (documented): activations are finite; codes hold only
 *    the nibbles of -4..4; buffers are at least as large as their stated shapes.
 *  - Thread-safe: no state besides the thread-local error message.
 */
#ifndef TQ_H_
#define TQ_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t tq_status;
#define TQ_OK 0
#define TQ_ERR_INVALID (-1)   /* bad shape, null pointer or out-of-range argument */
#define TQ_ERR_ALIGN (-2)     /* a pointer misses its required alignment */
#define TQ_ERR_WORKSPACE (-3) /* workspace smaller than tq_moe_workspace_bytes */
#define TQ_ERR_DEVICE (-4)    /* a HIP launch or runtime call failed */

#define TQ_BLOCK 256       /* weights (and activations) per block */
#define TQ_BLOCK_BYTES 128 /* packed code bytes per block */

/* One tq matrix in the persistent layout above. codes: 128-byte aligned; scales:
 * 2-byte aligned. n >= 1; 256 <= k <= 16384, k % 256 == 0. */
typedef struct {
  int32_t n;
  int32_t k;
  const uint8_t* codes;
  const uint16_t* scales;
} tq_mat;

/* The routed experts of one MoE layer. Expert e's gate and up matrices are
 * [inter][hidden] and its down matrix [hidden][inter], each in the persistent layout,
 * at gate_codes + e * stride_codes[0] (bytes), gate_scales + e * stride_scales[0]
 * (f16 elements), and likewise for up [1] and down [2]. hidden and inter are multiples
 * of 256 in [256, 16384]; every codes pointer and byte stride is a multiple of 128. */
typedef struct {
  int32_t n_experts;
  int32_t hidden;
  int32_t inter;
  const uint8_t* gate_codes;
  const uint16_t* gate_scales;
  const uint8_t* up_codes;
  const uint16_t* up_scales;
  const uint8_t* down_codes;
  const uint16_t* down_scales;
  int64_t stride_codes[3];
  int64_t stride_scales[3];
} tq_experts;

/* Bytes of the codes plane (n * k / 2) and of the scales plane (2 * n * k / 256) of an
 * n x k matrix; 0 if k % 256 != 0 or n < 0. Sec. 2.2: 4.0625 bits/weight in total. */
size_t tq_codes_bytes(int32_t n, int32_t k);
size_t tq_scales_bytes(int32_t n, int32_t k);

/* The same two sizes under the names of the boundary's specification. */
size_t tq_packed_codes_bytes(int32_t n, int32_t k);
size_t tq_packed_scales_bytes(int32_t n, int32_t k);

/* Pack a folded code plane on the host (Sec. 2.2 persistent format). c: host [n][k]
 * codes in -4..4; s_f16: host [n][k/256] binary16 bit patterns; codes_out: host,
 * tq_codes_bytes(n, k); scales_out: host, n * (k/256) elements (a copy of s_f16).
 * TQ_ERR_INVALID if a code is outside -4..4 (the outputs are then unspecified). */
tq_status tq_pack_host(const int8_t* c, const uint16_t* s_f16, int32_t n, int32_t k, uint8_t* codes_out,
                       uint16_t* scales_out);

/* Fold and pack on the host (Sec. 2.1 fold, Sec. 2.2 persistent format).
 * t1, t2: host [n][k] trits in {-1,0,1}; codes_out: host, tq_codes_bytes(n, k) bytes.
 * Writes c = 3*t1 + t2 as nibbles c & 15 in the layout above. TQ_ERR_INVALID if a
 * trit is out of range (codes_out is then unspecified). */
tq_status tq_fold_pack_host(const int8_t* t1, const int8_t* t2, int32_t n, int32_t k,
                            uint8_t* codes_out);

/* Inverse of the packing on the host: codes (host, layout above) -> c_out (host [n][k]
 * int8 in -4..4). TQ_ERR_INVALID if a nibble is not that of -4..4 (5..11). */
tq_status tq_unpack_host(const uint8_t* codes, int32_t n, int32_t k, int8_t* c_out);

/* Synthetic matrix generated on the device, folded and packed in place: trits and
 * scales follow the SplitMix64 counter recipe keyed by `key` (word(key, i) is the i-th
 * SplitMix64 output from state `key`; element e = r*k + col takes t1, t2 from the 16-bit
 * fields (0,1) of word(key, e/2) if e is even and (2,3) if odd, trit = ((f*3)>>16) - 1;
 * scale j = r*kb + b is 0x1419 + ((hi32(word(key, n*k/2 + j)) * 0x1A4E) >> 32) as f16
 * bits, i.e. uniform over the f16 values in [1e-3, 1e-1]). For benchmark and test
 * workloads too large to draw on the host; the fold and pack are those of
 * tq_fold_pack_host. codes: 128-byte aligned, tq_codes_bytes(n, k); scales: n * kb. */
tq_status tq_synth_weights(uint64_t key, int32_t n, int32_t k, uint8_t* codes,
                           uint16_t* scales, void* stream);

/* Activation quantizer (Sec. 2.2 block-quantized activations; rule stated above).
 * x [t][k] fp32 (16-byte aligned) -> q [t][k] int8 (16-byte aligned), d [t][kb] fp32,
 * bsum [t][kb] int32. t >= 0 (t = 0 is a no-op); k % 256 == 0, k <= 16384. */
tq_status tq_quantize_act(const float* x, int64_t t, int32_t k, int8_t* q, float* d,
                          int32_t* bsum, void* stream);

/* Tied quantizer (Sec. 2.1: with the plane scales tied at alpha = (3s, s), the solver's
 * alternating plane and scale updates fit the uniform quantizer W_hat = s*c, c in -4..4):
 * w [n][k] fp32 (finite; 4-byte aligned) -> codes and scales in the persistent layout
 * above (codes 128-byte aligned, tq_codes_bytes(n, k); scales [n][kb]). Per 256-weight
 * block, the reading taken (the paper gives no start, stopping rule or precision):
 *   amax = max|w|; amax < 2^-100 -> s = 0, c = 0. Otherwise start at s = amax/4, then
 *   code step c = clamp(rne(fl32(w / s)), -4, 4) (IEEE fp32 division) and scale step
 *   s = fl32(<w,c> / <c,c>), with <w,c> summed in fp64 by pairwise halving
 *   (v[i] += v[i+h] for h = 128, 64, ..., 1) and <c,c> exact, until a code step repeats
 *   the previous codes or max_iter code steps were taken (1..255). The stored scale is
 *   f16(s) (nearest even, saturating at 65504) and the stored codes are the code step at
 *   that scale (zero if it is 0). iters: NULL or [n][kb] bytes, the code steps taken per
 *   block (0 for a zero block). Deterministic; n >= 0 (0 is a no-op). */
tq_status tq_tied_quantize(const float* w, int32_t n, int32_t k, int32_t max_iter, uint8_t* codes,
                           uint16_t* scales, uint8_t* iters, void* stream);

/* The serving dot pass for one matrix and t tokens (Sec. 2.2): y[t][n] fp32 =
 * sum_b f32(s[r][b]) * d[t][b] * isum[t][r][b]. q, d as from tq_quantize_act (q 16-byte
 * aligned); bsum is accepted so callers can pass the quantizer's whole output, but the
 * signed nibbles need no offset correction and the kernel does not read it (may be NULL). isum_dbg: NULL, or a [t][n][kb] int32 buffer that receives the
 * exact block sums (debug and parity; same kernel, one extra store per block).
 * t >= 0 (t = 0 is a no-op). */
tq_status tq_gemv(const tq_mat* w, const int8_t* q, const float* d, const int32_t* bsum,
                  int64_t t, float* y, int32_t* isum_dbg, void* stream);

/* As tq_gemv, and also times the kernel with two host-created HIP events (hipEvent_t,
 * passed as void*): the kernel is launched with hipExtLaunchKernelGGL, so events[0] and
 * events[1] carry its own start and stop timestamps. For benchmarks; neither event may
 * be NULL. */
tq_status tq_gemv_timed(const tq_mat* w, const int8_t* q, const float* d, const int32_t* bsum,
                        int64_t t, float* y, int32_t* isum_dbg, void* stream, void* const* events);

/* The dot pass for one matrix on fp32 activations (Sec. 2.2, quantization included):
 * x [t][k] fp32 (16-byte aligned) is quantized per 256-block by the rule above into
 * q [t][k] (16-byte aligned), d [t][kb], bsum [t][kb] (outputs, caller-owned), and
 * y [t][n] = the tq_gemv pass on them. One token is one launch: every workgroup
 * quantizes x into its LDS beside its weight loads (workgroup 0 also writes q, d,
 * bsum), and y is bitwise what tq_quantize_act followed by tq_gemv gives. Several tokens
 * (or n * k / 2 >= 2^32 code bytes): those two launches. isum_dbg as in tq_gemv. */
tq_status tq_gemv_f32(const tq_mat* w, const float* x, int64_t t, float* y, int8_t* q, float* d, int32_t* bsum,
                      int32_t* isum_dbg, void* stream);

/* As tq_gemv_f32, timed with two host-created HIP events: at one token they carry the
 * kernel's own start/stop timestamps; otherwise they are recorded on the stream before
 * the quantizer and after the dot pass. */
tq_status tq_gemv_f32_timed(const tq_mat* w, const float* x, int64_t t, float* y, int8_t* q, float* d,
                            int32_t* bsum, int32_t* isum_dbg, void* stream, void* const* events);

/* ---------------------------------------------------------------------------------
 * Free-scale two-plane variant (Sec. 2.1: PTQTP's W ~ alpha1*T1 + alpha2*T2 with two
 * free scales per group, the family the tie constrains; Sec. 4.1, the quality table's
 * note: the free pair does not fold, so it is served as its two trit planes, stored
 * apart: 4.125 bits/weight). The ablation of the fold: same blocks, same activations,
 * one integer pass per plane.
 *   codes  [n][kb][128] bytes, 128-byte aligned. Chunk j (bytes 16j .. 16j+15 of a
 *          block) covers columns 32j .. 32j+31: bytes 16j .. 16j+7 are plane 1, bytes
 *          16j+8 .. 16j+15 plane 2. Within a plane's 8 bytes, byte 4u + b (u = 0, 1;
 *          b = 0..3), bits 2s .. 2s+1 (s = 0..3) hold the trit of column
 *          32j + 16u + 4s + b as 2-bit two's complement (00 = 0, 01 = +1, 11 = -1; 10
 *          never occurs): shifted to a byte's top two bits it reads as 64*t.
 *   scales [n][kb][2] IEEE binary16 bit patterns (alpha1, alpha2 of row r, block b),
 *          4-byte aligned. Bytes: 128 + 4 per 256 weights = 4.125 bits/weight.
 * Pass: isum_p[t][r][b] = sum_i Tp[r][256b+i] * q[t][256b+i] (exact int32, p = 1, 2),
 *   y[t][r] = sum_b d[t][b] * (f32(alpha1) * isum_1 + f32(alpha2) * isum_2) in fp32.
 * --------------------------------------------------------------------------------- */
typedef struct {
  int32_t n;
  int32_t k;
  const uint8_t* codes;
  const uint16_t* scales; /* [n][kb][2] */
} tq_mat2;

/* Pack two trit planes on the host into the two-plane layout above. t1, t2: host
 * [n][k] in {-1,0,1}; codes_out: host, tq_codes_bytes(n, k) bytes (the same byte count
 * as the folded plane). TQ_ERR_INVALID if a trit is out of range (codes_out is then
 * unspecified). The scales need no packing: [n][kb][2] f16 is their layout. */
tq_status tq_pack2_host(const int8_t* t1, const int8_t* t2, int32_t n, int32_t k, uint8_t* codes_out);

/* Inverse of tq_pack2_host on the host. TQ_ERR_INVALID on the unused pattern 10. */
tq_status tq_unpack2_host(const uint8_t* codes, int32_t n, int32_t k, int8_t* t1_out, int8_t* t2_out);

/* Free-scale solver (Sec. 2.1: PTQTP's alternation of plane and scale updates with two
 * free scales per group), started from a tied fit of the same weights (tq_tied_quantize
 * output: its codes and f16 scales) and written in the two-plane layout above. Per
 * 256-weight block, the reading taken (the paper gives no start, stop rule or
 * precision):
 *   start: planes = the unfolded tied codes, (alpha1, alpha2) = (3 s, s) with s the tied
 *   f16 scale; s = 0 gives a zero fit. Then, until a plane step repeats the previous
 *   planes or max_iter plane steps were taken (1..255):
 *   scale step: with a = <T1,T1>, b = <T1,T2>, c = <T2,T2> (exact), u = <w,T1> and
 *   v = <w,T2> (fp64 products, pairwise-halving sums as in tq_tied_quantize), and
 *   det = a c - b^2: if det > 0, alpha1 = fl32((c u - b v) / det), alpha2 =
 *   fl32((a v - b u) / det), each fp64 operation rounded on its own (no fused
 *   multiply-add); otherwise the scales stay;
 *   plane step: each weight takes the first pair (t1, t2), t1 and then t2 in the order
 *   0, -1, +1, with the least |w - (alpha1 t1 + alpha2 t2)| in fp64.
 *   The stored scales are f16 (nearest even, saturating at +-65504) and the stored planes
 *   a plane step at those scales. iters: NULL or [n][kb] bytes, the plane steps taken
 *   per block (0 for a zero block). w finite, 4-byte aligned; tied codes 128-byte, tied
 *   scales 2-byte, codes2 128-byte, scales2 ([n][kb][2]) 4-byte aligned. Deterministic. */
tq_status tq_free_quantize(const float* w, int32_t n, int32_t k, int32_t max_iter, const uint8_t* tied_codes,
                           const uint16_t* tied_scales, uint8_t* codes2, uint16_t* scales2, uint8_t* iters,
                           void* stream);

/* The two-plane pass for one matrix and t tokens (formula above). q, d as from
 * tq_quantize_act (q 16-byte aligned). isum_dbg: NULL, or a [t][n][kb][2] int32 buffer
 * that receives the exact per-plane block sums (plane 1 first). n >= 1, 256 <= k <=
 * 16384, t >= 0 (t = 0 is a no-op). */
tq_status tq_gemv2(const tq_mat2* w, const int8_t* q, const float* d, int64_t t, float* y,
                   int32_t* isum_dbg, void* stream);

/* As tq_gemv2, with the kernel's own start/stop timestamps in two host-created HIP
 * events (as tq_gemv_timed). */
tq_status tq_gemv2_timed(const tq_mat2* w, const int8_t* q, const float* d, int64_t t, float* y,
                         int32_t* isum_dbg, void* stream, void* const* events);

/* ---------------------------------------------------------------------------------
 * MXFP4 reference arm (Sec. 2.3: the released expert bytes, e2m1 (fp4) codes whose
 * groups of 32 share an e8m0 scale, Sec. 2.1, served by an integer kernel through the doubled
 * e2m1 values {0,1,2,3,4,6,8,12}, the e8m0 scale absorbing the /2).
 *   codes  [n][kb][128] bytes, 128-byte aligned: 16-byte block j of a row covers
 *          elements 32j .. 32j+31; its byte i holds element 32j+i in the low nibble and
 *          32j+16+i in the high nibble, each an e2m1 code (bit 3 sign, bits 2..1 exponent
 *          with bias 1, bit 0 mantissa; exponent 0 is subnormal).
 *   scales [n][k/32] e8m0 bytes, 2^(E - 127) (E = 255, NaN, must not occur).
 *   Bytes: 16 + 1 per 32 weights = 4.25 bits/weight, the paper's 17-byte blocks with
 *   codes and scales in two planes.
 * Pass: isum[t][r][j] = sum_i 2*e2m1(c[r][32j+i]) * q[t][32j+i] (exact int32),
 *   y[t][r] = sum_j f32(2^(E[r][j] - 128) * d[t][j/8]) * isum[t][r][j] in fp32.
 * Precondition (not checked): each 2^(E - 128) * d is a normal fp32 value and the sums
 * stay within the fp32 range.
 * --------------------------------------------------------------------------------- */
typedef struct {
  int32_t n;
  int32_t k;
  const uint8_t* codes;
  const uint8_t* scales; /* [n][k/32] e8m0 */
} tq_mat_mx;

/* Pack e2m1 codes on the host into the layout above. c4: host [n][k] codes 0..15;
 * codes_out: host, n * k / 2 bytes. TQ_ERR_INVALID if a code exceeds 15. */
tq_status tq_mx_pack_host(const uint8_t* c4, int32_t n, int32_t k, uint8_t* codes_out);

/* Inverse of tq_mx_pack_host on the host. */
tq_status tq_mx_unpack_host(const uint8_t* codes, int32_t n, int32_t k, uint8_t* c4_out);

/* The MXFP4 arm's pass for one matrix and t tokens (formula above). q, d as from
 * tq_quantize_act (q 16-byte aligned). isum_dbg: NULL, or a [t][n][k/32] int32 buffer
 * that receives the exact 32-element block sums. n >= 1, 256 <= k <= 16384, t >= 0. */
tq_status tq_gemv_mx(const tq_mat_mx* w, const int8_t* q, const float* d, int64_t t, float* y,
                     int32_t* isum_dbg, void* stream);

/* As tq_gemv_mx, with the kernel's own start/stop timestamps in two host-created HIP
 * events (as tq_gemv_timed). */
tq_status tq_gemv_mx_timed(const tq_mat_mx* w, const int8_t* q, const float* d, int64_t t, float* y,
                           int32_t* isum_dbg, void* stream, void* const* events);

/* Routed-expert MoE layer over the folded experts (Sec. 2.2 dot pass applied to every
 * routed gate/up/down projection; the paper's layers are 43 x 3 projections x 256
 * experts, Sec. 2.1). For every token t and slot j < topk with e = topk_idx[t][j]:
 *   xq = quantize(x[t]);  g = W_gate[e] xq;  u = W_up[e] xq  (dot pass, fp32)
 *   h = SiLU(g) * u  (fp32, SiLU(z) = z / (1 + exp(-z)));  hq = quantize(h)
 *   y[t][j] = W_down[e] hq;   out[t] = sum_j topk_w[t][j] * y[t][j]  (ascending j)
 * A slot whose expert id lies outside [0, n_experts) contributes nothing and sets a
 * device flag that tq_moe_status reports. Duplicate ids in a token's list are separate
 * slots. x: [t][hidden] fp32 (16-byte aligned); topk_idx, topk_w: [t][topk];
 * out: [t][hidden] fp32, overwritten. 1 <= topk <= 64, topk <= n_experts.
 * ws: device workspace of at least tq_moe_workspace_bytes(ex, t, topk) bytes, 256-byte
 * aligned; its contents on entry are ignored, and on return it holds the stage buffers
 * described by tq_moe_workspace_layout (for staged parity checks). Calls that share a
 * workspace must be ordered on one stream.
 * flags: 0 (automatic path choice), or TQ_MOE_FORCE_VALU / TQ_MOE_FORCE_MFMA to pin
 * the per-expert path (VALU dot4 for few tokens per expert, int8 MFMA for many; the
 * automatic choice mixes the two below 2048 slots, see tq_moe_path).
 * Single-token steps (t == 1, topk <= 8, topk * inter <= 16384) take a path of their
 * own unless TQ_MOE_FORCE_MFMA is given (tq_moe_path). The grouped paths address the
 * quantized activations with 32-bit offsets: TQ_ERR_INVALID if t * topk * max(hidden,
 * inter) >= 2^31 (and t > 1 or TQ_MOE_FORCE_MFMA).
 * Streams: every launch follows the work queued on `stream`, and work queued on `stream`
 * after the call follows every launch. The grouped MFMA path (and the mixed path with
 * TQ_MOE_DEBUG_STAGES) runs each projection as two launches that write disjoint
 * outputs, the second on a stream the library owns (one per device, default priority,
 * created by the first such call on the device that is not made under stream capture),
 * forked from and joined back to `stream` by events; under capture the fork and join
 * become graph edges. Until that stream exists, or if it could not be created, the two
 * launches run in order on `stream`.
 * TQ_MOE_DEBUG_STAGES (may be or-ed with either): the same kernels, each taking one
 * extra branch on a kernel argument, also leave in the workspace, past the stage buffers,
 * every routed slot's g and u (fp32) and the exact int32 block sums of its gate, up and
 * down dot passes (offsets g, u, gsum, usum, dsum of tq_moe_workspace_layout); the
 * workspace must then hold total_debug bytes. Rows of unrouted slots are not written.
 * The outputs are bitwise those of the same call without the flag. */
#define TQ_MOE_FORCE_VALU 1
#define TQ_MOE_FORCE_MFMA 2
#define TQ_MOE_DEBUG_STAGES 4
tq_status tq_moe_grouped(const tq_experts* ex, const float* x, int64_t t,
                         const int32_t* topk_idx, const float* topk_w, int32_t topk,
                         float* out, void* ws, size_t ws_bytes, int32_t flags, void* stream);
size_t tq_moe_workspace_bytes(const tq_experts* ex, int64_t t, int32_t topk);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation): tq_moe_grouped with its workspace
 * taken from a fixed device array of tq_moe_noalloc_max_bytes() bytes (16 MiB) that the
 * library holds on every GPU it runs on until the process ends, one array per device,
 * that of the calling thread's current device (the stream must belong to it). The call
 * itself allocates and frees nothing. Arguments and results as tq_moe_grouped; the
 * caller still owns x, topk_idx, topk_w and out. TQ_ERR_WORKSPACE, before any launch, if
 * the call's workspace (tq_moe_workspace_bytes, or the layout's total_debug with
 * TQ_MOE_DEBUG_STAGES) exceeds the array: about 600 slots (t * topk) at hidden 4096 and
 * inter 2048. Every call on a GPU shares that GPU's array, and the array keeps the last
 * call's stage buffers (readable at the offsets of tq_moe_workspace_layout only by the
 * library): calls that may overlap on one GPU (other streams, other threads) race and
 * must be ordered by the caller. No part of the array needs clearing between calls. It
 * creates no stream or event either: the grouped MFMA path's second stream (see
 * tq_moe_grouped) serves it once an earlier tq_moe_grouped call on the device made one;
 * until then its two launches per projection run in order on `stream`. */
size_t tq_moe_noalloc_max_bytes(void);
tq_status tq_moe_grouped_noalloc(const tq_experts* ex, const float* x, int64_t t, const int32_t* topk_idx,
                                 const float* topk_w, int32_t topk, float* out, int32_t flags, void* stream);

/* The path tq_moe_grouped takes for these arguments: TQ_MOE_PATH_T1 (single token: a
 * gate/up kernel, then a down kernel with the requantization and the weighted combine
 * fused), TQ_MOE_PATH_VALU (dispatch + grouped VALU dot4 kernels), TQ_MOE_PATH_MFMA
 * (dispatch + grouped int8 MFMA kernels), TQ_MOE_PATH_MIXED (the automatic choice for
 * fewer than 2048 slots and more than 2 tokens: dispatch + one launch per projection
 * whose first workgroups run the 32-token MFMA tiles of the experts of more than 2 slots
 * and the others the grouped VALU tasks of the remaining experts); -1 if the arguments
 * are invalid. Host only, no device work. */
#define TQ_MOE_PATH_T1 0
#define TQ_MOE_PATH_VALU 1
#define TQ_MOE_PATH_MFMA 2
#define TQ_MOE_PATH_MIXED 3
int32_t tq_moe_path(const tq_experts* ex, int64_t t, int32_t topk, int32_t flags);

/* Byte offsets, inside the workspace, of the stage buffers tq_moe_grouped leaves behind
 * (S = t * topk slots, slot s = t * topk + j):
 *   xq [t][hidden] int8, xd [t][hidden/256] fp32, xb [t][hidden/256] int32;
 *   h [S][inter] fp32; hq [S][inter] int8, hd [S][inter/256] fp32, hb [S][inter/256] int32;
 *   yd [S][hidden] fp32 (per-slot down output, before the routing weight);
 *   flags: int32, bit 0 set if an expert id was out of range;
 *   total: the workspace size without the debug dump (tq_moe_workspace_bytes).
 * Dispatch lists of the grouped paths (t > 1, or TQ_MOE_FORCE_MFMA; not written by the
 * single-token path): n_active int32 = A, the number of distinct routed experts;
 * active [A] int32 their ids in the order the work queues take them; act_off [A + 1]
 * int32 offsets into slot_list [S] int32, which lists each active expert's slots (slot
 * order within an expert unspecified).
 * Debug dump (TQ_MOE_DEBUG_STAGES only): g, u [S][inter] fp32; gsum, usum
 * [S][inter][hidden/256] int32; dsum [S][hidden][inter/256] int32; total_debug: the
 * workspace size the flag needs. */
typedef struct {
  size_t xq, xd, xb, h, hq, hd, hb, yd, flags;
  size_t total;
  size_t n_active, active, act_off, slot_list;
  size_t g, u, gsum, usum, dsum;
  size_t total_debug;
} tq_moe_layout;
tq_status tq_moe_workspace_layout(const tq_experts* ex, int64_t t, int32_t topk,
                                  tq_moe_layout* out);

/* As tq_moe_grouped, and also times each stage with host-created HIP events
 * (hipEvent_t, passed as void*): events[2*i] and events[2*i + 1] bracket stage i, for
 * i < tq_moe_stage_count(). A stage's kernel is launched with hipExtLaunchKernelGGL, so
 * its pair carries that kernel's own start and stop timestamps; a grouped MFMA stage run
 * as two launches on two streams has its pair recorded on `stream` before the fork and
 * after the join (it spans both launches, and the event commands' own cost); a stage
 * with no kernel on the path taken (a single-token step fuses the prologue, requant and
 * combine into its two kernels) has its pair recorded back to back. For per-stage timing
 * in benchmarks; no event may be NULL. */
int32_t tq_moe_stage_count(void);
const char* tq_moe_stage_name(int32_t i);
tq_status tq_moe_grouped_timed(const tq_experts* ex, const float* x, int64_t t,
                               const int32_t* topk_idx, const float* topk_w, int32_t topk,
                               float* out, void* ws, size_t ws_bytes, int32_t flags,
                               void* stream, void* const* events);

/* Synchronizes `stream`, then copies the workspace's device flags word to *flags_out
 * (host): bit 0 set if an expert id was out of range in the last call. Returns TQ_OK, or
 * TQ_ERR_DEVICE if the stream reports an error. */
tq_status tq_moe_status(const void* ws, const tq_experts* ex, int64_t t, int32_t topk,
                        int32_t* flags_out, void* stream);

/* ---------------------------------------------------------------------------------
 * Host-tier expert streaming (Sec. 2.2: the folded planes are the stored file itself,
 * so fetching a missing expert projection costs a single contiguous read, and serving
 * from HBM or from the host tier runs the same kernels on the same bytes: an expert
 * gives the same output bits wherever it was cached; the
 * paper's store keeps pinned RAM and LRU slots in front of the file). Tiers here: every
 * expert in pinned host memory, a pool of expert slots in HBM.
 * An expert record is one contiguous range: gate, up, down codes, then gate, up, down
 * scales, each piece 128-byte aligned, tq_expert_record_bytes(hidden, inter) bytes in
 * all. The same record layout serves the host store ([n_experts] records) and the slot
 * pool ([n_slots] records); tq_experts_from_records describes either to tq_moe_grouped.
 * A streamed step: tq_cache_map (host: expert ids -> slots, LRU eviction), tq_cache_fetch
 * (enqueue one host-to-device copy per miss and the slot ids), then tq_moe_grouped on
 * the pool's descriptor with the slot ids as topk_idx, all on one stream.
 * --------------------------------------------------------------------------------- */

/* Bytes of one expert record (a multiple of 128); 0 for an invalid shape. */
size_t tq_expert_record_bytes(int32_t hidden, int32_t inter);

/* Fills *out (host) for n_records expert records at `base` (device or host address,
 * 128-byte aligned): the projections' pointers inside record 0 and the record size as
 * every stride. hidden, inter: multiples of 256 in [256, 16384]. */
tq_status tq_experts_from_records(const void* base, int32_t n_records, int32_t hidden, int32_t inter,
                                  tq_experts* out);

/* Bytes of the LRU planner's state (host memory, owned by the caller, 8-byte aligned);
 * 0 if n_experts or n_slots < 1. */
size_t tq_cache_state_bytes(int32_t n_experts, int32_t n_slots);

/* Empties the pool. */
tq_status tq_cache_init(void* state, int32_t n_experts, int32_t n_slots);

/* Host only. ids: host [n] expert ids of one step (duplicates allowed). Writes
 * slots_out (host [n]): each id's slot. Experts not resident are placed in order of first
 * appearance, each in an empty slot (lowest index) if any, else in the least recently
 * used slot that this step does not use (lowest index on ties); misses_out (host, up to
 * 2n int32) receives the (expert, slot) pairs to copy and *n_miss_out their count.
 * TQ_ERR_INVALID, with the pool unchanged, if an id is outside [0, n_experts) or the
 * step names more distinct experts than there are slots. Deterministic. */
tq_status tq_cache_map(void* state, const int32_t* ids, int64_t n, int32_t* slots_out,
                       int32_t* misses_out, int32_t* n_miss_out);

/* Enqueues on `stream` one host-to-device copy of record_bytes per miss (host_store
 * record `expert` -> dev_slots record `slot`), then the copy of the n slot ids
 * slots_host -> slots_dev. host_store and slots_host should be pinned host memory (for
 * asynchronous copies) and must stay unchanged until the copies have executed.
 * Every miss and slot id is checked against the state's store and pool sizes before
 * anything is enqueued. */
tq_status tq_cache_fetch(const void* state, const void* host_store, void* dev_slots, size_t record_bytes,
                         const int32_t* misses, int32_t n_miss, const int32_t* slots_host,
                         int32_t* slots_dev, int64_t n, void* stream);

/* Benchmark ceiling (not part of the method): one launch that reads `bytes` (a multiple
 * of 16) from src with nontemporal 16-byte loads, each byte once, and keeps only an XOR of
 * them (sink: one uint32 that is practically never written), timed like tq_gemv_timed
 * (events[0], events[1]: the kernel's own start and stop timestamps). The dot pass's
 * throughput is reported as a fraction of this rate on the same byte count. */
tq_status tq_stream_read_timed(const void* src, size_t bytes, uint32_t* sink, void* stream, void* const* events);

/* Thread-local description of the last failed call on this thread ("" if none). */
const char* tq_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TQ_H_ */
