"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each pin is a function of an ``Oracle`` handle that raises AssertionError when the
oracle is wrong. The pins are chosen so that a plausible mistake anywhere in the
oracle (a transposed plane, a dropped factor, a wrong index or rounding rule) fails at
least one of them; ``test_oracle_mutants.py`` checks exactly that by running them
against deliberately broken builds. None of them re-derives the oracle's formula by
re-calling the oracle: the references are paper values (``golden/paper_facts.json``),
closed forms, invariants, library routines (numpy, scipy) and pure-Python brute force
on tiny inputs (``brute.py``).
"""
from __future__ import annotations

import json
import os
from fractions import Fraction

import numpy as np

import brute

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_facts.json")))

PINS = []


def pin(fn):
    PINS.append(fn)
    return fn


def _f16(vals):
    return np.asarray(vals, dtype=np.float16).view(np.uint16)


def _f16_to_np64(bits):
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


# --------------------------------------------------------------------------------------
# Fold / unfold (Sec. 2.1 tied composite; Sec. 2.2)
# --------------------------------------------------------------------------------------

@pin
def fold_table_matches_paper(o):
    rows = np.array(GOLDEN["fold_table"]["rows_t1_t2_c"])
    c = o.fold(rows[:, 0], rows[:, 1])
    assert c.tolist() == rows[:, 2].tolist()


@pin
def fold_is_bijection_onto_nine_levels(o):
    t1, t2 = np.meshgrid([-1, 0, 1], [-1, 0, 1], indexing="ij")
    c = o.fold(t1.ravel(), t2.ravel())
    assert sorted(c.tolist()) == list(range(-4, 5))


@pin
def unfold_inverts_fold(o):
    t1, t2 = np.meshgrid([-1, 0, 1], [-1, 0, 1], indexing="ij")
    u1, u2 = o.unfold(o.fold(t1.ravel(), t2.ravel()))
    assert u1.tolist() == t1.ravel().tolist() and u2.tolist() == t2.ravel().tolist()
    c = np.arange(-4, 5, dtype=np.int8)
    assert o.fold(*o.unfold(c)).tolist() == c.tolist()
    rng = np.random.default_rng(7)
    a = rng.integers(-1, 2, 5000).astype(np.int8)
    b = rng.integers(-1, 2, 5000).astype(np.int8)
    v1, v2 = o.unfold(o.fold(a, b))
    assert np.array_equal(v1, a) and np.array_equal(v2, b)


@pin
def fold_equals_tied_two_plane_model(o):
    # W_hat = 3s*T1 + s*T2 must equal s*c with c = fold(T1, T2) (Sec. 2.1); s dyadic so
    # the fp64 products are exact.
    t1, t2 = np.meshgrid([-1, 0, 1], [-1, 0, 1], indexing="ij")
    t1, t2 = t1.ravel().astype(np.int8), t2.ravel().astype(np.int8)
    c = o.fold(t1, t2).astype(np.float64)
    for s in (1.0, 0.5, 2.0 ** -7, 3.0):
        assert np.array_equal(o.two_plane_dequant(t1, t2, 3 * s, s), s * c)


@pin
def level_sets_match_paper(o):
    t1, t2 = np.meshgrid([-1, 0, 1], [-1, 0, 1], indexing="ij")
    t1, t2 = t1.ravel().astype(np.int8), t2.ravel().astype(np.int8)
    ls = GOLDEN["level_sets"]
    for ratio, levels in ls["in_units_of_alpha2"].items():
        got = sorted(set(o.two_plane_dequant(t1, t2, float(ratio), 1.0).tolist()))
        assert got == [float(v) for v in levels], (ratio, got)
        assert len(set(np.diff(got).tolist())) == 1  # uniformly spaced
    gen = sorted(set(o.two_plane_dequant(t1, t2, ls["generic_ratio_example"], 1.0).tolist()))
    assert len(gen) == ls["generic_distinct_levels"] and len(set(np.round(np.diff(gen), 12).tolist())) > 1
    # ratio 1/3: nine uniform levels with the plane labels exchanged
    inv = sorted(set(o.two_plane_dequant(t1, t2, 1.0, 3.0).tolist()))
    assert inv == [float(v) for v in ls["in_units_of_alpha2"]["3"]]
    # signs absorb into a plane
    neg = sorted(set(o.two_plane_dequant(t1, t2, -3.0, 1.0).tolist()))
    assert neg == [float(v) for v in ls["in_units_of_alpha2"]["3"]]


# --------------------------------------------------------------------------------------
# f16 scale decode (Sec. 2.1: the scales are stored as f16)
# --------------------------------------------------------------------------------------

@pin
def f16_decode_matches_numpy_all_patterns(o):
    bits = np.arange(0, 65536, 97, dtype=np.uint16)  # every 97th pattern incl. subnormals
    bits = np.concatenate([bits, np.array([0x0001, 0x03FF, 0x0400, 0x3C00, 0x7BFF, 0x7C00, 0xFC00, 0x8001], dtype=np.uint16)])
    got = o.f16_to_f64(bits)
    ref = _f16_to_np64(bits)
    both_nan = np.isnan(got) & np.isnan(ref)
    assert np.array_equal(got[~both_nan], ref[~both_nan])
    assert np.array_equal(np.isnan(got), np.isnan(ref))


@pin
def dequant_matches_numpy_f16(o):
    rng = np.random.default_rng(3)
    c = rng.integers(-4, 5, (5, 512)).astype(np.int8)
    s = _f16(rng.uniform(1e-3, 1e-1, (5, 2)))
    w = o.dequant(c, s)
    ref = np.repeat(_f16_to_np64(s), 256, axis=1) * c
    assert np.array_equal(w, ref)


# --------------------------------------------------------------------------------------
# Activation quantizer (Sec. 2.2 block-quantized activations; reading: 256-blocks,
# absmax/127 in fp32, round half to even)
# --------------------------------------------------------------------------------------

def _block(vals, fill=0.0):
    x = np.full(256, fill, dtype=np.float32)
    x[: len(vals)] = vals
    return x


@pin
def quantize_unit_scale_rounds_half_to_even(o):
    # amax = 127 -> inv = 127/127 = 1 exactly -> q = rne(x) (closed form)
    vals = [127, 0.5, 1.5, 2.5, -2.5, -0.5, 3.5, -3.5, 126.5, 0.49999997, -1.5000001, 64.0]
    want = [127, 0, 2, 2, -2, 0, 4, -4, 126, 0, -2, 64]
    q, d, b = o.quantize(_block(vals))
    assert q[0, : len(want)].tolist() == want and not q[0, len(want):].any()
    assert d[0, 0] == np.float32(1.0) and b[0, 0] == sum(want)


@pin
def quantize_scale_254_halves(o):
    # amax = 254 -> inv = 0.5 exactly, d = 2 -> q = rne(x / 2)
    vals = [254, 1, 3, 5, -5, 7, -254, 2, -1]
    want = [127, 0, 2, 2, -2, 4, -127, 1, 0]
    q, d, b = o.quantize(_block(vals))
    assert q[0, : len(want)].tolist() == want and d[0, 0] == np.float32(2.0)
    assert b[0, 0] == sum(want)


@pin
def quantize_amax_element_and_error_bound(o):
    rng = np.random.default_rng(11)
    for scale in (1e-6, 3e-3, 1.0, 37.0, 1e5):
        x = (rng.standard_normal((3, 1024)) * scale).astype(np.float32)
        q, d, b = o.quantize(x)
        for t in range(3):
            for blk in range(4):
                xs = x[t, blk * 256:(blk + 1) * 256].astype(np.float64)
                qs = q[t, blk * 256:(blk + 1) * 256].astype(np.int64)
                i = int(np.argmax(np.abs(xs)))
                assert qs[i] == (127 if xs[i] > 0 else -127)
                assert np.abs(qs).max() <= 127
                dd = float(d[t, blk])
                assert abs(dd - np.abs(xs).max() / 127) <= 2 ** -23 * dd
                assert np.all(np.abs(xs - dd * qs) <= dd * (0.5 + 2 ** -14))
                assert b[t, blk] == qs.sum()


@pin
def quantize_odd_symmetry(o):
    rng = np.random.default_rng(5)
    x = rng.standard_normal((2, 512)).astype(np.float32)
    q1, d1, b1 = o.quantize(x)
    q2, d2, b2 = o.quantize(-x)
    assert np.array_equal(q2, -q1) and np.array_equal(d1, d2) and np.array_equal(b2, -b1)


@pin
def quantize_blocks_are_independent_and_zero_block(o):
    rng = np.random.default_rng(9)
    x = rng.standard_normal((1, 768)).astype(np.float32)
    x[0, 256:512] = 0.0
    q, d, b = o.quantize(x)
    assert d[0, 1] == 0 and b[0, 1] == 0 and not q[0, 256:512].any()
    # below 2^-100 a block quantizes to zeros; at 2^-100 it does not
    tiny = np.zeros((1, 512), np.float32)
    tiny[0, :256] = np.float32(2.0 ** -101) * np.linspace(-1, 1, 256, dtype=np.float32)
    tiny[0, 256:] = np.float32(2.0 ** -100) * np.linspace(-1, 1, 256, dtype=np.float32)
    qt, dt, _ = o.quantize(tiny)
    assert dt[0, 0] == 0 and not qt[0, :256].any()
    assert dt[0, 1] > 0 and qt[0, 256] == -127 and qt[0, 511] == 127
    # a large value at index 255 changes block 0 only; at index 256 block 1 only
    y = x.copy(); y[0, 255] = 1000.0
    qy, dy, _ = o.quantize(y)
    assert dy[0, 0] != d[0, 0] and dy[0, 1] == d[0, 1] and dy[0, 2] == d[0, 2]
    assert np.array_equal(qy[0, 256:], q[0, 256:])
    z = x.copy(); z[0, 256] = 1000.0
    qz, dz, _ = o.quantize(z)
    assert dz[0, 0] == d[0, 0] and dz[0, 1] == np.float32(np.float32(1000.0) / np.float32(127))
    assert np.array_equal(qz[0, :256], q[0, :256]) and np.array_equal(qz[0, 512:], q[0, 512:])


@pin
def quantize_matches_brute_force(o):
    rng = np.random.default_rng(13)
    x = (rng.standard_normal((2, 512)) * rng.uniform(0.01, 100, (2, 1))).astype(np.float32)
    q, d, b = o.quantize(x)
    for t in range(2):
        bq, bd, bb = brute.quantize(x[t].tolist())
        assert q[t].tolist() == bq and d[t].tolist() == [float(v) for v in bd] and b[t].tolist() == bb


# --------------------------------------------------------------------------------------
# Integer dot pass and scale combine (Sec. 2.2)
# --------------------------------------------------------------------------------------

@pin
def dot_brute_force_all_codes_small_block(o):
    # every 4-element code vector over {-4..4} against a grid of int8 activation vectors
    codes = np.array(np.meshgrid(*[np.arange(-4, 5)] * 4, indexing="ij")).reshape(4, -1).T.astype(np.int8)
    acts = [np.array(v, dtype=np.int8) for v in ([127, -127, 1, 0], [-128, 127, -1, 5], [3, -7, 11, -13])]
    for a in acts:
        ref = codes.astype(np.int64) @ a.astype(np.int64)
        got = np.array([o.dot_i8(cv, a) for cv in codes])
        assert np.array_equal(got, ref)
    # extremes of the block bound |isum| <= 4 * 127 * 256
    assert o.dot_i8(np.full(256, 4, np.int8), np.full(256, 127, np.int8)) == 130048
    assert o.dot_i8(np.full(256, -4, np.int8), np.full(256, 127, np.int8)) == -130048
    assert o.dot_i8(np.full(256, -4, np.int8), np.full(256, -128, np.int8)) == 131072


@pin
def block_sums_equal_trit_plane_identity(o):
    # isum = sum c*q = 3*(T1.q) + (T2.q) exactly (Sec. 2.1 fold, Sec. 2.2 one dot pass),
    # the right side computed from the planes with numpy int64 matmuls.
    rng = np.random.default_rng(17)
    n, k, t = 6, 768, 3
    t1 = rng.integers(-1, 2, (n, k)).astype(np.int8)
    t2 = rng.integers(-1, 2, (n, k)).astype(np.int8)
    c = o.fold(t1, t2)
    q = rng.integers(-127, 128, (t, k)).astype(np.int8)
    s = np.full((n, k // 256), 0x3C00, np.uint16)
    d = np.ones((t, k // 256), np.float32)
    y, a, isum = o.gemv(c, s, q, d, want_isum=True)
    for b in range(k // 256):
        sl = slice(b * 256, (b + 1) * 256)
        ref = 3 * (q[:, sl].astype(np.int64) @ t1[:, sl].T.astype(np.int64)) + q[:, sl].astype(np.int64) @ t2[:, sl].T.astype(np.int64)
        assert np.array_equal(isum[:, :, b], ref)
    # offset form of the same sum: with u = c + 4, sum u*q - 4*sum q
    u = c.astype(np.int64) + 4
    for b in range(k // 256):
        sl = slice(b * 256, (b + 1) * 256)
        off = q[:, sl].astype(np.int64) @ u[:, sl].T - 4 * q[:, sl].astype(np.int64).sum(1, keepdims=True)
        assert np.array_equal(isum[:, :, b], off)


@pin
def gemv_unit_scales_is_exact_integer_dot(o):
    # s = 1 (f16 0x3C00) and integer activations with amax 127 per block (so d = 1):
    # y equals the exact integer product; also checks rows vs tokens are not swapped
    rng = np.random.default_rng(19)
    n, k, t = 5, 512, 3
    c = rng.integers(-4, 5, (n, k)).astype(np.int8)
    x = rng.integers(-126, 127, (t, k)).astype(np.float32)
    x[:, 0] = 127; x[:, 256] = -127
    q, d, _ = o.quantize(x)
    assert np.all(d == 1.0)
    y, _ = o.gemv(c, np.full((n, 2), 0x3C00, np.uint16), q, d)
    ref = x.astype(np.int64) @ c.T.astype(np.int64)
    assert np.array_equal(y, ref.astype(np.float64))


@pin
def gemv_scales_by_powers_of_two_exactly(o):
    rng = np.random.default_rng(23)
    n, k = 4, 512
    c = rng.integers(-4, 5, (n, k)).astype(np.int8)
    s = _f16(rng.uniform(1e-3, 1e-1, (n, 2)))
    x = rng.standard_normal((2, k)).astype(np.float32)
    q, d, _ = o.quantize(x)
    y, _ = o.gemv(c, s, q, d)
    s2 = s.copy(); s2[2, :] += 0x0400  # exponent + 1: row 2's scales doubled
    y2, _ = o.gemv(c, s2, q, d)
    assert np.array_equal(y2[:, 2], 2 * y[:, 2])
    assert np.array_equal(np.delete(y2, 2, axis=1), np.delete(y, 2, axis=1))
    s3 = s.copy(); s3[1, 1] += 0x0400  # only block 1 of row 1
    y3, _, i3 = o.gemv(c, s3, q, d, want_isum=True)
    _, _, i1 = o.gemv(c, s, q, d, want_isum=True)
    term = _f16_to_np64(s[1, 1]) * d[:, 1].astype(np.float64) * i1[:, 1, 1]
    assert np.allclose(y3[:, 1] - y[:, 1], term, rtol=1e-12, atol=0)


@pin
def gemv_matches_dequant_matmul_within_quantization_bound(o):
    # |y - W_hat x| <= sum_b s_b d_b (0.5 + 2^-14) sum_i |c_i|  (+ fp64 slack); W_hat built
    # with numpy's own f16 decode, so a transposed scale index or a dropped factor fails.
    rng = np.random.default_rng(29)
    n, k, t = 7, 1024, 2
    c = rng.integers(-4, 5, (n, k)).astype(np.int8)
    s = _f16(np.exp(rng.uniform(np.log(1e-3), np.log(1e-1), (n, k // 256))))
    x = rng.standard_normal((t, k)).astype(np.float32)
    q, d, _ = o.quantize(x)
    y, a = o.gemv(c, s, q, d)
    W = np.repeat(_f16_to_np64(s), 256, axis=1) * c
    ref = x.astype(np.float64) @ W.T
    absc = np.abs(c.astype(np.float64)).reshape(n, k // 256, 256).sum(2)  # [n][kb]
    bound = (_f16_to_np64(s)[None, :, :] * d.astype(np.float64)[:, None, :] * absc[None]).sum(2) * (0.5 + 2 ** -14)
    assert np.all(np.abs(y - ref) <= bound * (1 + 1e-9) + 1e-12)
    assert np.all(np.abs(y) <= a * (1 + 1e-15))


@pin
def gemv_matches_exact_rational_brute_force(o):
    rng = np.random.default_rng(31)
    n, k = 3, 512
    c = rng.integers(-4, 5, (n, k)).astype(np.int8)
    s = _f16(rng.uniform(1e-3, 1e-1, (n, 2)))
    x = rng.standard_normal((1, k)).astype(np.float32)
    q, d, _ = o.quantize(x)
    y, a = o.gemv(c, s, q, d)
    ex = brute.gemv_exact(c.tolist(), s.tolist(), q[0].tolist(), d[0].tolist())
    for r in range(n):
        assert abs(Fraction(float(y[0, r])) - ex[r]) <= Fraction(float(a[0, r])) * Fraction(1, 2 ** 50)


# --------------------------------------------------------------------------------------
# Free-scale two-plane pass (Sec. 2.1 alpha1*T1 + alpha2*T2; Sec. 4.1: the planes stored
# apart, 4.125 bits/weight, one integer pass per plane)
# --------------------------------------------------------------------------------------

def _planes(rng, n, k):
    return (rng.integers(-1, 2, (n, k)).astype(np.int8), rng.integers(-1, 2, (n, k)).astype(np.int8))


@pin
def gemv2_plane_sums_scales_and_quantization_bound(o):
    # isum per plane against numpy int64 matmuls; absref against the terms rebuilt from
    # numpy's f16 decode; y against the dequantized two-plane matmul within the
    # activation quantizer's error bound (|x - d q| <= d (0.5 + 2^-14) per element).
    rng = np.random.default_rng(61)
    n, k, t = 6, 1024, 3
    t1, t2 = _planes(rng, n, k)
    a = _f16(np.exp(rng.uniform(np.log(1e-3), np.log(1e-1), (n, k // 256, 2))))
    x = rng.standard_normal((t, k)).astype(np.float32)
    q, d, _ = o.quantize(x)
    y, ab, isum = o.gemv2(t1, t2, a, q, d, want_isum=True)
    af = _f16_to_np64(a)
    terms = np.zeros((t, n))
    for b in range(k // 256):
        sl = slice(b * 256, (b + 1) * 256)
        for p_, tp in enumerate((t1, t2)):
            ref = q[:, sl].astype(np.int64) @ tp[:, sl].T.astype(np.int64)
            assert np.array_equal(isum[:, :, b, p_], ref)
            terms += np.abs(af[None, :, b, p_] * d[:, b, None].astype(np.float64) * ref)
    assert np.allclose(ab, terms, rtol=1e-12, atol=0)
    W = np.repeat(af[:, :, 0], 256, axis=1) * t1 + np.repeat(af[:, :, 1], 256, axis=1) * t2
    ref = x.astype(np.float64) @ W.T
    absw = np.abs(W).reshape(n, k // 256, 256).sum(2)
    bound = (d.astype(np.float64)[:, None, :] * absw[None]).sum(2) * (0.5 + 2 ** -14)
    assert np.all(np.abs(y - ref) <= bound * (1 + 1e-9) + 1e-12)
    bad = t1.copy(); bad[2, 5] = 2
    try:
        o.gemv2(bad, t2, a, q, d)
    except Exception:  # noqa: BLE001 - the oracle must refuse a value outside -1..1
        pass
    else:
        raise AssertionError("gemv2 accepted a trit outside -1..1")


@pin
def gemv2_tied_scales_reproduce_the_folded_pass(o):
    # alpha = (3s, s) with 3s exact in f16 (fraction bits a multiple of 4): the block sums
    # meet the fold identity 3(T1.q) + (T2.q) = c.q exactly, checked with numpy on the
    # folded codes, and y equals the folded pass up to fp64 rounding.
    rng = np.random.default_rng(67)
    n, k, t = 5, 768, 2
    t1, t2 = _planes(rng, n, k)
    c = (3 * t1.astype(np.int16) + t2).astype(np.int8)
    s = (rng.integers(0x1419, 0x2E66, (n, k // 256)) & ~3).astype(np.uint16)
    s3 = _f16(3 * _f16_to_np64(s))
    assert np.array_equal(_f16_to_np64(s3), 3 * _f16_to_np64(s))
    a = np.stack([s3, s], axis=2)
    x = rng.standard_normal((t, k)).astype(np.float32)
    q, d, _ = o.quantize(x)
    y2, ab2, isum = o.gemv2(t1, t2, a, q, d, want_isum=True)
    for b in range(k // 256):
        sl = slice(b * 256, (b + 1) * 256)
        folded = q[:, sl].astype(np.int64) @ c[:, sl].T.astype(np.int64)
        assert np.array_equal(3 * isum[:, :, b, 0].astype(np.int64) + isum[:, :, b, 1], folded)
    sf = _f16_to_np64(s)
    yf = np.zeros((t, n))
    for b in range(k // 256):
        sl = slice(b * 256, (b + 1) * 256)
        yf += sf[None, :, b] * d[:, b, None].astype(np.float64) * (q[:, sl].astype(np.int64) @ c[:, sl].T.astype(np.int64))
    assert np.all(np.abs(y2 - yf) <= ab2 * 2.0 ** -45)


@pin
def gemv2_one_empty_plane_is_one_ternary_pass(o):
    # With T2 = 0 the pass is the single-plane pass over T1 at scale alpha1 (codes in
    # -1..1 are valid nine-level codes), term for term; likewise T1 = 0 with alpha2.
    rng = np.random.default_rng(71)
    n, k, t = 4, 512, 2
    t1, t2 = _planes(rng, n, k)
    z = np.zeros_like(t1)
    a = _f16(rng.uniform(1e-3, 1e-1, (n, k // 256, 2)))
    x = rng.standard_normal((t, k)).astype(np.float32)
    q, d, _ = o.quantize(x)
    for keep, p_ in ((t1, 0), (t2, 1)):
        planes = (keep, z) if p_ == 0 else (z, keep)
        y2, ab2 = o.gemv2(*planes, a, q, d)
        y1, ab1 = o.gemv(keep, np.ascontiguousarray(a[:, :, p_]), q, d)
        assert np.array_equal(y2, y1) and np.array_equal(ab2, ab1)


@pin
def gemv2_plane_exchange_and_sign_symmetry(o):
    rng = np.random.default_rng(73)
    n, k, t = 4, 512, 2
    t1, t2 = _planes(rng, n, k)
    a = _f16(rng.uniform(1e-3, 1e-1, (n, k // 256, 2)))
    x = rng.standard_normal((t, k)).astype(np.float32)
    q, d, _ = o.quantize(x)
    y, ab, isum = o.gemv2(t1, t2, a, q, d, want_isum=True)
    ys, abs_, isums = o.gemv2(t2, t1, np.ascontiguousarray(a[:, :, ::-1]), q, d, want_isum=True)
    assert np.array_equal(isums, isum[..., ::-1])
    assert np.all(np.abs(ys - y) <= ab * 2.0 ** -50) and np.allclose(abs_, ab, rtol=1e-14)
    neg = a.copy(); neg[:, :, 1] ^= 0x8000  # -alpha2 with -T2: every term unchanged
    yn, abn, isn = o.gemv2(t1, (-t2).astype(np.int8), neg, q, d, want_isum=True)
    assert np.array_equal(yn, y) and np.array_equal(abn, ab)
    assert np.array_equal(isn[..., 1], -isum[..., 1]) and np.array_equal(isn[..., 0], isum[..., 0])


@pin
def gemv2_matches_exact_rational_brute_force(o):
    rng = np.random.default_rng(79)
    n, k = 3, 512
    t1, t2 = _planes(rng, n, k)
    a = _f16(rng.uniform(1e-3, 1e-1, (n, k // 256, 2)))
    x = rng.standard_normal((1, k)).astype(np.float32)
    q, d, _ = o.quantize(x)
    y, ab = o.gemv2(t1, t2, a, q, d)
    ex = brute.gemv2_exact(t1.tolist(), t2.tolist(), a.tolist(), q[0].tolist(), d[0].tolist())
    for r in range(n):
        assert abs(Fraction(float(y[0, r])) - ex[r]) <= Fraction(float(ab[0, r])) * Fraction(1, 2 ** 50)


# --------------------------------------------------------------------------------------
# MXFP4 reference arm (Sec. 2.3: doubled-e2m1 integers, e8m0 scale per 32 absorbing /2)
# --------------------------------------------------------------------------------------

def _paper_e2m1_values():
    """e2m1 values of codes 0..15 from the paper's doubled set (Sec. 2.3) halved; codes
    8..15 are the negatives (the format's top bit is the sign)."""
    mags = [Fraction(v, 2) for v in GOLDEN["doubled_e2m1_magnitudes"]["values"]]
    return mags + [-m for m in mags]


@pin
def e2m1_decodes_match_the_paper_set(o):
    doubled = GOLDEN["doubled_e2m1_magnitudes"]["values"]
    assert [o.e2m1_doubled(c) for c in range(8)] == doubled
    assert [o.e2m1_doubled(c | 8) for c in range(8)] == [-v for v in doubled]
    vals = _paper_e2m1_values()
    for c in range(16):
        assert Fraction(o.e2m1_to_f64(c)) == vals[c]
        assert 2 * Fraction(o.e2m1_to_f64(c)) == o.e2m1_doubled(c)
    assert np.signbit(o.e2m1_to_f64(8))  # the sign bit of code 8 is a negative zero


@pin
def e8m0_matches_numpy_ldexp(o):
    for e in range(255):
        assert o.e8m0_to_f64(e) == float(np.ldexp(1.0, e - 127))
    assert np.isnan(o.e8m0_to_f64(255))


def _mx_case(rng, n, k, t):
    c4 = rng.integers(0, 16, (n, k)).astype(np.uint8)
    e8 = rng.integers(110, 135, (n, k // 32)).astype(np.uint8)
    x = rng.standard_normal((t, k)).astype(np.float32)
    return c4, e8, x


@pin
def gemv_mx_block_sums_and_exponent_steps(o):
    rng = np.random.default_rng(83)
    n, k, t = 5, 512, 3
    c4, e8, x = _mx_case(rng, n, k, t)
    q, d, _ = o.quantize(x)
    y, ab, isum = o.gemv_mx(c4, e8, q, d, want_isum=True)
    dbl = np.array([int(2 * v) for v in _paper_e2m1_values()], dtype=np.int64)[c4]
    for j in range(k // 32):
        sl = slice(32 * j, 32 * (j + 1))
        assert np.array_equal(isum[:, :, j], q[:, sl].astype(np.int64) @ dbl[:, sl].T)
    e2 = e8.copy(); e2[3] += 1  # every block scale of row 3 doubled: y doubles exactly
    y2, ab2 = o.gemv_mx(c4, e2, q, d)
    assert np.array_equal(y2[:, 3], 2 * y[:, 3]) and np.array_equal(np.delete(y2, 3, 1), np.delete(y, 3, 1))
    e3 = e8.copy(); e3[1, 5] += 2  # one 32-block of row 1 times 4
    y3, _ = o.gemv_mx(c4, e3, q, d)
    term = np.ldexp(1.0, int(e8[1, 5]) - 128) * d[:, 0].astype(np.float64) * isum[:, 1, 5]
    assert np.allclose(y3[:, 1] - y[:, 1], 3 * term, rtol=1e-12, atol=1e-300)
    assert np.all(np.abs(y) <= ab * (1 + 1e-15))
    for bad_c4, bad_e8 in ((np.where(c4 == 3, 16, c4).astype(np.uint8), e8), (c4, np.full_like(e8, 255))):
        try:
            o.gemv_mx(bad_c4, bad_e8, q, d)
        except Exception:  # noqa: BLE001 - the oracle must refuse codes > 15 and NaN scales
            continue
        raise AssertionError("gemv_mx accepted an invalid code or a NaN scale")


@pin
def gemv_mx_absorbs_the_half_exactly(o):
    # the integer arm (doubled codes, 2^(E - 128)) equals the float-dequantized dot
    # (e2m1 values from the paper's set, 2^(E - 127)) in exact rational arithmetic
    rng = np.random.default_rng(89)
    n, k = 3, 512
    c4, e8, x = _mx_case(rng, n, k, 1)
    q, d, _ = o.quantize(x)
    y, ab = o.gemv_mx(c4, e8, q, d)
    ex = brute.gemv_mx_exact(_paper_e2m1_values(), c4.tolist(), e8.tolist(), q[0].tolist(), d[0].tolist())
    for r in range(n):
        assert abs(Fraction(float(y[0, r])) - ex[r]) <= Fraction(float(ab[0, r])) * Fraction(1, 2 ** 50)


# --------------------------------------------------------------------------------------
# Synthetic weight stream (input generation): SplitMix64 published outputs + recipe
# --------------------------------------------------------------------------------------

@pin
def splitmix64_known_answers(o):
    # SplitMix64 seeded with 0: first three outputs (Steele, Lea & Flood 2014 reference
    # generator as published with xorshift/xoshiro).
    assert [o.splitmix64_word(0, i) for i in range(3)] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]
    for key, i in ((12345, 0), (2 ** 63 + 7, 99), (2 ** 64 - 1, 2 ** 40)):
        assert o.splitmix64_word(key, i) == brute.splitmix64_word(key, i)


@pin
def synth_matrix_follows_recipe(o):
    key, n, k = 0xDEADBEEF12345678, 3, 512
    t1, t2, s = o.synth_matrix(key, n, k)
    for e in (0, 1, 2, 3, 511, 512, 1023, 1535):
        w = brute.splitmix64_word(key, e >> 1)
        sh = 32 if e & 1 else 0
        f1, f2 = (w >> sh) & 0xFFFF, (w >> (sh + 16)) & 0xFFFF
        assert t1.ravel()[e] == ((f1 * 3) >> 16) - 1 and t2.ravel()[e] == ((f2 * 3) >> 16) - 1
    for j in (0, 1, 5):
        w = brute.splitmix64_word(key, n * k // 2 + j)
        assert s.ravel()[j] == 0x1419 + (((w >> 32) * (0x2E66 - 0x1419 + 1)) >> 32)
    # a row window reproduces the same rows
    w1, w2, ws = o.synth_matrix(key, n, k, row0=1, rows=2)
    assert np.array_equal(w1, t1[1:]) and np.array_equal(w2, t2[1:]) and np.array_equal(ws, s[1:])


@pin
def synth_distributions(o):
    t1, t2, s = o.synth_matrix(0x1234, 64, 4096)
    for t in (t1, t2):
        f = np.bincount(t.ravel() + 1, minlength=3) / t.size
        assert set(np.unique(t).tolist()) == {-1, 0, 1} and np.all(np.abs(f - 1 / 3) < 0.005)
    c = o.fold(t1, t2)
    f = np.bincount(c.ravel() + 4, minlength=9) / c.size
    assert np.all(np.abs(f - 1 / 9) < 0.004)  # uniform nine-level codes
    v = _f16_to_np64(s)
    assert v.min() >= 1e-3 and v.max() <= 1e-1
    lg = np.log10(v.ravel())
    h = np.histogram(lg, bins=4, range=(-3, -1))[0] / lg.size
    assert np.all(np.abs(h - 0.25) < 0.05)  # log-uniform


# --------------------------------------------------------------------------------------
# Routed-expert layer (workload definition around the dot pass)
# --------------------------------------------------------------------------------------

def _tiny_experts(o, E=3, H=256, I=256, seed=41):
    rng = np.random.default_rng(seed)
    ex = {}
    for e in range(E):
        ex[e] = {p: (rng.integers(-4, 5, shape).astype(np.int8), _f16(rng.uniform(5e-3, 5e-2, (shape[0], shape[1] // 256))))
                 for p, shape in (("gate", (I, H)), ("up", (I, H)), ("down", (H, I)))}
    return ex


@pin
def silu_matches_scipy(o):
    from scipy.special import expit
    z = np.linspace(-30, 30, 601)
    assert np.allclose(o.silu(z), z * expit(z), rtol=1e-14, atol=1e-300)
    assert o.silu(np.array([0.0]))[0] == 0.0


@pin
def moe_matches_pure_python_brute_force(o):
    ex = _tiny_experts(o)
    rng = np.random.default_rng(43)
    x = (rng.standard_normal((2, 256)) * 3).astype(np.float32)
    idx = np.array([[2, 0], [1, 2]], np.int32)
    w = np.array([[0.75, 0.25], [0.4, 0.6]], np.float32)
    out, oa, _ = o.moe(x, idx, w, lambda e: ex[e])
    for t in range(2):
        ref = brute.moe_token(x[t], idx[t], w[t], {e: {p: (v[0].tolist(), v[1].tolist()) for p, v in ex[e].items()} for e in ex})
        assert np.all(np.abs(out[t] - np.array(ref)) <= 1e-9 * oa[t] + 1e-300)


@pin
def moe_invariants(o):
    ex = _tiny_experts(o, E=4)
    rng = np.random.default_rng(47)
    x = rng.standard_normal((3, 256)).astype(np.float32)
    idx = np.array([[0, 1, 2], [3, 2, 1], [1, 3, 0]], np.int32)
    w = rng.uniform(0.1, 1, (3, 3)).astype(np.float32)
    out, oa, _ = o.moe(x, idx, w, lambda e: ex[e])
    out2, _, _ = o.moe(x, idx, (2 * w).astype(np.float32), lambda e: ex[e])
    assert np.array_equal(out2, 2 * out)  # linear in the routing weights
    perm = [2, 0, 1]
    outp, _, _ = o.moe(x, idx[:, perm], w[:, perm], lambda e: ex[e])
    assert np.all(np.abs(outp - out) <= 1e-13 * oa)  # slot order only reorders a sum
    same = lambda e: ex[0]
    a1, _, _ = o.moe(x, idx, w, same)
    a2, _, _ = o.moe(x, (idx + 1) % 4, w, same)
    assert np.array_equal(a1, a2)  # identical experts: indices do not matter
    z, _, _ = o.moe(np.zeros_like(x), idx, w, lambda e: ex[e])
    assert not z.any()
    # top-1 with weight 1 is the plain expert chain
    o1, _, st = o.moe(x[:1], idx[:1, :1], np.ones((1, 1), np.float32), lambda e: ex[e])
    assert np.array_equal(o1[0], st[(0, 0)]["yd"])


# --------------------------------------------------------------------------------------
# Tied solver (Sec. 2.1: alternating updates against one scale = fitting W_hat = s*c)
# --------------------------------------------------------------------------------------

def _sq_err(w, c, s16):
    """Per-block squared error of s*c against w (fp64), [n][kb]."""
    n, k = w.shape
    sd = _f16_to_np64(s16)
    d = w.astype(np.float64).reshape(n, k // 256, 256) - sd[:, :, None] * c.reshape(n, k // 256, 256)
    return (d * d).sum(-1)


@pin
def f32_to_f16_matches_numpy(o):
    rng = np.random.default_rng(51)
    xs = (rng.standard_normal(4000) * 10.0 ** rng.uniform(-9, 4.8, 4000)).astype(np.float32)
    xs = xs[np.abs(xs) < 65504]
    # exact halfway cases between neighbouring f16 values, in normal and subnormal ranges
    half = [1 + 2 ** -11, 1 + 3 * 2 ** -11, 2 ** -14 + 2 ** -25, 3 * 2 ** -25, 2 ** -25, 2048 + 1, 2048 + 3]
    xs = np.concatenate([xs, np.array(half + [-h for h in half] + [65504.0, 65519.0, 0.0, -0.0], np.float32)])
    for x in xs:
        assert o.f32_to_f16(float(x)) == int(np.float32(x).astype(np.float16).view(np.uint16)), x
    for x in (65520.0, 1e6, -70000.0):  # saturation (numpy would give inf)
        assert o.f32_to_f16(x) == (0x7BFF | (0x8000 if x < 0 else 0))


@pin
def tied_recovers_exact_uniform_grid(o):
    # W = s*c with an f16 scale and +-4 present: the start is exact and the first scale
    # step reproduces it, so the codes, the scale and a two-step stop are all exact
    rng = np.random.default_rng(52)
    n, kb = 3, 4
    c = rng.integers(-4, 5, (n, kb * 256)).astype(np.int8)
    c[:, ::256] = 4 * np.where(rng.random((n, kb)) < 0.5, 1, -1)
    s = _f16_to_np64(_f16(np.exp(rng.uniform(np.log(1e-3), np.log(10), (n, kb))))).astype(np.float32)
    w = (np.repeat(s, 256, axis=1) * c).astype(np.float32)
    cc, ss, it = o.tied_quantize(w)
    assert np.array_equal(cc, c) and np.array_equal(ss, _f16(s)) and np.all(it == 2)


@pin
def tied_codes_are_the_best_levels_at_the_stored_scale(o):
    rng = np.random.default_rng(53)
    w = (rng.standard_normal((16, 4096)) * rng.uniform(0.01, 3, (16, 1))).astype(np.float32)
    c, s16, _ = o.tied_quantize(w)
    sd = np.repeat(_f16_to_np64(s16), 256, axis=1)
    e = (w.astype(np.float64) - sd * c) ** 2
    for v in range(-4, 5):  # exhaustive over the nine levels, element by element
        assert np.all(e <= (w.astype(np.float64) - sd * v) ** 2 * (1 + 1e-12) + 1e-300)


@pin
def tied_single_step_is_round_half_even_at_the_start_scale(o):
    # max_iter = 1: the scale stays amax/4 (f16-exact here) and the codes are the plain
    # rounding of w/s, halves to even
    s = 0.125
    w = np.array([4, -4, 0.5, 1.5, 2.5, -2.5, -3.5, 0.49, 3.7, -0.5] * 25 + [0.0] * 6, np.float32) * s
    w = np.tile(w, (2, 1))
    c, s16, it = o.tied_quantize(w, max_iter=1)
    assert np.all(it == 1) and np.all(_f16_to_np64(s16) == s)
    assert np.array_equal(c, np.clip(np.rint(w / np.float32(s)), -4, 4).astype(np.int8))


@pin
def tied_improves_on_the_start_and_nears_the_best_scale(o):
    rng = np.random.default_rng(54)
    w = rng.standard_normal((6, 256)).astype(np.float32)
    c, s16, _ = o.tied_quantize(w)
    err = _sq_err(w, c, s16)[:, 0]
    # the start: s = amax/4 (as f16), codes by rounding
    s0 = _f16(np.abs(w).max(1) / 4.0)
    c0 = np.clip(np.rint(w / _f16_to_np64(s0)[:, None]), -4, 4)
    err0 = _sq_err(w, c0, s0[:, None])[:, 0]
    assert np.all(err <= err0 * (1 + 1e-6))
    # brute force over every f16 scale in a wide range, codes chosen per element
    best = np.full(6, np.inf)
    for sb in range(0x1000, 0x4400):  # 2^-12 .. 4
        sd = float(np.uint16(sb).view(np.float16))
        cb = np.clip(np.rint(w / sd), -4, 4)
        best = np.minimum(best, ((w - sd * cb) ** 2).sum(1))
    # (alternating minimization stops at a local optimum: within 8% here, where the
    # start alone is 50-90% worse)
    assert np.all(err >= best * (1 - 1e-9)) and np.all(err <= best * 1.2)


@pin
def tied_invariants(o):
    rng = np.random.default_rng(55)
    w = (rng.standard_normal((3, 768)) * 0.05).astype(np.float32)
    w[1, 256:512] = 0.0                 # an all-zero block
    w[2, :256] = np.float32(2.0 ** -110)  # a block below the 2^-100 floor
    c, s16, it = o.tied_quantize(w)
    for r, b in ((1, 1), (2, 0)):
        assert s16[r, b] == 0 and it[r, b] == 0 and not c[r, 256 * b:256 * b + 256].any()
    cn, sn, _ = o.tied_quantize(-w)  # odd symmetry
    assert np.array_equal(cn, -c) and np.array_equal(sn, s16)
    c4, s4, _ = o.tied_quantize(w * np.float32(4))  # power-of-two equivariance
    keep = (s16 != 0) & (s16 < 0x7000)
    assert np.array_equal(c4, c)
    assert np.array_equal(_f16_to_np64(s4)[keep], 4 * _f16_to_np64(s16)[keep])
    perm = [2, 0, 1]  # blocks are independent of one another
    wp = w.reshape(3, 3, 256)[:, perm].reshape(3, 768)
    cp, sp, _ = o.tied_quantize(wp)
    assert np.array_equal(cp.reshape(3, 3, 256), c.reshape(3, 3, 256)[:, perm]) and np.array_equal(sp, s16[:, perm])
    c2, s2, it2 = o.tied_quantize(w)  # deterministic
    assert np.array_equal(c2, c) and np.array_equal(s2, s16) and np.array_equal(it2, it)


# --------------------------------------------------------------------------------------
# Free-scale solver (Sec. 2.1: PTQTP's alternation with two free scales; started from the
# tied fit, whose constrained family it contains)
# --------------------------------------------------------------------------------------

_FREE_ORDER = (0, -1, 1)


def _free_fit(o, w, max_iter=16):
    c, s, _ = o.tied_quantize(w)
    t1, t2, a, it = o.free_quantize(w, c, s, max_iter)
    return c, s, t1, t2, a, it


def _block_sq_errs(w, t1, t2, a, c, s):
    n, k = w.shape
    kb = k // 256
    W = w.astype(np.float64).reshape(n, kb, 256)
    af = _f16_to_np64(a)
    rf = t1.reshape(n, kb, 256) * af[:, :, 0, None] + t2.reshape(n, kb, 256) * af[:, :, 1, None]
    rt = c.astype(np.float64).reshape(n, kb, 256) * _f16_to_np64(s)[:, :, None]
    return ((W - rf) ** 2).sum(2), ((W - rt) ** 2).sum(2)


@pin
def free_planes_are_the_best_pairs_at_the_stored_scales(o):
    # 131072 weights, also stopped early (max_iter 2), so that many elements sit near a
    # decision boundary that moves when the scales are rounded to f16
    w = np.random.default_rng(97).standard_normal((32, 4096)).astype(np.float32) * np.float32(0.02)
    cands = [(x, y) for x in _FREE_ORDER for y in _FREE_ORDER]
    for max_iter in (16, 2):
        c, s, t1, t2, a, _ = _free_fit(o, w, max_iter)
        af = _f16_to_np64(a).astype(np.float32).astype(np.float64)
        a1 = np.repeat(af[:, :, 0], 256, axis=1)
        a2 = np.repeat(af[:, :, 1], 256, axis=1)
        errs = np.stack([np.abs(w.astype(np.float64) - (a1 * x + a2 * y)) for x, y in cands])  # [9][n][k]
        best = np.argmin(errs, axis=0)  # first minimum in the documented order
        assert np.array_equal(t1, np.array([c_[0] for c_ in cands])[best])
        assert np.array_equal(t2, np.array([c_[1] for c_ in cands])[best])


@pin
def free_first_scale_step_is_least_squares_on_the_tied_planes(o):
    rng = np.random.default_rng(101)
    w = (rng.standard_normal((4, 512)) * 0.03).astype(np.float32)
    c, s, _ = o.tied_quantize(w)
    _, _, a, it = o.free_quantize(w, c, s, max_iter=1)
    assert np.all(it == 1)
    t1, t2 = o.unfold(c)
    for r in range(4):
        for b in range(2):
            sl = slice(256 * b, 256 * (b + 1))
            A = np.stack([t1[r, sl], t2[r, sl]], axis=1).astype(np.float64)
            sol = np.linalg.lstsq(A, w[r, sl].astype(np.float64), rcond=None)[0]
            got = _f16_to_np64(a[r, b])
            assert np.all(np.abs(got - sol) <= np.abs(sol) * 2.0 ** -10), (r, b, got, sol)


@pin
def free_error_is_below_the_tied_fit(o):
    # started from the tied fit, each half-step is a least-squares optimum given the
    # other half: no block ends worse than the tied fit beyond the f16 rounding of its
    # two scales, and the matrix's error is strictly lower (the paper's observation)
    w = gen_float_weights(103, 32, 1024)
    c, s, t1, t2, a, _ = _free_fit(o, w)
    ef, et = _block_sq_errs(w, t1, t2, a, c, s)
    assert np.all(ef <= et * (1 + 2.0 ** -10))
    assert ef.sum() < et.sum() * (1 - 1e-4)


@pin
def free_recovers_a_tied_grid_exactly_and_invariants(o):
    rng = np.random.default_rng(107)
    n, k = 4, 768
    cc = rng.integers(-4, 5, (n, k)).astype(np.int8)
    cc[:, ::256] = 4  # every block reaches the outer level
    sb = (rng.integers(0x1C00, 0x2800, (n, k // 256)) & ~3).astype(np.uint16)  # 3s exact in f16
    w = (cc.astype(np.float64) * np.repeat(_f16_to_np64(sb), 256, axis=1)).astype(np.float32)
    w[1, 256:512] = 0.0  # a zero block
    c, s, t1, t2, a, it = _free_fit(o, w)
    ef, _ = _block_sq_errs(w, t1, t2, a, c, s)
    assert np.all(ef == 0.0)
    assert np.all(a[1, 1] == 0) and it[1, 1] == 0 and not t1[1, 256:512].any() and not t2[1, 256:512].any()
    live = np.ones((n, k // 256), bool); live[1, 1] = False
    assert np.array_equal(_f16_to_np64(a[..., 0])[live], 3 * _f16_to_np64(sb)[live])
    assert np.array_equal(a[..., 1][live], sb[live])
    # a zero tied scale gives a zero fit whatever codes come with it
    cz = c.copy(); cz[3, :256] = 3
    sz = s.copy(); sz[3, 0] = 0
    z = o.free_quantize(w, cz, sz)
    assert not z[0][3, :256].any() and not z[1][3, :256].any() and not z[2][3, 0].any() and z[3][3, 0] == 0
    # determinism and block independence: a row on its own gives the same fit
    again = o.free_quantize(w, c, s)
    assert all(np.array_equal(x, y) for x, y in zip(again, (t1, t2, a, it)))
    one = o.free_quantize(w[2:3], c[2:3], s[2:3])
    assert np.array_equal(one[0], t1[2:3]) and np.array_equal(one[2], a[2:3])


def gen_float_weights(seed, n, k):
    r = np.random.default_rng(seed)
    sigma = np.exp(np.log(0.005) + r.random((n, 1)) * (np.log(0.05) - np.log(0.005)))
    return (r.standard_normal((n, k)) * sigma).astype(np.float32)
