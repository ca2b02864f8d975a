"""Pure-Python brute force for tiny cases (independent of the C oracle).

Integer work in Python ints, the scale combine in exact rational arithmetic, the
quantizer's fp32 decisions with numpy float32 scalars (IEEE single precision, round to
nearest even). Sizes stay tiny: this is a checker for the oracle, not a fast path.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np


def f16_exact(bits: int) -> Fraction:
    return Fraction(float(np.array([bits], dtype=np.uint16).view(np.float16)[0]))


def quantize_block(xs):
    xs = [np.float32(v) for v in xs]
    amax = np.float32(0)
    for v in xs:
        a = np.float32(abs(v))
        if a > amax:
            amax = a
    if amax == 0:
        return [0] * len(xs), np.float32(0), 0
    inv = np.float32(np.float32(127) / amax)
    d = np.float32(amax / np.float32(127))
    q = []
    for v in xs:
        r = int(np.rint(np.float32(v * inv)))
        q.append(max(-127, min(127, r)))
    return q, d, sum(q)


def quantize(x, blk=256):
    """x: list of floats (one token). Returns (q list, d list, bsum list)."""
    q, d, b = [], [], []
    for i in range(0, len(x), blk):
        qq, dd, bb = quantize_block(x[i:i + blk])
        q += qq
        d.append(dd)
        b.append(bb)
    return q, d, b


def gemv_exact(c, s, q, d):
    """c: rows of ints, s: rows of f16 bits, q: list of ints, d: list of fp32.
    Returns exact rational y per row."""
    k = len(q)
    out = []
    for r, row in enumerate(c):
        acc = Fraction(0)
        for b in range(k // 256):
            isum = sum(int(row[b * 256 + i]) * int(q[b * 256 + i]) for i in range(256))
            acc += f16_exact(int(s[r][b])) * Fraction(float(d[b])) * isum
        out.append(acc)
    return out


def gemv2_exact(t1, t2, a, q, d):
    """Free-scale two-plane pass. t1, t2: rows of trits, a: rows of [alpha1, alpha2]
    f16 bit pairs per block, q: list of ints, d: list of fp32. Exact rational y per row:
    sum over blocks of d * (alpha1 * (T1 . q) + alpha2 * (T2 . q))."""
    k = len(q)
    out = []
    for r in range(len(t1)):
        acc = Fraction(0)
        for b in range(k // 256):
            cols = range(b * 256, (b + 1) * 256)
            s1 = sum(int(t1[r][i]) * int(q[i]) for i in cols)
            s2 = sum(int(t2[r][i]) * int(q[i]) for i in cols)
            db = Fraction(float(d[b]))
            acc += db * (f16_exact(int(a[r][b][0])) * s1 + f16_exact(int(a[r][b][1])) * s2)
        out.append(acc)
    return out


def gemv_mx_exact(e2m1_values, c4, e8, q, d):
    """MXFP4 pass in exact rationals from the float decode: weights = e2m1 value (from
    the given 16-entry table) * 2^(E - 127), activations = d * q. c4: rows of codes, e8:
    rows of exponents per 32, q: list of ints, d: list of fp32 per 256."""
    k = len(q)
    out = []
    for r in range(len(c4)):
        acc = Fraction(0)
        for i in range(k):
            e = int(e8[r][i // 32]) - 127
            scale = Fraction(2) ** e
            acc += Fraction(e2m1_values[int(c4[r][i])]) * scale * Fraction(float(d[i // 256])) * int(q[i])
        out.append(acc)
    return out


def silu(z: float) -> float:
    return z / (1.0 + math.exp(-z))


def moe_token(x, idx_row, w_row, experts):
    """One token of the routed-expert layer; experts[e] = {"gate": (c, s), ...}.
    Returns the output as a list of floats (fp64 from exact partials)."""
    q, d, _ = quantize(list(x))
    out = [Fraction(0)] * len(x)
    for e, wj in zip(idx_row, w_row):
        ex = experts[int(e)]
        g = gemv_exact(*ex["gate"], q, d)
        u = gemv_exact(*ex["up"], q, d)
        h = [float(np.float32(silu(float(gi)) * float(ui))) for gi, ui in zip(g, u)]
        qh, dh, _ = quantize(h)
        yd = gemv_exact(*ex["down"], qh, dh)
        out = [o + Fraction(float(wj)) * v for o, v in zip(out, yd)]
    return [float(v) for v in out]


SM64_GAMMA = 0x9E3779B97F4A7C15
M64 = (1 << 64) - 1


def splitmix64_word(key: int, i: int) -> int:
    z = (key + (i + 1) * SM64_GAMMA) & M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)
