"""CPU oracle for the tied-trit-plane expert dot pass: Python side.

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this module. It wraps the plain C oracle
(``tq_oracle.c``) and strings its functions into the routed-expert MoE layer the
workloads define. It imports nothing from the HIP path.

Definitions followed (paper sections):
  fold / unfold ............ Sec. 2.1 (tied composite c = 3*t1 + t2), Sec. 2.2
  f16 scale, dequant ....... Sec. 2.1 (W_hat = s*c, scales serialized to f16)
  activation quantizer ..... Sec. 2.2 (block-quantized activations; block, scale and
                             rounding rule are this oracle's stated reading)
  integer dot + combine .... Sec. 2.2 (one integer dot pass, a single fp32
                             multiply-add for each block), evaluated exactly / in fp64
  MXFP4 arm ................ Sec. 2.3 (doubled-e2m1 integer dot, e8m0 scale per 32
                             absorbing the /2) with Sec. 2.1's description of the format
  free-scale solver ........ Sec. 2.1 (PTQTP's alternation with two free scales, started
                             from the tied fit; start, stop rule and precision are this
                             oracle's stated reading)
  free-scale two planes .... Sec. 2.1 (alpha1*T1 + alpha2*T2, free scales) and Sec. 4.1
                             (the unfolded pair is served as its two planes, stored
                             apart: 4.125 bits/weight, one integer pass per plane)
  tied solver .............. Sec. 2.1 (alternating code and scale updates against one
                             scale per group; start, stop rule and precision are this
                             oracle's stated reading)
  routed-expert layer ...... gate/up/down projections of the routed experts (Sec. 1,
                             Sec. 2.1: 43 layers x 3 projections x 256 experts); the
                             layer's glue (SiLU(gate)*up, requantized hidden, softmax-
                             weighted sum after down) is the workload's definition.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
DEFAULT_LIB = os.path.join(HERE, "liboracle.so")

_i64 = ctypes.c_int64
_vp = ctypes.c_void_p


def _p(a: np.ndarray) -> ctypes.c_void_p:
    assert a.flags["C_CONTIGUOUS"], "oracle buffers must be C-contiguous"
    return ctypes.c_void_p(a.ctypes.data)


class OracleError(RuntimeError):
    pass


class Oracle:
    """Handle on one build of the C oracle (tests may load mutated builds)."""

    def __init__(self, lib_path: str = DEFAULT_LIB):
        if not os.path.exists(lib_path):
            from . import build as _b
            _b.build(out=lib_path)
        L = ctypes.CDLL(lib_path)
        self._L = L
        for name, args, res in [
            ("orc_fold", [_vp, _vp, _i64, _vp], ctypes.c_int),
            ("orc_unfold", [_vp, _i64, _vp, _vp], ctypes.c_int),
            ("orc_two_plane_dequant", [_vp, _vp, _i64, ctypes.c_double, ctypes.c_double, _vp], ctypes.c_int),
            ("orc_f16_to_f64", [ctypes.c_uint16], ctypes.c_double),
            ("orc_dequant", [_vp, _vp, _i64, _i64, _vp], ctypes.c_int),
            ("orc_quantize", [_vp, _i64, _i64, _i64, _vp, _vp, _vp], ctypes.c_int),
            ("orc_dot_i8", [_vp, _vp, _i64], ctypes.c_int64),
            ("orc_gemv", [_vp, _vp, _i64, _i64, _vp, _vp, _i64, _vp, _vp, _vp], ctypes.c_int),
            ("orc_gemv2", [_vp, _vp, _vp, _i64, _i64, _vp, _vp, _i64, _vp, _vp, _vp], ctypes.c_int),
            ("orc_free_quantize", [_vp, _i64, _i64, ctypes.c_int, _vp, _vp, _vp, _vp, _vp, _vp], ctypes.c_int),
            ("orc_e2m1_to_f64", [ctypes.c_uint8], ctypes.c_double),
            ("orc_e2m1_doubled", [ctypes.c_uint8], ctypes.c_int),
            ("orc_e8m0_to_f64", [ctypes.c_uint8], ctypes.c_double),
            ("orc_gemv_mx", [_vp, _vp, _i64, _i64, _vp, _vp, _i64, _vp, _vp, _vp], ctypes.c_int),
            ("orc_splitmix64_word", [ctypes.c_uint64, ctypes.c_uint64], ctypes.c_uint64),
            ("orc_synth_matrix", [ctypes.c_uint64, _i64, _i64, _i64, _i64, _vp, _vp, _vp], ctypes.c_int),
            ("orc_f32_to_f16", [ctypes.c_float], ctypes.c_uint16),
            ("orc_tied_quantize", [_vp, _i64, _i64, ctypes.c_int, _vp, _vp, _vp], ctypes.c_int),
            ("orc_set_threads", [ctypes.c_int], ctypes.c_int),
        ]:
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res

    def set_threads(self, n: int = 0) -> int:
        """Threads of the row-parallel dot pass (n <= 0: leave as is); returns the count
        in effect."""
        return int(self._L.orc_set_threads(n))

    @staticmethod
    def _check(rc: int, what: str):
        if rc != 0:
            raise OracleError(f"{what}: invalid input (rc={rc})")

    # -- fold (Sec. 2.1) -------------------------------------------------------------
    def fold(self, t1, t2) -> np.ndarray:
        t1 = np.ascontiguousarray(t1, dtype=np.int8)
        t2 = np.ascontiguousarray(t2, dtype=np.int8)
        assert t1.shape == t2.shape
        c = np.empty_like(t1)
        self._check(self._L.orc_fold(_p(t1), _p(t2), t1.size, _p(c)), "fold")
        return c

    def unfold(self, c):
        c = np.ascontiguousarray(c, dtype=np.int8)
        t1 = np.empty_like(c)
        t2 = np.empty_like(c)
        self._check(self._L.orc_unfold(_p(c), c.size, _p(t1), _p(t2)), "unfold")
        return t1, t2

    def two_plane_dequant(self, t1, t2, alpha1: float, alpha2: float) -> np.ndarray:
        t1 = np.ascontiguousarray(t1, dtype=np.int8)
        t2 = np.ascontiguousarray(t2, dtype=np.int8)
        w = np.empty(t1.shape, dtype=np.float64)
        self._check(self._L.orc_two_plane_dequant(_p(t1), _p(t2), t1.size, alpha1, alpha2, _p(w)), "two_plane_dequant")
        return w

    # -- f16 scales and dequant (Sec. 2.1) ------------------------------------------
    def f16_to_f64(self, bits) -> np.ndarray:
        bits = np.asarray(bits, dtype=np.uint16).ravel()
        return np.array([self._L.orc_f16_to_f64(int(b)) for b in bits], dtype=np.float64)

    def dequant(self, c, s) -> np.ndarray:
        c = np.ascontiguousarray(c, dtype=np.int8)
        s = np.ascontiguousarray(s, dtype=np.uint16)
        n, k = c.shape
        assert s.shape == (n, k // 256)
        w = np.empty((n, k), dtype=np.float64)
        self._check(self._L.orc_dequant(_p(c), _p(s), n, k, _p(w)), "dequant")
        return w

    # -- activation quantizer (Sec. 2.2, reading stated in tq_oracle.c) --------------
    def quantize(self, x, blk: int = 256):
        x = np.ascontiguousarray(x, dtype=np.float32)
        if x.ndim == 1:
            x = x[None, :]
        t, k = x.shape
        q = np.empty((t, k), dtype=np.int8)
        d = np.empty((t, k // blk), dtype=np.float32)
        bs = np.empty((t, k // blk), dtype=np.int32)
        self._check(self._L.orc_quantize(_p(x), t, k, blk, _p(q), _p(d), _p(bs)), "quantize")
        return q, d, bs

    # -- integer dot and the serving pass (Sec. 2.2) ---------------------------------
    def dot_i8(self, a, b) -> int:
        a = np.ascontiguousarray(a, dtype=np.int8)
        b = np.ascontiguousarray(b, dtype=np.int8)
        assert a.size == b.size
        return int(self._L.orc_dot_i8(_p(a), _p(b), a.size))

    def gemv(self, c, s, q, d, want_isum: bool = False):
        """y[t][r], absref[t][r] in fp64 (and isum[t][r][b] int32 if asked)."""
        c = np.ascontiguousarray(c, dtype=np.int8)
        s = np.ascontiguousarray(s, dtype=np.uint16)
        q = np.ascontiguousarray(q, dtype=np.int8)
        d = np.ascontiguousarray(d, dtype=np.float32)
        if q.ndim == 1:
            q = q[None, :]
            d = d.reshape(1, -1)
        n, k = c.shape
        t = q.shape[0]
        assert q.shape == (t, k) and d.shape == (t, k // 256) and s.shape == (n, k // 256)
        y = np.empty((t, n), dtype=np.float64)
        a = np.empty((t, n), dtype=np.float64)
        isum = np.empty((t, n, k // 256), dtype=np.int32) if want_isum else None
        self._check(self._L.orc_gemv(_p(c), _p(s), n, k, _p(q), _p(d), t, _p(y), _p(a),
                                     _p(isum) if want_isum else None), "gemv")
        return (y, a, isum) if want_isum else (y, a)

    def gemv2(self, t1, t2, a, q, d, want_isum: bool = False):
        """Free-scale two-plane pass: t1, t2 trit planes [n][k] in -1..1, a f16 bits
        [n][k/256][2] (alpha1, alpha2). y[t][r], absref[t][r] in fp64 (and isum
        [t][r][b][2] int32, plane 1 then plane 2, if asked)."""
        t1 = np.ascontiguousarray(t1, dtype=np.int8)
        t2 = np.ascontiguousarray(t2, dtype=np.int8)
        a = np.ascontiguousarray(a, dtype=np.uint16)
        q = np.ascontiguousarray(q, dtype=np.int8)
        d = np.ascontiguousarray(d, dtype=np.float32)
        if q.ndim == 1:
            q = q[None, :]
            d = d.reshape(1, -1)
        n, k = t1.shape
        t = q.shape[0]
        assert t2.shape == (n, k) and a.shape == (n, k // 256, 2)
        assert q.shape == (t, k) and d.shape == (t, k // 256)
        y = np.empty((t, n), dtype=np.float64)
        ab = np.empty((t, n), dtype=np.float64)
        isum = np.empty((t, n, k // 256, 2), dtype=np.int32) if want_isum else None
        self._check(self._L.orc_gemv2(_p(t1), _p(t2), _p(a), n, k, _p(q), _p(d), t, _p(y), _p(ab),
                                      _p(isum) if want_isum else None), "gemv2")
        return (y, ab, isum) if want_isum else (y, ab)

    # -- MXFP4 reference arm (Sec. 2.3) ---------------------------------------------
    def e2m1_to_f64(self, code: int) -> float:
        return float(self._L.orc_e2m1_to_f64(code))

    def e2m1_doubled(self, code: int) -> int:
        return int(self._L.orc_e2m1_doubled(code))

    def e8m0_to_f64(self, e: int) -> float:
        return float(self._L.orc_e8m0_to_f64(e))

    def gemv_mx(self, c4, e8, q, d, want_isum: bool = False):
        """MXFP4 integer arm: c4 [n][k] e2m1 codes (0..15), e8 [n][k/32] e8m0 scales.
        y[t][r], absref[t][r] in fp64 (and isum [t][r][k/32] int32 if asked)."""
        c4 = np.ascontiguousarray(c4, dtype=np.uint8)
        e8 = np.ascontiguousarray(e8, dtype=np.uint8)
        q = np.ascontiguousarray(q, dtype=np.int8)
        d = np.ascontiguousarray(d, dtype=np.float32)
        if q.ndim == 1:
            q = q[None, :]
            d = d.reshape(1, -1)
        n, k = c4.shape
        t = q.shape[0]
        assert e8.shape == (n, k // 32) and q.shape == (t, k) and d.shape == (t, k // 256)
        y = np.empty((t, n), dtype=np.float64)
        ab = np.empty((t, n), dtype=np.float64)
        isum = np.empty((t, n, k // 32), dtype=np.int32) if want_isum else None
        self._check(self._L.orc_gemv_mx(_p(c4), _p(e8), n, k, _p(q), _p(d), t, _p(y), _p(ab),
                                        _p(isum) if want_isum else None), "gemv_mx")
        return (y, ab, isum) if want_isum else (y, ab)

    # -- synthetic weights (input generation; SplitMix64 counter stream) -------------
    # -- tied solver (Sec. 2.1) ---------------------------------------------------------
    def f32_to_f16(self, x: float) -> int:
        return int(self._L.orc_f32_to_f16(ctypes.c_float(x)))

    def tied_quantize(self, w, max_iter: int = 16):
        """W [n][k] fp32 -> (codes int8 [n][k] in -4..4, f16 scale bits [n][k/256],
        code steps taken per block)."""
        w = np.ascontiguousarray(w, dtype=np.float32)
        n, k = w.shape
        c = np.empty((n, k), dtype=np.int8)
        s = np.empty((n, k // 256), dtype=np.uint16)
        it = np.empty((n, k // 256), dtype=np.uint8)
        self._check(self._L.orc_tied_quantize(_p(w), n, k, max_iter, _p(c), _p(s), _p(it)), "tied_quantize")
        return c, s, it

    def free_quantize(self, w, c_tied, s_tied, max_iter: int = 16):
        """Free-scale fit started from a tied fit: W [n][k] fp32, the tied codes and f16
        scales -> (t1, t2 int8 [n][k], f16 scale pairs [n][k/256][2], plane steps per block)."""
        w = np.ascontiguousarray(w, dtype=np.float32)
        c_tied = np.ascontiguousarray(c_tied, dtype=np.int8)
        s_tied = np.ascontiguousarray(s_tied, dtype=np.uint16)
        n, k = w.shape
        assert c_tied.shape == (n, k) and s_tied.shape == (n, k // 256)
        t1 = np.empty((n, k), dtype=np.int8)
        t2 = np.empty((n, k), dtype=np.int8)
        a = np.empty((n, k // 256, 2), dtype=np.uint16)
        it = np.empty((n, k // 256), dtype=np.uint8)
        self._check(self._L.orc_free_quantize(_p(w), n, k, max_iter, _p(c_tied), _p(s_tied), _p(t1), _p(t2), _p(a),
                                              _p(it)), "free_quantize")
        return t1, t2, a, it

    def splitmix64_word(self, key: int, i: int) -> int:
        return int(self._L.orc_splitmix64_word(key & (2**64 - 1), i))

    def synth_matrix(self, key: int, n: int, k: int, row0: int = 0, rows: int | None = None):
        rows = n - row0 if rows is None else rows
        t1 = np.empty((rows, k), dtype=np.int8)
        t2 = np.empty((rows, k), dtype=np.int8)
        s = np.empty((rows, k // 256), dtype=np.uint16)
        self._check(self._L.orc_synth_matrix(key & (2**64 - 1), n, k, row0, rows, _p(t1), _p(t2), _p(s)), "synth")
        return t1, t2, s

    def synth_codes(self, key: int, n: int, k: int, row0: int = 0, rows: int | None = None):
        """Logical codes c = fold(t1, t2) [rows][k] and scales of a synthetic matrix."""
        t1, t2, s = self.synth_matrix(key, n, k, row0, rows)
        return self.fold(t1, t2), s

    # -- routed-expert MoE layer ------------------------------------------------------
    @staticmethod
    def silu(z):
        """SiLU(z) = z * sigmoid(z) = z / (1 + exp(-z)), fp64."""
        z = np.asarray(z, dtype=np.float64)
        return z / (1.0 + np.exp(-z))

    def expert_slot(self, ex: dict, x_row, want_isum: bool = False):
        """One (token, expert) slot: quantize x, gate/up dot pass, h = SiLU(g)*u,
        quantize h (as fp32), down dot pass. Returns a dict of every stage (with the exact
        block sums of the three dot passes, [rows][blocks] int32, if asked)."""
        qx, dx, bx = self.quantize(x_row)
        g, ga, gi = self.gemv(*ex["gate"], qx, dx, want_isum=True)
        u, ua, ui = self.gemv(*ex["up"], qx, dx, want_isum=True)
        h = self.silu(g[0]) * u[0]
        h32 = h.astype(np.float32)
        qh, dh, bh = self.quantize(h32)
        yd, ya, yi = self.gemv(*ex["down"], qh, dh, want_isum=True)
        st = dict(qx=qx[0], dx=dx[0], bx=bx[0], g=g[0], g_abs=ga[0], u=u[0], u_abs=ua[0],
                  h=h, qh=qh[0], dh=dh[0], bh=bh[0], yd=yd[0], yd_abs=ya[0])
        if want_isum:
            st.update(g_isum=gi[0], u_isum=ui[0], yd_isum=yi[0])
        return st

    def moe(self, x, idx, w, get_expert, tokens=None):
        """Routed-expert layer for the listed tokens (default: all).

        x [T][H] fp32; idx [T][topk] expert ids; w [T][topk] fp32 routing weights;
        get_expert(e) -> {"gate": (c, s), "up": (c, s), "down": (c, s)} logical codes.
        out[t] = sum_j w[t][j] * y_down(slot t,j), accumulated in ascending j (fp64).
        Returns (out [len(tokens)][H], out_abs, stages {(t, j): dict}).
        """
        x = np.asarray(x, dtype=np.float32)
        T, H = x.shape
        tokens = list(range(T)) if tokens is None else list(tokens)
        by_expert: dict[int, list] = {}
        for t in tokens:
            for j in range(idx.shape[1]):
                by_expert.setdefault(int(idx[t, j]), []).append((t, j))
        stages = {}
        for e in sorted(by_expert):
            ex = get_expert(e)
            for (t, j) in by_expert[e]:
                stages[(t, j)] = self.expert_slot(ex, x[t])
        out = np.zeros((len(tokens), H), dtype=np.float64)
        out_abs = np.zeros((len(tokens), H), dtype=np.float64)
        for n_t, t in enumerate(tokens):
            for j in range(idx.shape[1]):
                st = stages[(t, j)]
                out[n_t] += float(w[t, j]) * st["yd"]
                out_abs[n_t] += abs(float(w[t, j])) * st["yd_abs"]
        return out, out_abs, stages


_default: Oracle | None = None


def get() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default


def expert_getter(seed: int, layer: int, hidden: int, inter: int, oracle: Oracle | None = None):
    """get_expert(e) for the synthetic workloads: gate/up are [inter][hidden],
    down is [hidden][inter], drawn from the SplitMix64 streams keyed in synth.gen."""
    from synth import gen
    o = oracle or get()
    cache: dict[int, dict] = {}

    def get_expert(e: int) -> dict:
        if e not in cache:
            if len(cache) > 4:
                cache.clear()
            cache[e] = {
                "gate": o.synth_codes(gen.matrix_key(seed, layer, e, gen.PROJ_GATE), inter, hidden),
                "up": o.synth_codes(gen.matrix_key(seed, layer, e, gen.PROJ_UP), inter, hidden),
                "down": o.synth_codes(gen.matrix_key(seed, layer, e, gen.PROJ_DOWN), hidden, inter),
            }
        return cache[e]

    return get_expert
