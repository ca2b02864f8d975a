"""Python binding of libtq (include/tq.h): argument marshalling only.

Every function here has the name of the C entry point it calls and does no compute of
its own: it checks dtypes, shapes, devices and contiguity, passes raw pointers and the
caller's HIP stream, and raises ``TqError`` on a non-zero status. PyTorch provides
device memory and streams. If ``libtq.so`` has not been built the import fails; there
is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# TQ_LIBRARY names an alternate build of the same library (e.g. one built with other tile
# shapes); by default the in-tree build is loaded.
LIB_PATH = os.environ.get("TQ_LIBRARY") or os.path.join(_HERE, "libtq.so")

TQ_OK = 0
TQ_ERR_INVALID = -1
TQ_ERR_ALIGN = -2
TQ_ERR_WORKSPACE = -3
TQ_ERR_DEVICE = -4
TQ_MOE_FORCE_VALU = 1
TQ_MOE_FORCE_MFMA = 2
TQ_MOE_DEBUG_STAGES = 4
TQ_MOE_PATH_T1, TQ_MOE_PATH_VALU, TQ_MOE_PATH_MFMA, TQ_MOE_PATH_MIXED = 0, 1, 2, 3


class TqError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


class tq_mat(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("k", ctypes.c_int32), ("codes", ctypes.c_void_p), ("scales", ctypes.c_void_p)]


class tq_mat2(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("k", ctypes.c_int32), ("codes", ctypes.c_void_p), ("scales", ctypes.c_void_p)]


class tq_mat_mx(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("k", ctypes.c_int32), ("codes", ctypes.c_void_p), ("scales", ctypes.c_void_p)]


class tq_experts(ctypes.Structure):
    _fields_ = [
        ("n_experts", ctypes.c_int32), ("hidden", ctypes.c_int32), ("inter", ctypes.c_int32),
        ("gate_codes", ctypes.c_void_p), ("gate_scales", ctypes.c_void_p),
        ("up_codes", ctypes.c_void_p), ("up_scales", ctypes.c_void_p),
        ("down_codes", ctypes.c_void_p), ("down_scales", ctypes.c_void_p),
        ("stride_codes", ctypes.c_int64 * 3), ("stride_scales", ctypes.c_int64 * 3),
    ]


class tq_moe_layout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_size_t) for n in ("xq", "xd", "xb", "h", "hq", "hd", "hb", "yd", "flags", "total",
                                               "n_active", "active", "act_off", "slot_list",
                                               "g", "u", "gsum", "usum", "dsum", "total_debug")]


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2608_08910_amd.build` (hipcc, gfx950)")

_L = ctypes.CDLL(LIB_PATH)
_vp, _i32, _i64, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
_P = ctypes.POINTER
for _name, _args, _res in [
    ("tq_codes_bytes", [_i32, _i32], _sz),
    ("tq_scales_bytes", [_i32, _i32], _sz),
    ("tq_fold_pack_host", [_vp, _vp, _i32, _i32, _vp], _i32),
    ("tq_unpack_host", [_vp, _i32, _i32, _vp], _i32),
    ("tq_packed_codes_bytes", [_i32, _i32], _sz),
    ("tq_packed_scales_bytes", [_i32, _i32], _sz),
    ("tq_pack_host", [_vp, _vp, _i32, _i32, _vp, _vp], _i32),
    ("tq_synth_weights", [ctypes.c_uint64, _i32, _i32, _vp, _vp, _vp], _i32),
    ("tq_quantize_act", [_vp, _i64, _i32, _vp, _vp, _vp, _vp], _i32),
    ("tq_tied_quantize", [_vp, _i32, _i32, _i32, _vp, _vp, _vp, _vp], _i32),
    ("tq_gemv", [_P(tq_mat), _vp, _vp, _vp, _i64, _vp, _vp, _vp], _i32),
    ("tq_gemv_timed", [_P(tq_mat), _vp, _vp, _vp, _i64, _vp, _vp, _vp, _P(_vp)], _i32),
    ("tq_gemv_f32", [_P(tq_mat), _vp, _i64, _vp, _vp, _vp, _vp, _vp, _vp], _i32),
    ("tq_gemv_f32_timed", [_P(tq_mat), _vp, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _P(_vp)], _i32),
    ("tq_pack2_host", [_vp, _vp, _i32, _i32, _vp], _i32),
    ("tq_unpack2_host", [_vp, _i32, _i32, _vp, _vp], _i32),
    ("tq_free_quantize", [_vp, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp], _i32),
    ("tq_gemv2", [_P(tq_mat2), _vp, _vp, _i64, _vp, _vp, _vp], _i32),
    ("tq_gemv2_timed", [_P(tq_mat2), _vp, _vp, _i64, _vp, _vp, _vp, _P(_vp)], _i32),
    ("tq_mx_pack_host", [_vp, _i32, _i32, _vp], _i32),
    ("tq_mx_unpack_host", [_vp, _i32, _i32, _vp], _i32),
    ("tq_gemv_mx", [_P(tq_mat_mx), _vp, _vp, _i64, _vp, _vp, _vp], _i32),
    ("tq_gemv_mx_timed", [_P(tq_mat_mx), _vp, _vp, _i64, _vp, _vp, _vp, _P(_vp)], _i32),
    ("tq_expert_record_bytes", [_i32, _i32], _sz),
    ("tq_experts_from_records", [_vp, _i32, _i32, _i32, _P(tq_experts)], _i32),
    ("tq_cache_state_bytes", [_i32, _i32], _sz),
    ("tq_cache_init", [_vp, _i32, _i32], _i32),
    ("tq_cache_map", [_vp, _vp, _i64, _vp, _vp, _P(_i32)], _i32),
    ("tq_cache_fetch", [_vp, _vp, _vp, _sz, _vp, _i32, _vp, _vp, _i64, _vp], _i32),
    ("tq_moe_workspace_bytes", [_P(tq_experts), _i64, _i32], _sz),
    ("tq_moe_path", [_P(tq_experts), _i64, _i32, _i32], _i32),
    ("tq_moe_workspace_layout", [_P(tq_experts), _i64, _i32, _P(tq_moe_layout)], _i32),
    ("tq_moe_grouped", [_P(tq_experts), _vp, _i64, _vp, _vp, _i32, _vp, _vp, _sz, _i32, _vp], _i32),
    ("tq_moe_grouped_timed", [_P(tq_experts), _vp, _i64, _vp, _vp, _i32, _vp, _vp, _sz, _i32, _vp, _P(_vp)], _i32),
    ("tq_stream_read_timed", [_vp, _sz, _vp, _vp, _P(_vp)], _i32),
    ("tq_moe_noalloc_max_bytes", [], _sz),
    ("tq_moe_grouped_noalloc", [_P(tq_experts), _vp, _i64, _vp, _vp, _i32, _vp, _i32, _vp], _i32),
    ("tq_moe_stage_count", [], _i32),
    ("tq_moe_stage_name", [_i32], ctypes.c_char_p),
    ("tq_moe_status", [_vp, _P(tq_experts), _i64, _i32, _P(_i32), _vp], _i32),
    ("tq_last_error", [], ctypes.c_char_p),
]:
    _f = getattr(_L, _name)
    _f.argtypes = _args
    _f.restype = _res


def tq_last_error() -> str:
    return _L.tq_last_error().decode()


def _ok(st: int):
    if st != TQ_OK:
        raise TqError(st, tq_last_error())


def _stream(stream) -> int | None:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _dev(t: torch.Tensor, dtype: torch.dtype, name: str, shape=None) -> int:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name}: expected a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected dtype {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    return t.data_ptr()


def _host(a: np.ndarray, dtype, name: str, shape=None) -> int:
    if not isinstance(a, np.ndarray) or a.dtype != dtype or not a.flags["C_CONTIGUOUS"]:
        raise TypeError(f"{name}: expected a C-contiguous numpy array of {np.dtype(dtype)}")
    if shape is not None and a.shape != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {a.shape}")
    return a.ctypes.data


# -- persistent format ------------------------------------------------------------------

def tq_codes_bytes(n: int, k: int) -> int:
    return int(_L.tq_codes_bytes(n, k))


def tq_scales_bytes(n: int, k: int) -> int:
    return int(_L.tq_scales_bytes(n, k))


def tq_fold_pack_host(t1: np.ndarray, t2: np.ndarray) -> np.ndarray:
    """Host fold + pack of trit planes [n][k] into codes [n][k/256][128] (uint8)."""
    n, k = t1.shape
    out = np.empty((n, k // 256, 128), dtype=np.uint8)
    _ok(_L.tq_fold_pack_host(_host(t1, np.int8, "t1"), _host(t2, np.int8, "t2", (n, k)), n, k, _host(out, np.uint8, "codes")))
    return out


def tq_pack_host(c: np.ndarray, s_f16: np.ndarray):
    """Host pack of a folded code plane c [n][k] (-4..4) and f16 scale bits [n][k/256]:
    returns (codes [n][k/256][128] uint8, scales [n][k/256] uint16)."""
    n, k = c.shape
    codes = np.empty((n, k // 256, 128), dtype=np.uint8)
    scales = np.empty((n, k // 256), dtype=np.uint16)
    _ok(_L.tq_pack_host(_host(c, np.int8, "c"), _host(s_f16, np.uint16, "s_f16", (n, k // 256)), n, k,
                        _host(codes, np.uint8, "codes"), _host(scales, np.uint16, "scales")))
    return codes, scales


def tq_unpack_host(codes: np.ndarray, n: int, k: int) -> np.ndarray:
    out = np.empty((n, k), dtype=np.int8)
    _ok(_L.tq_unpack_host(_host(codes, np.uint8, "codes"), n, k, _host(out, np.int8, "c_out")))
    return out


@dataclass
class TqMatrix:
    """One matrix in the persistent layout: codes [n][kb][128] uint8, scales [n][kb] int16
    (f16 bit patterns; torch has no uint16 arithmetic we need, int16 carries the bits)."""
    n: int
    k: int
    codes: torch.Tensor
    scales: torch.Tensor

    @staticmethod
    def empty(n: int, k: int, device="cuda") -> "TqMatrix":
        return TqMatrix(n, k, torch.empty((n, k // 256, 128), dtype=torch.uint8, device=device),
                        torch.empty((n, k // 256), dtype=torch.int16, device=device))

    def desc(self) -> tq_mat:
        _dev(self.codes, torch.uint8, "codes", (self.n, self.k // 256, 128))
        _dev(self.scales, torch.int16, "scales", (self.n, self.k // 256))
        return tq_mat(self.n, self.k, self.codes.data_ptr(), self.scales.data_ptr())


def tq_synth_weights(key: int, m: TqMatrix, stream=None):
    _ok(_L.tq_synth_weights(key & (2**64 - 1), m.n, m.k, _dev(m.codes, torch.uint8, "codes", (m.n, m.k // 256, 128)),
                            _dev(m.scales, torch.int16, "scales", (m.n, m.k // 256)), _stream(stream)))


def tq_tied_quantize(w: torch.Tensor, m: TqMatrix, iters: torch.Tensor | None = None, max_iter: int = 16,
                     stream=None):
    """Tied quantizer: w [n][k] fp32 -> m's codes and f16 scales; iters: None or a
    [n][k/256] uint8 tensor that receives the code steps taken per block."""
    n, k = w.shape
    if (m.n, m.k) != (n, k):
        raise ValueError(f"tq_tied_quantize: matrix is {m.n}x{m.k}, weights {n}x{k}")
    it = 0 if iters is None else _dev(iters, torch.uint8, "iters", (n, k // 256))
    _ok(_L.tq_tied_quantize(_dev(w, torch.float32, "w"), n, k, max_iter,
                            _dev(m.codes, torch.uint8, "codes", (n, k // 256, 128)),
                            _dev(m.scales, torch.int16, "scales", (n, k // 256)), it or None, _stream(stream)))


# -- dot pass -----------------------------------------------------------------------------

def tq_quantize_act(x: torch.Tensor, q: torch.Tensor, d: torch.Tensor, bsum: torch.Tensor, stream=None):
    t, k = x.shape
    _ok(_L.tq_quantize_act(_dev(x, torch.float32, "x"), t, k, _dev(q, torch.int8, "q", (t, k)),
                           _dev(d, torch.float32, "d", (t, k // 256)), _dev(bsum, torch.int32, "bsum", (t, k // 256)),
                           _stream(stream)))


def tq_gemv(m: TqMatrix, q: torch.Tensor, d: torch.Tensor, bsum: torch.Tensor, y: torch.Tensor,
            isum_dbg: torch.Tensor | None = None, stream=None):
    t = q.shape[0]
    desc = m.desc()
    dbg = None if isum_dbg is None else _dev(isum_dbg, torch.int32, "isum_dbg", (t, m.n, m.k // 256))
    _ok(_L.tq_gemv(ctypes.byref(desc), _dev(q, torch.int8, "q", (t, m.k)), _dev(d, torch.float32, "d", (t, m.k // 256)),
                   _dev(bsum, torch.int32, "bsum", (t, m.k // 256)), t, _dev(y, torch.float32, "y", (t, m.n)), dbg,
                   _stream(stream)))


def tq_gemv_timed(m: TqMatrix, q: torch.Tensor, d: torch.Tensor, bsum: torch.Tensor, y: torch.Tensor, events,
                  isum_dbg: torch.Tensor | None = None, stream=None):
    """events: two torch.cuda.Event(enable_timing=True) that receive the kernel's own start
    and stop timestamps."""
    if len(events) != 2:
        raise ValueError("need 2 events")
    for ev in events:  # torch creates the HIP event on its first record
        if ev.cuda_event == 0:
            ev.record()
    arr = (_vp * 2)(*[ev.cuda_event for ev in events])
    t = q.shape[0]
    desc = m.desc()
    dbg = None if isum_dbg is None else _dev(isum_dbg, torch.int32, "isum_dbg", (t, m.n, m.k // 256))
    _ok(_L.tq_gemv_timed(ctypes.byref(desc), _dev(q, torch.int8, "q", (t, m.k)), _dev(d, torch.float32, "d", (t, m.k // 256)),
                         _dev(bsum, torch.int32, "bsum", (t, m.k // 256)), t, _dev(y, torch.float32, "y", (t, m.n)), dbg,
                         _stream(stream), arr))


def _gemv_f32_args(m: TqMatrix, x, y, q, d, bsum, isum_dbg):
    t = x.shape[0]
    dbg = None if isum_dbg is None else _dev(isum_dbg, torch.int32, "isum_dbg", (t, m.n, m.k // 256))
    return (ctypes.byref(m.desc()), _dev(x, torch.float32, "x", (t, m.k)), t, _dev(y, torch.float32, "y", (t, m.n)),
            _dev(q, torch.int8, "q", (t, m.k)), _dev(d, torch.float32, "d", (t, m.k // 256)),
            _dev(bsum, torch.int32, "bsum", (t, m.k // 256)), dbg)


def tq_gemv_f32(m: TqMatrix, x: torch.Tensor, y: torch.Tensor, q: torch.Tensor, d: torch.Tensor, bsum: torch.Tensor,
                isum_dbg: torch.Tensor | None = None, stream=None):
    """The dot pass on fp32 activations (quantized in the same launch at one token);
    q, d, bsum receive the quantized activations."""
    _ok(_L.tq_gemv_f32(*_gemv_f32_args(m, x, y, q, d, bsum, isum_dbg), _stream(stream)))


def tq_gemv_f32_timed(m: TqMatrix, x: torch.Tensor, y: torch.Tensor, q: torch.Tensor, d: torch.Tensor,
                      bsum: torch.Tensor, events, isum_dbg: torch.Tensor | None = None, stream=None):
    if len(events) != 2:
        raise ValueError("need 2 events")
    for ev in events:
        if ev.cuda_event == 0:
            ev.record()
    arr = (_vp * 2)(*[ev.cuda_event for ev in events])
    _ok(_L.tq_gemv_f32_timed(*_gemv_f32_args(m, x, y, q, d, bsum, isum_dbg), _stream(stream), arr))


# -- free-scale two-plane variant -----------------------------------------------------------

def tq_pack2_host(t1: np.ndarray, t2: np.ndarray) -> np.ndarray:
    """Host pack of two trit planes [n][k] into two-plane codes [n][k/256][128] (uint8)."""
    n, k = t1.shape
    out = np.empty((n, k // 256, 128), dtype=np.uint8)
    _ok(_L.tq_pack2_host(_host(t1, np.int8, "t1"), _host(t2, np.int8, "t2", (n, k)), n, k, _host(out, np.uint8, "codes")))
    return out


def tq_unpack2_host(codes: np.ndarray, n: int, k: int):
    t1 = np.empty((n, k), dtype=np.int8)
    t2 = np.empty((n, k), dtype=np.int8)
    _ok(_L.tq_unpack2_host(_host(codes, np.uint8, "codes"), n, k, _host(t1, np.int8, "t1_out"), _host(t2, np.int8, "t2_out")))
    return t1, t2


@dataclass
class TqMatrix2:
    """One matrix in the two-plane layout: codes [n][kb][128] uint8, scales [n][kb][2]
    int16 (alpha1, alpha2 as f16 bit patterns)."""
    n: int
    k: int
    codes: torch.Tensor
    scales: torch.Tensor

    @staticmethod
    def empty(n: int, k: int, device="cuda") -> "TqMatrix2":
        return TqMatrix2(n, k, torch.empty((n, k // 256, 128), dtype=torch.uint8, device=device),
                         torch.empty((n, k // 256, 2), dtype=torch.int16, device=device))

    def desc(self) -> tq_mat2:
        _dev(self.codes, torch.uint8, "codes", (self.n, self.k // 256, 128))
        _dev(self.scales, torch.int16, "scales", (self.n, self.k // 256, 2))
        return tq_mat2(self.n, self.k, self.codes.data_ptr(), self.scales.data_ptr())


def tq_free_quantize(w: torch.Tensor, tied: TqMatrix, out: TqMatrix2, iters: torch.Tensor | None = None,
                     max_iter: int = 16, stream=None):
    """Free-scale solver: w [n][k] fp32 and its tied fit -> out's two planes and scale pairs;
    iters: None or a [n][k/256] uint8 tensor that receives the plane steps per block."""
    n, k = w.shape
    if (tied.n, tied.k) != (n, k) or (out.n, out.k) != (n, k):
        raise ValueError("tq_free_quantize: matrices must match the weights' shape")
    it = 0 if iters is None else _dev(iters, torch.uint8, "iters", (n, k // 256))
    _ok(_L.tq_free_quantize(_dev(w, torch.float32, "w"), n, k, max_iter,
                            _dev(tied.codes, torch.uint8, "tied codes", (n, k // 256, 128)),
                            _dev(tied.scales, torch.int16, "tied scales", (n, k // 256)),
                            _dev(out.codes, torch.uint8, "codes2", (n, k // 256, 128)),
                            _dev(out.scales, torch.int16, "scales2", (n, k // 256, 2)), it or None, _stream(stream)))


def _gemv2_args(m: TqMatrix2, q, d, y, isum_dbg):
    t = q.shape[0]
    desc = m.desc()
    dbg = None if isum_dbg is None else _dev(isum_dbg, torch.int32, "isum_dbg", (t, m.n, m.k // 256, 2))
    return (ctypes.byref(desc), _dev(q, torch.int8, "q", (t, m.k)), _dev(d, torch.float32, "d", (t, m.k // 256)), t,
            _dev(y, torch.float32, "y", (t, m.n)), dbg)


def tq_gemv2(m: TqMatrix2, q: torch.Tensor, d: torch.Tensor, y: torch.Tensor, isum_dbg: torch.Tensor | None = None,
             stream=None):
    _ok(_L.tq_gemv2(*_gemv2_args(m, q, d, y, isum_dbg), _stream(stream)))


def tq_gemv2_timed(m: TqMatrix2, q: torch.Tensor, d: torch.Tensor, y: torch.Tensor, events,
                   isum_dbg: torch.Tensor | None = None, stream=None):
    if len(events) != 2:
        raise ValueError("need 2 events")
    for ev in events:  # torch creates the HIP event on its first record
        if ev.cuda_event == 0:
            ev.record()
    arr = (_vp * 2)(*[ev.cuda_event for ev in events])
    _ok(_L.tq_gemv2_timed(*_gemv2_args(m, q, d, y, isum_dbg), _stream(stream), arr))


# -- MXFP4 reference arm ---------------------------------------------------------------------

def tq_mx_pack_host(c4: np.ndarray) -> np.ndarray:
    """Host pack of e2m1 codes [n][k] (0..15) into MXFP4 code bytes [n][k/256][128]."""
    n, k = c4.shape
    out = np.empty((n, k // 256, 128), dtype=np.uint8)
    _ok(_L.tq_mx_pack_host(_host(c4, np.uint8, "c4"), n, k, _host(out, np.uint8, "codes")))
    return out


def tq_mx_unpack_host(codes: np.ndarray, n: int, k: int) -> np.ndarray:
    out = np.empty((n, k), dtype=np.uint8)
    _ok(_L.tq_mx_unpack_host(_host(codes, np.uint8, "codes"), n, k, _host(out, np.uint8, "c4_out")))
    return out


@dataclass
class TqMatrixMx:
    """One matrix of the MXFP4 arm: codes [n][kb][128] uint8, scales [n][k/32] uint8 (e8m0)."""
    n: int
    k: int
    codes: torch.Tensor
    scales: torch.Tensor

    @staticmethod
    def empty(n: int, k: int, device="cuda") -> "TqMatrixMx":
        return TqMatrixMx(n, k, torch.empty((n, k // 256, 128), dtype=torch.uint8, device=device),
                          torch.empty((n, k // 32), dtype=torch.uint8, device=device))

    def desc(self) -> tq_mat_mx:
        _dev(self.codes, torch.uint8, "codes", (self.n, self.k // 256, 128))
        _dev(self.scales, torch.uint8, "scales", (self.n, self.k // 32))
        return tq_mat_mx(self.n, self.k, self.codes.data_ptr(), self.scales.data_ptr())


def _gemv_mx_args(m: TqMatrixMx, q, d, y, isum_dbg):
    t = q.shape[0]
    desc = m.desc()
    dbg = None if isum_dbg is None else _dev(isum_dbg, torch.int32, "isum_dbg", (t, m.n, m.k // 32))
    return (ctypes.byref(desc), _dev(q, torch.int8, "q", (t, m.k)), _dev(d, torch.float32, "d", (t, m.k // 256)), t,
            _dev(y, torch.float32, "y", (t, m.n)), dbg)


def tq_gemv_mx(m: TqMatrixMx, q: torch.Tensor, d: torch.Tensor, y: torch.Tensor, isum_dbg: torch.Tensor | None = None,
               stream=None):
    _ok(_L.tq_gemv_mx(*_gemv_mx_args(m, q, d, y, isum_dbg), _stream(stream)))


def tq_gemv_mx_timed(m: TqMatrixMx, q: torch.Tensor, d: torch.Tensor, y: torch.Tensor, events,
                     isum_dbg: torch.Tensor | None = None, stream=None):
    if len(events) != 2:
        raise ValueError("need 2 events")
    for ev in events:  # torch creates the HIP event on its first record
        if ev.cuda_event == 0:
            ev.record()
    arr = (_vp * 2)(*[ev.cuda_event for ev in events])
    _ok(_L.tq_gemv_mx_timed(*_gemv_mx_args(m, q, d, y, isum_dbg), _stream(stream), arr))


# -- routed-expert MoE layer ----------------------------------------------------------------

@dataclass
class TqExperts:
    """Routed experts of one layer, stacked: gate/up codes [E][inter][hidden/256][128],
    down codes [E][hidden][inter/256][128], scales likewise [E][rows][kb] (f16 bits)."""
    n_experts: int
    hidden: int
    inter: int
    codes: tuple  # (gate, up, down) uint8 tensors
    scales: tuple  # (gate, up, down) int16 tensors

    @staticmethod
    def empty(n_experts: int, hidden: int, inter: int, device="cuda") -> "TqExperts":
        shapes = [(inter, hidden), (inter, hidden), (hidden, inter)]
        codes = tuple(torch.empty((n_experts, n, k // 256, 128), dtype=torch.uint8, device=device) for n, k in shapes)
        scales = tuple(torch.empty((n_experts, n, k // 256), dtype=torch.int16, device=device) for n, k in shapes)
        return TqExperts(n_experts, hidden, inter, codes, scales)

    def shape(self, proj: int):
        return [(self.inter, self.hidden), (self.inter, self.hidden), (self.hidden, self.inter)][proj]

    def matrix(self, e: int, proj: int) -> TqMatrix:
        n, k = self.shape(proj)
        return TqMatrix(n, k, self.codes[proj][e], self.scales[proj][e])

    def desc(self) -> tq_experts:
        d = tq_experts()
        d.n_experts, d.hidden, d.inter = self.n_experts, self.hidden, self.inter
        for p, (cn, sn) in enumerate((("gate_codes", "gate_scales"), ("up_codes", "up_scales"), ("down_codes", "down_scales"))):
            n, k = self.shape(p)
            _dev(self.codes[p], torch.uint8, cn, (self.n_experts, n, k // 256, 128))
            _dev(self.scales[p], torch.int16, sn, (self.n_experts, n, k // 256))
            setattr(d, cn, self.codes[p].data_ptr())
            setattr(d, sn, self.scales[p].data_ptr())
            d.stride_codes[p] = n * (k // 256) * 128
            d.stride_scales[p] = n * (k // 256)
        return d


# -- host-tier expert streaming --------------------------------------------------------------

def tq_expert_record_bytes(hidden: int, inter: int) -> int:
    return int(_L.tq_expert_record_bytes(hidden, inter))


def tq_experts_from_records(base: int, n_records: int, hidden: int, inter: int) -> tq_experts:
    d = tq_experts()
    _ok(_L.tq_experts_from_records(base, n_records, hidden, inter, ctypes.byref(d)))
    return d


@dataclass
class TqExpertRecords:
    """Experts stored as contiguous records (one per expert, tq_expert_record_bytes each)
    in one uint8 tensor [n_records][record_bytes] (device: resident experts or the slot
    pool; pinned host: the host store). Usable wherever a TqExperts is."""
    n_experts: int
    hidden: int
    inter: int
    data: torch.Tensor

    @staticmethod
    def empty(n: int, hidden: int, inter: int, device="cuda", pin_memory: bool = False) -> "TqExpertRecords":
        rb = tq_expert_record_bytes(hidden, inter)
        if device == "cpu":
            data = torch.empty((n, rb), dtype=torch.uint8, pin_memory=pin_memory)
        else:
            data = torch.empty((n, rb), dtype=torch.uint8, device=device)
        return TqExpertRecords(n, hidden, inter, data)

    @property
    def record_bytes(self) -> int:
        return tq_expert_record_bytes(self.hidden, self.inter)

    def desc(self) -> tq_experts:
        if tuple(self.data.shape) != (self.n_experts, self.record_bytes) or self.data.dtype != torch.uint8 \
                or not self.data.is_contiguous():
            raise ValueError("records: expected a contiguous uint8 tensor [n][record_bytes]")
        return tq_experts_from_records(self.data.data_ptr(), self.n_experts, self.hidden, self.inter)


class TqCache:
    """The LRU slot planner's state (host memory) and its two calls."""

    def __init__(self, n_experts: int, n_slots: int):
        nb = int(_L.tq_cache_state_bytes(n_experts, n_slots))
        if nb == 0:
            raise TqError(TQ_ERR_INVALID, "tq_cache_state_bytes: invalid sizes")
        self.state = np.zeros((nb + 7) // 8, dtype=np.int64)
        self.n_experts, self.n_slots = n_experts, n_slots
        _ok(_L.tq_cache_init(self.state.ctypes.data, n_experts, n_slots))

    def map(self, ids: np.ndarray, slots_out: np.ndarray | None = None):
        """ids: int32 expert ids (any shape). Returns (slots, misses [m][2] (expert, slot))."""
        ids = np.ascontiguousarray(ids, dtype=np.int32)
        slots = np.empty(ids.shape, dtype=np.int32) if slots_out is None else slots_out
        if slots.shape != ids.shape or slots.dtype != np.int32 or not slots.flags["C_CONTIGUOUS"]:
            raise ValueError("slots_out: int32, C-contiguous, same shape as ids")
        misses = np.empty((max(ids.size, 1), 2), dtype=np.int32)
        nm = ctypes.c_int32(0)
        _ok(_L.tq_cache_map(self.state.ctypes.data, ids.ctypes.data, ids.size, slots.ctypes.data, misses.ctypes.data,
                            ctypes.byref(nm)))
        return slots, misses[:nm.value]

    def fetch(self, store: TqExpertRecords, pool: TqExpertRecords, misses: np.ndarray, slots_host: torch.Tensor,
              slots_dev: torch.Tensor, stream=None):
        """Enqueue the misses' record copies (host store -> device pool) and the slot ids
        (slots_host, a pinned int32 tensor -> slots_dev)."""
        misses = np.ascontiguousarray(misses, dtype=np.int32)
        if store.record_bytes != pool.record_bytes:
            raise ValueError("store and pool records differ")
        if slots_host.device.type != "cpu" or slots_host.dtype != torch.int32 or not slots_host.is_contiguous():
            raise TypeError("slots_host: a contiguous int32 host tensor (pinned for an asynchronous copy)")
        _dev(slots_dev, torch.int32, "slots_dev", tuple(slots_host.shape))
        _ok(_L.tq_cache_fetch(self.state.ctypes.data, store.data.data_ptr(), pool.data.data_ptr(), pool.record_bytes,
                              misses.ctypes.data if misses.size else None, misses.shape[0],
                              slots_host.data_ptr(), slots_dev.data_ptr(), slots_host.numel(), _stream(stream)))


def tq_moe_workspace_bytes(ex: TqExperts, t: int, topk: int) -> int:
    return int(_L.tq_moe_workspace_bytes(ctypes.byref(ex.desc()), t, topk))


def tq_moe_path(ex: TqExperts, t: int, topk: int, flags: int = 0) -> int:
    p = int(_L.tq_moe_path(ctypes.byref(ex.desc()), t, topk, flags))
    if p < 0:
        raise TqError(TQ_ERR_INVALID, tq_last_error())
    return p


def moe_workspace(ex: TqExperts, t: int, topk: int, device="cuda", debug: bool = False) -> torch.Tensor:
    """A device workspace for tq_moe_grouped: tq_moe_workspace_bytes(ex, t, topk) bytes, or
    with debug=True the layout's total_debug bytes (room for the TQ_MOE_DEBUG_STAGES dump)."""
    n = tq_moe_workspace_layout(ex, t, topk)["total_debug"] if debug else tq_moe_workspace_bytes(ex, t, topk)
    return torch.empty(n, dtype=torch.uint8, device=device)


def tq_moe_workspace_layout(ex: TqExperts, t: int, topk: int) -> dict:
    lay = tq_moe_layout()
    _ok(_L.tq_moe_workspace_layout(ctypes.byref(ex.desc()), t, topk, ctypes.byref(lay)))
    return {n: int(getattr(lay, n)) for n, _ in tq_moe_layout._fields_}


def _moe_args(ex, x, topk_idx, topk_w, out, ws):
    t, h = x.shape
    topk = topk_idx.shape[1]
    if h != ex.hidden:
        raise ValueError(f"x: hidden {h} != experts' hidden {ex.hidden}")
    return (ctypes.byref(ex.desc()), _dev(x, torch.float32, "x"), t, _dev(topk_idx, torch.int32, "topk_idx", (t, topk)),
            _dev(topk_w, torch.float32, "topk_w", (t, topk)), topk, _dev(out, torch.float32, "out", (t, h)),
            _dev(ws, torch.uint8, "ws"), ws.numel())


def tq_moe_grouped(ex: TqExperts, x, topk_idx, topk_w, out, ws, flags: int = 0, stream=None):
    _ok(_L.tq_moe_grouped(*_moe_args(ex, x, topk_idx, topk_w, out, ws), flags, _stream(stream)))


def tq_stream_read_timed(src: torch.Tensor, nbytes: int, sink: torch.Tensor, events, stream=None):
    """The benchmark's streaming-read ceiling: read nbytes from the start of src (a
    contiguous device tensor) in one launch, timed by events (two torch.cuda.Event)."""
    if not src.is_cuda or not src.is_contiguous() or src.numel() * src.element_size() < nbytes:
        raise ValueError("src: a contiguous device tensor of at least nbytes")
    _dev(sink, torch.int32, "sink")
    for ev in events:
        if ev.cuda_event == 0:
            ev.record()
    arr = (_vp * 2)(events[0].cuda_event, events[1].cuda_event)
    _ok(_L.tq_stream_read_timed(src.data_ptr(), nbytes, sink.data_ptr(), _stream(stream), arr))


def tq_moe_noalloc_max_bytes() -> int:
    return int(_L.tq_moe_noalloc_max_bytes())


def tq_moe_grouped_noalloc(ex: TqExperts, x, topk_idx, topk_w, out, flags: int = 0, stream=None):
    """tq_moe_grouped on the library's fixed per-device scratch array (no workspace)."""
    t, h = x.shape
    topk = topk_idx.shape[1]
    if h != ex.hidden:
        raise ValueError(f"x: hidden {h} != experts' hidden {ex.hidden}")
    _ok(_L.tq_moe_grouped_noalloc(ctypes.byref(ex.desc()), _dev(x, torch.float32, "x"), t,
                                  _dev(topk_idx, torch.int32, "topk_idx", (t, topk)),
                                  _dev(topk_w, torch.float32, "topk_w", (t, topk)), topk,
                                  _dev(out, torch.float32, "out", (t, h)), flags, _stream(stream)))


def tq_moe_stage_count() -> int:
    return int(_L.tq_moe_stage_count())


def tq_moe_stage_name(i: int) -> str:
    return _L.tq_moe_stage_name(i).decode()


def tq_moe_grouped_timed(ex: TqExperts, x, topk_idx, topk_w, out, ws, events, flags: int = 0, stream=None):
    """events: 2 * tq_moe_stage_count() torch.cuda.Event(enable_timing=True) objects;
    events[2i], events[2i+1] bracket stage i."""
    n = 2 * tq_moe_stage_count()
    if len(events) != n:
        raise ValueError(f"need {n} events")
    for ev in events:  # torch creates the HIP event on its first record
        if ev.cuda_event == 0:
            ev.record()
    arr = (_vp * n)(*[ev.cuda_event for ev in events])
    _ok(_L.tq_moe_grouped_timed(*_moe_args(ex, x, topk_idx, topk_w, out, ws), flags, _stream(stream), arr))


def tq_moe_status(ws, ex: TqExperts, t: int, topk: int, stream=None) -> int:
    v = ctypes.c_int32(0)
    _ok(_L.tq_moe_status(_dev(ws, torch.uint8, "ws"), ctypes.byref(ex.desc()), t, topk, ctypes.byref(v), _stream(stream)))
    return v.value
