"""Host-side checks of the C-ABI library (no GPU needed): exports, persistent-format
arithmetic, host fold/pack against the oracle's fold, and argument validation."""
import ctypes
import json
import os
import re

import numpy as np
import pytest
import torch

from paper_2608_08910_amd import tq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = open(os.path.join(ROOT, "include", "tq.h")).read()
GOLDEN = json.load(open(os.path.join(ROOT, "tests", "golden", "paper_facts.json")))

no_gpu_only = pytest.mark.skipif(torch.cuda.is_available(),
                                 reason="feeds fake device pointers to validation paths; host-only")


def declared_functions():
    body = re.sub(r"/\*.*?\*/", "", HEADER, flags=re.S)
    return sorted(set(re.findall(r"\b(tq_[a-z0-9_]+)\s*\(", body)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 15
    lib = ctypes.CDLL(tq.LIB_PATH)
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_every_defined_entry_point_is_declared():
    # the reverse direction: an extern "C" definition in the sources without a declaration
    # in the header would be an entry point no C caller can see
    csrc = os.path.join(ROOT, "paper_2608_08910_amd", "csrc")
    defined = set()
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".hip", ".cpp")):
            src = open(os.path.join(csrc, f)).read()
            defined |= set(re.findall(r'extern "C"\s+[\w\s\*]*?\b(tq_[a-z0-9_]+)\s*\(', src))
    assert {"tq_quantize_act", "tq_gemv", "tq_moe_grouped"} <= defined
    missing = sorted(defined - set(declared_functions()))
    assert not missing, missing


@pytest.mark.parametrize("lang", ["c", "c++"])
def test_header_compiles_standalone(lang, tmp_path):
    import shutil
    import subprocess
    cc = shutil.which("gcc" if lang == "c" else "g++")
    if cc is None:
        pytest.skip("no host compiler")
    src = tmp_path / ("h.c" if lang == "c" else "h.cpp")
    src.write_text('#include "tq.h"\nint main(void) { return (int)sizeof(tq_experts) > 0 ? 0 : 1; }\n')
    r = subprocess.run([cc, "-fsyntax-only", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"), str(src)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_format_size_is_paper_bits_per_weight():
    bpw = GOLDEN["bits_per_weight"]
    assert bpw["tq2_0_fx4_block_bytes"] * 8 / bpw["tq2_0_fx4_block_weights"] == bpw["tq2_0_fx4"]
    for n, k in ((2048, 4096), (4096, 2048), (2048, 7168), (1, 256)):
        total = tq.tq_codes_bytes(n, k) + tq.tq_scales_bytes(n, k)
        assert total * 8 / (n * k) == bpw["tq2_0_fx4"]
    assert tq.tq_codes_bytes(4, 300) == 0 and tq.tq_scales_bytes(-1, 256) == 0


def test_pack_layout_bytes_hand_built():
    # one row, one block: column i holds code c_i; byte 16j+i must be
    # (c[32j+i] & 15) | (c[32j+16+i] & 15) << 4 (4-bit two's complement nibbles)
    cols = np.arange(256)
    c = ((cols * 7) % 9 - 4).astype(np.int8)
    t1 = np.floor_divide(c.astype(int) + 4, 3) - 1
    t2 = c.astype(int) - 3 * t1
    codes = tq.tq_fold_pack_host(t1.astype(np.int8)[None], t2.astype(np.int8)[None])
    for j in range(8):
        for i in range(16):
            want = (int(c[32 * j + i]) & 15) | ((int(c[32 * j + 16 + i]) & 15) << 4)
            assert codes[0, 0, 16 * j + i] == want
    # masking a byte's high nibble, or moving its low nibble up, gives 16c as int8
    b = codes[0, 0].astype(np.uint8)
    for j in range(8):
        hi16 = (b[16 * j:16 * j + 16] & 0xF0).view(np.int8).astype(int)
        lo16 = ((b[16 * j:16 * j + 16] << 4) & 0xF0).astype(np.uint8).view(np.int8).astype(int)
        assert np.array_equal(lo16, 16 * c[32 * j:32 * j + 16].astype(int))
        assert np.array_equal(hi16, 16 * c[32 * j + 16:32 * j + 32].astype(int))


def test_fold_pack_unpack_matches_oracle_fold(oracle):
    rng = np.random.default_rng(1)
    for n, k in ((3, 256), (5, 768), (2, 7168)):
        t1 = rng.integers(-1, 2, (n, k)).astype(np.int8)
        t2 = rng.integers(-1, 2, (n, k)).astype(np.int8)
        codes = tq.tq_fold_pack_host(t1, t2)
        assert codes.shape == (n, k // 256, 128)
        assert np.array_equal(tq.tq_unpack_host(codes, n, k), oracle.fold(t1, t2))
        for nib in (codes & 0xF, codes >> 4):  # nibbles of -4..4 only: 0..4, 12..15
            assert ((nib <= 4) | (nib >= 12)).all()


def test_fold_pack_rejects_bad_trits_and_unpack_bad_nibbles():
    t = np.zeros((1, 256), np.int8)
    bad = t.copy(); bad[0, 17] = 2
    with pytest.raises(tq.TqError) as e:
        tq.tq_fold_pack_host(bad, t)
    assert e.value.status == tq.TQ_ERR_INVALID and "trit" in str(e.value)
    codes = tq.tq_fold_pack_host(t, t)
    for bad_byte in (0x54, 0x0B, 0x84, 0x07):  # a nibble of 5, 11, 8 or 7: no code
        c2 = codes.copy()
        c2[0, 0, 5] = bad_byte
        with pytest.raises(tq.TqError):
            tq.tq_unpack_host(c2, 1, 256)
    c2 = codes.copy()
    c2[0, 0, 5] = 0xC4  # -4 and 4: valid
    assert tq.tq_unpack_host(c2, 1, 256)[0, 5] == 4 and tq.tq_unpack_host(c2, 1, 256)[0, 21] == -4


def test_two_plane_size_is_paper_bits_per_weight():
    # two trit planes at 2 bits plus two f16 scales per 256 weights (Table 1: 4.125)
    want = GOLDEN["bits_per_weight"]["free_scale_two_plane"]
    for n, k in ((2048, 4096), (4096, 2048), (1, 256)):
        total = tq.tq_codes_bytes(n, k) + 2 * tq.tq_scales_bytes(n, k)
        assert total * 8 / (n * k) == want


def test_pack2_layout_bytes_hand_built():
    # byte 16j + 8p + 4u + b, bits 2s..2s+1 = plane p's trit of column 32j + 16u + 4s + b,
    # 2-bit two's complement; shifted to the byte's top pair it reads as 64t
    cols = np.arange(256)
    t1 = ((cols * 5) % 3 - 1).astype(np.int8)
    t2 = ((cols * 7 + 1) % 3 - 1).astype(np.int8)
    codes = tq.tq_pack2_host(t1[None], t2[None])[0, 0]
    for j in range(8):
        for p, tp in enumerate((t1, t2)):
            for u in range(2):
                for b in range(4):
                    byte = int(codes[16 * j + 8 * p + 4 * u + b])
                    for sh in range(4):
                        col = 32 * j + 16 * u + 4 * sh + b
                        assert (byte >> (2 * sh)) & 3 == int(tp[col]) & 3
                        top = np.array([(byte << (6 - 2 * sh)) & 0xC0], np.uint8).view(np.int8)[0]
                        assert int(top) == 64 * int(tp[col])


def test_pack2_round_trip_and_rejections():
    rng = np.random.default_rng(5)
    for n, k in ((3, 256), (4, 768), (2, 7168)):
        t1 = rng.integers(-1, 2, (n, k)).astype(np.int8)
        t2 = rng.integers(-1, 2, (n, k)).astype(np.int8)
        codes = tq.tq_pack2_host(t1, t2)
        assert codes.shape == (n, k // 256, 128)
        u1, u2 = tq.tq_unpack2_host(codes, n, k)
        assert np.array_equal(u1, t1) and np.array_equal(u2, t2)
        pairs = np.stack([(codes >> (2 * s)) & 3 for s in range(4)])
        assert not (pairs == 2).any()  # the unused pattern never occurs
    z = np.zeros((1, 256), np.int8)
    bad = z.copy(); bad[0, 9] = -2
    with pytest.raises(tq.TqError) as e:
        tq.tq_pack2_host(z, bad)
    assert e.value.status == tq.TQ_ERR_INVALID and "trit" in str(e.value)
    codes = tq.tq_pack2_host(z, z)
    codes[0, 0, 3] = 0x08  # pattern 10 in bits 2..3
    with pytest.raises(tq.TqError):
        tq.tq_unpack2_host(codes, 1, 256)


def test_mx_size_is_paper_bits_per_weight():
    # 16 code bytes + 1 e8m0 byte per 32 weights (Sec. 2.3: 17-byte / 32-element blocks)
    bpw = GOLDEN["bits_per_weight"]
    assert bpw["mxfp4_block_bytes"] * 8 / bpw["mxfp4_block_weights"] == bpw["mxfp4"]
    for n, k in ((2048, 4096), (1, 256)):
        total = tq.tq_codes_bytes(n, k) + n * (k // 32)
        assert total * 8 / (n * k) == bpw["mxfp4"]


def test_mx_pack_layout_round_trip_and_rejections():
    # byte i of 16-byte block j: element 32j + i in the low nibble, 32j + 16 + i high
    rng = np.random.default_rng(9)
    c4 = rng.integers(0, 16, (3, 512)).astype(np.uint8)
    codes = tq.tq_mx_pack_host(c4)
    flat = codes.reshape(3, -1)
    for r in range(3):
        for j in range(512 // 32):
            for i in range(16):
                byte = int(flat[r, 16 * j + i])
                assert byte & 15 == c4[r, 32 * j + i] and byte >> 4 == c4[r, 32 * j + 16 + i]
    assert np.array_equal(tq.tq_mx_unpack_host(codes, 3, 512), c4)
    bad = c4.copy(); bad[1, 7] = 16
    with pytest.raises(tq.TqError) as e:
        tq.tq_mx_pack_host(bad)
    assert e.value.status == tq.TQ_ERR_INVALID


FAKE = 0x7F0000000000  # 256-byte aligned, never dereferenced: every call below is invalid


@no_gpu_only
def test_gemv_validation_errors_before_launch():
    L = tq._L
    cases = [
        (tq.tq_mat(0, 4096, FAKE, FAKE), 1, tq.TQ_ERR_INVALID),       # n < 1
        (tq.tq_mat(16, 300, FAKE, FAKE), 1, tq.TQ_ERR_INVALID),       # k % 256
        (tq.tq_mat(16, 32768, FAKE, FAKE), 1, tq.TQ_ERR_INVALID),     # k too large
        (tq.tq_mat(16, 4096, FAKE + 16, FAKE), 1, tq.TQ_ERR_ALIGN),   # codes alignment
        (tq.tq_mat(16, 4096, None, FAKE), 1, tq.TQ_ERR_INVALID),      # null codes
        (tq.tq_mat(16, 4096, FAKE, FAKE), -1, tq.TQ_ERR_INVALID),     # t < 0
    ]
    for m, t, want in cases:
        st = L.tq_gemv(ctypes.byref(m), FAKE, FAKE, FAKE, t, FAKE, None, None)
        assert st == want, (m.n, m.k, t, st, tq.tq_last_error())
        assert tq.tq_last_error()
    st = L.tq_gemv(ctypes.byref(tq.tq_mat(16, 4096, FAKE, FAKE)), FAKE + 4, FAKE, FAKE, 1, FAKE, None, None)
    assert st == tq.TQ_ERR_ALIGN  # q must be 16-byte aligned
    # t == 0 is a no-op that touches nothing
    assert L.tq_gemv(ctypes.byref(tq.tq_mat(16, 4096, FAKE, FAKE)), FAKE, FAKE, FAKE, 0, FAKE, None, None) == tq.TQ_OK


@no_gpu_only
def test_gemv2_validation_errors_before_launch():
    L = tq._L
    cases = [
        (tq.tq_mat2(0, 4096, FAKE, FAKE), 1, tq.TQ_ERR_INVALID),       # n < 1
        (tq.tq_mat2(16, 300, FAKE, FAKE), 1, tq.TQ_ERR_INVALID),       # k % 256
        (tq.tq_mat2(16, 32768, FAKE, FAKE), 1, tq.TQ_ERR_INVALID),     # k too large
        (tq.tq_mat2(16, 4096, FAKE + 16, FAKE), 1, tq.TQ_ERR_ALIGN),   # codes alignment
        (tq.tq_mat2(16, 4096, FAKE, FAKE + 2), 1, tq.TQ_ERR_ALIGN),    # scale pairs: 4 bytes
        (tq.tq_mat2(16, 4096, None, FAKE), 1, tq.TQ_ERR_INVALID),      # null codes
        (tq.tq_mat2(16, 4096, FAKE, FAKE), -1, tq.TQ_ERR_INVALID),     # t < 0
    ]
    for m, t, want in cases:
        st = L.tq_gemv2(ctypes.byref(m), FAKE, FAKE, t, FAKE, None, None)
        assert st == want, (m.n, m.k, t, st, tq.tq_last_error())
        assert tq.tq_last_error()
    assert L.tq_gemv2(ctypes.byref(tq.tq_mat2(16, 4096, FAKE, FAKE)), FAKE + 4, FAKE, 1, FAKE, None, None) == tq.TQ_ERR_ALIGN
    assert L.tq_gemv2(ctypes.byref(tq.tq_mat2(16, 4096, FAKE, FAKE)), FAKE, FAKE, 0, FAKE, None, None) == tq.TQ_OK


@no_gpu_only
def test_gemv_mx_validation_errors_before_launch():
    L = tq._L
    for m, t, want in [
        (tq.tq_mat_mx(0, 4096, FAKE, FAKE), 1, tq.TQ_ERR_INVALID),
        (tq.tq_mat_mx(16, 300, FAKE, FAKE), 1, tq.TQ_ERR_INVALID),
        (tq.tq_mat_mx(16, 32768, FAKE, FAKE), 1, tq.TQ_ERR_INVALID),
        (tq.tq_mat_mx(16, 4096, FAKE + 16, FAKE), 1, tq.TQ_ERR_ALIGN),
        (tq.tq_mat_mx(16, 4096, FAKE, None), 1, tq.TQ_ERR_INVALID),
        (tq.tq_mat_mx(16, 4096, FAKE, FAKE), -1, tq.TQ_ERR_INVALID),
    ]:
        st = L.tq_gemv_mx(ctypes.byref(m), FAKE, FAKE, t, FAKE, None, None)
        assert st == want, (m.n, m.k, t, st, tq.tq_last_error())
    assert L.tq_gemv_mx(ctypes.byref(tq.tq_mat_mx(16, 4096, FAKE, FAKE + 1)), FAKE + 4, FAKE, 1, FAKE, None, None) == tq.TQ_ERR_ALIGN
    assert L.tq_gemv_mx(ctypes.byref(tq.tq_mat_mx(16, 4096, FAKE, FAKE + 1)), FAKE, FAKE, 0, FAKE, None, None) == tq.TQ_OK


@no_gpu_only
def test_free_quantize_validation_errors_before_launch():
    L = tq._L
    ok = (FAKE, 4, 256, 16, FAKE, FAKE, FAKE, FAKE, None, None)
    def call(**kw):
        args = list(ok)
        for i, v in kw.items():
            args[int(i[1:])] = v
        return L.tq_free_quantize(*args)
    assert call(a2=300) == tq.TQ_ERR_INVALID          # k % 256
    assert call(a1=-1) == tq.TQ_ERR_INVALID           # n < 0
    assert call(a3=0) == tq.TQ_ERR_INVALID            # max_iter
    assert call(a3=256) == tq.TQ_ERR_INVALID
    assert call(a4=None) == tq.TQ_ERR_INVALID         # tied codes
    assert call(a6=FAKE + 64) == tq.TQ_ERR_ALIGN      # codes2
    assert call(a7=FAKE + 2) == tq.TQ_ERR_ALIGN       # scale pairs
    assert call(a5=FAKE + 1) == tq.TQ_ERR_ALIGN       # tied scales
    assert call(a1=0) == tq.TQ_OK                     # nothing to do


@no_gpu_only
def test_tied_quantize_validation_errors_before_launch():
    L = tq._L
    assert L.tq_tied_quantize(FAKE, 4, 300, 16, FAKE, FAKE, None, None) == tq.TQ_ERR_INVALID  # k % 256
    assert L.tq_tied_quantize(FAKE, -1, 256, 16, FAKE, FAKE, None, None) == tq.TQ_ERR_INVALID  # n < 0
    assert L.tq_tied_quantize(FAKE, 4, 256, 0, FAKE, FAKE, None, None) == tq.TQ_ERR_INVALID  # max_iter
    assert L.tq_tied_quantize(FAKE, 4, 256, 256, FAKE, FAKE, None, None) == tq.TQ_ERR_INVALID
    assert L.tq_tied_quantize(None, 4, 256, 16, FAKE, FAKE, None, None) == tq.TQ_ERR_INVALID
    assert L.tq_tied_quantize(FAKE, 4, 256, 16, FAKE + 64, FAKE, None, None) == tq.TQ_ERR_ALIGN  # codes
    assert L.tq_tied_quantize(FAKE + 2, 4, 256, 16, FAKE, FAKE, None, None) == tq.TQ_ERR_ALIGN  # w
    assert L.tq_tied_quantize(FAKE, 0, 256, 16, FAKE, FAKE, None, None) == tq.TQ_OK  # nothing to do
    assert "max_iter" in (L.tq_tied_quantize(FAKE, 4, 256, 0, FAKE, FAKE, None, None) and tq.tq_last_error())


def test_quantize_validation_errors_before_launch():
    L = tq._L
    assert L.tq_quantize_act(FAKE, 1, 300, FAKE, FAKE, FAKE, None) == tq.TQ_ERR_INVALID
    assert L.tq_quantize_act(FAKE, -1, 256, FAKE, FAKE, FAKE, None) == tq.TQ_ERR_INVALID
    assert L.tq_quantize_act(FAKE + 4, 1, 256, FAKE, FAKE, FAKE, None) == tq.TQ_ERR_ALIGN
    assert L.tq_quantize_act(None, 1, 256, FAKE, FAKE, FAKE, None) == tq.TQ_ERR_INVALID
    assert L.tq_quantize_act(FAKE, 0, 256, FAKE, FAKE, FAKE, None) == tq.TQ_OK


def _experts_desc(E=8, H=512, I=256):
    d = tq.tq_experts()
    d.n_experts, d.hidden, d.inter = E, H, I
    for name in ("gate_codes", "gate_scales", "up_codes", "up_scales", "down_codes", "down_scales"):
        setattr(d, name, FAKE)
    for p, (n, k) in enumerate(((I, H), (I, H), (H, I))):
        d.stride_codes[p] = n * k // 2
        d.stride_scales[p] = n * k // 256
    return d


@no_gpu_only
def test_moe_validation_errors_before_launch():
    L = tq._L

    def call(d, t=2, topk=2, ws_bytes=None, flags=0, x=FAKE, out=FAKE, ws=FAKE):
        if ws_bytes is None:
            ws_bytes = L.tq_moe_workspace_bytes(ctypes.byref(d), t, topk)
        return L.tq_moe_grouped(ctypes.byref(d), x, t, FAKE, FAKE, topk, out, ws, ws_bytes, flags, None)

    d = _experts_desc()
    need = L.tq_moe_workspace_bytes(ctypes.byref(d), 2, 2)
    assert need > 0
    assert call(d, ws_bytes=need - 1) == tq.TQ_ERR_WORKSPACE
    assert call(d, topk=9) == tq.TQ_ERR_INVALID          # topk > n_experts
    assert call(d, topk=0) == tq.TQ_ERR_INVALID
    assert call(d, t=-1) == tq.TQ_ERR_INVALID
    assert call(d, flags=3) == tq.TQ_ERR_INVALID
    assert call(d, flags=8) == tq.TQ_ERR_INVALID
    assert call(d, flags=3 | tq.TQ_MOE_DEBUG_STAGES) == tq.TQ_ERR_INVALID
    # the debug stage dump needs the layout's total_debug bytes: the plain size is refused
    lay = tq.tq_moe_layout()
    assert L.tq_moe_workspace_layout(ctypes.byref(d), 2, 2, ctypes.byref(lay)) == tq.TQ_OK
    assert call(d, flags=tq.TQ_MOE_DEBUG_STAGES, ws_bytes=need) == tq.TQ_ERR_WORKSPACE
    assert call(d, flags=tq.TQ_MOE_DEBUG_STAGES | tq.TQ_MOE_FORCE_MFMA, ws_bytes=lay.total_debug - 1) \
        == tq.TQ_ERR_WORKSPACE
    assert call(d, x=FAKE + 4) == tq.TQ_ERR_ALIGN
    assert call(d, ws=FAKE + 128) == tq.TQ_ERR_ALIGN
    assert call(d, x=None) == tq.TQ_ERR_INVALID
    bad = _experts_desc(H=300)
    assert call(bad) == tq.TQ_ERR_INVALID
    bad = _experts_desc(); bad.stride_codes[1] = 100
    assert call(bad) == tq.TQ_ERR_ALIGN
    bad = _experts_desc(E=0)
    assert call(bad) == tq.TQ_ERR_INVALID
    bad = _experts_desc(); bad.down_scales = None
    assert call(bad) == tq.TQ_ERR_INVALID
    assert call(d, t=0) == tq.TQ_OK                      # no-op


def test_moe_workspace_layout_is_consistent():
    d = _experts_desc(E=256, H=4096, I=2048)
    lay = tq.tq_moe_layout()
    assert tq._L.tq_moe_workspace_layout(ctypes.byref(d), 32, 8, ctypes.byref(lay)) == tq.TQ_OK
    S = 32 * 8
    offs = sorted((getattr(lay, n), n) for n in ("xq", "xd", "xb", "h", "hq", "hd", "hb", "yd"))
    sizes = {"xq": 32 * 4096, "xd": 32 * 16 * 4, "xb": 32 * 16 * 4, "h": S * 2048 * 4, "hq": S * 2048,
             "hd": S * 8 * 4, "hb": S * 8 * 4, "yd": S * 4096 * 4}
    for (o1, n1), (o2, _) in zip(offs, offs[1:]):
        assert o1 % 256 == 0 and o1 + sizes[n1] <= o2
    assert offs[-1][0] + sizes[offs[-1][1]] <= lay.total
    assert lay.total == tq._L.tq_moe_workspace_bytes(ctypes.byref(d), 32, 8)
    assert lay.flags < offs[0][0] and lay.n_active < offs[0][0]
    # dispatch lists before the stage buffers; the debug dump after them, within total_debug
    for n, sz in (("active", 256 * 4), ("act_off", 257 * 4), ("slot_list", S * 4)):
        assert getattr(lay, n) % 256 == 0 and getattr(lay, n) + sz <= offs[0][0]
    dbg = sorted((getattr(lay, n), n) for n in ("g", "u", "gsum", "usum", "dsum"))
    dsz = {"g": S * 2048 * 4, "u": S * 2048 * 4, "gsum": S * 2048 * 16 * 4, "usum": S * 2048 * 16 * 4,
           "dsum": S * 4096 * 8 * 4}
    assert dbg[0][0] >= lay.total
    for (o1, n1), (o2, _) in zip(dbg, dbg[1:]):
        assert o1 % 256 == 0 and o1 + dsz[n1] <= o2
    assert dbg[-1][0] + dsz[dbg[-1][1]] <= lay.total_debug


def test_moe_path_choice():
    L = tq._L

    def path(d, t, topk, flags=0):
        return L.tq_moe_path(ctypes.byref(d), t, topk, flags)

    d = _experts_desc(E=256, H=4096, I=2048)
    assert path(d, 1, 8) == tq.TQ_MOE_PATH_T1
    assert path(d, 1, 8, tq.TQ_MOE_FORCE_MFMA) == tq.TQ_MOE_PATH_MFMA
    assert path(d, 1, 8, tq.TQ_MOE_FORCE_VALU) == tq.TQ_MOE_PATH_T1
    assert path(d, 32, 8) == tq.TQ_MOE_PATH_MIXED
    assert path(d, 32, 8, tq.TQ_MOE_FORCE_VALU) == tq.TQ_MOE_PATH_VALU
    assert path(d, 32, 8, tq.TQ_MOE_FORCE_MFMA) == tq.TQ_MOE_PATH_MFMA
    assert path(d, 2, 8) == tq.TQ_MOE_PATH_VALU  # (2 tokens: no expert has more than 2 slots)
    assert path(d, 3, 8) == tq.TQ_MOE_PATH_MIXED and path(d, 255, 8) == tq.TQ_MOE_PATH_MIXED
    assert path(d, 256, 8) == tq.TQ_MOE_PATH_MFMA  # 2048 slots
    assert path(d, 2048, 8) == tq.TQ_MOE_PATH_MFMA
    assert path(d, 2048, 8, tq.TQ_MOE_FORCE_VALU) == tq.TQ_MOE_PATH_VALU
    deep = _experts_desc(E=256, H=7168, I=2048)
    assert path(deep, 8, 8) == tq.TQ_MOE_PATH_MIXED
    assert path(deep, 1, 8) == tq.TQ_MOE_PATH_T1
    wide = _experts_desc(E=8, H=4096, I=4096)
    assert path(wide, 1, 4) == tq.TQ_MOE_PATH_T1
    assert path(wide, 1, 5) == tq.TQ_MOE_PATH_VALU  # 5 x 4096 requantized bytes exceed the LDS budget
    assert path(d, 0, 8) == -1 and path(d, 1, 0) == -1
    # both grouped paths address activations with 32-bit offsets: at S * max(H, I) = 2^31
    # every grouped call is refused; one token fewer fits either path
    big = _experts_desc(E=256, H=16384, I=2048)
    t_lim = (1 << 31) // (16384 * 8)
    assert path(big, t_lim, 8) == -1
    assert path(big, t_lim, 8, tq.TQ_MOE_FORCE_VALU) == -1
    assert path(big, t_lim, 8, tq.TQ_MOE_FORCE_MFMA) == -1
    assert path(big, t_lim - 1, 8) == tq.TQ_MOE_PATH_MFMA
    assert path(big, t_lim - 1, 8, tq.TQ_MOE_FORCE_VALU) == tq.TQ_MOE_PATH_VALU


def test_pack_host_matches_fold_pack(oracle):
    """tq_pack_host (a folded code plane plus f16 scales) writes the same code bytes as
    the fold of the trit planes that give those codes, copies the scales, and refuses a
    code outside -4..4; the size helpers under the specification's names agree."""
    rng = np.random.default_rng(44)
    n, k = 5, 768
    t1 = rng.integers(-1, 2, (n, k)).astype(np.int8)
    t2 = rng.integers(-1, 2, (n, k)).astype(np.int8)
    s = rng.integers(0, 0x7BFF, (n, k // 256)).astype(np.uint16)
    codes, scales = tq.tq_pack_host(oracle.fold(t1, t2), s)
    assert np.array_equal(codes, tq.tq_fold_pack_host(t1, t2))
    assert np.array_equal(scales, s)
    bad = oracle.fold(t1, t2)
    bad[2, 300] = 5
    with pytest.raises(tq.TqError):
        tq.tq_pack_host(bad, s)
    assert tq._L.tq_packed_codes_bytes(n, k) == tq.tq_codes_bytes(n, k) == n * k // 2
    assert tq._L.tq_packed_scales_bytes(n, k) == tq.tq_scales_bytes(n, k) == n * (k // 256) * 2
