"""GPU parity of the activation quantizer, the synthetic-weight generator and the single-
matrix dot pass (tq_quantize_act, tq_synth_weights, tq_gemv, and tq_gemv_f32 with the
quantization fused into the pass) against the CPU oracle.

Bar: quantized activations, block scales, block code sums, packed codes and the exact
int32 block sums are bit-exact; fp32 outputs agree within 1e-5 of the sum of the
absolute block terms (the order of the fp32 block sum is free on the GPU)."""
import numpy as np
import pytest
import torch

from gpu_util import announce, assert_close, device
from synth import gen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tq():
    device()
    from paper_2608_08910_amd import tq as _tq
    return _tq


def gpu_quantize(tq, x: np.ndarray):
    t, k = x.shape
    xd = torch.from_numpy(x).cuda()
    q = torch.empty((t, k), dtype=torch.int8, device="cuda")
    d = torch.empty((t, k // 256), dtype=torch.float32, device="cuda")
    b = torch.empty((t, k // 256), dtype=torch.int32, device="cuda")
    tq.tq_quantize_act(xd, q, d, b)
    torch.cuda.synchronize()
    return q, d, b


def special_blocks(k: int) -> np.ndarray:
    """Rows of hand-built edge blocks, tiled to width k."""
    rows = []
    z = np.zeros(256, np.float32)
    rows.append(z.copy())                                               # all zero
    r = z.copy(); r[:6] = [127, 0.5, 1.5, 2.5, -2.5, -0.5]; rows.append(r)  # unit scale, halves
    r = z.copy(); r[:4] = [254, 1, 3, -5]; rows.append(r)              # scale 2, halves
    r = z.copy(); r[100] = -3.0; rows.append(r)                         # one nonzero
    r = np.float32(2.0 ** -101) * np.linspace(-1, 1, 256, dtype=np.float32); rows.append(r)  # below 2^-100
    r = np.float32(2.0 ** -100) * np.linspace(-1, 1, 256, dtype=np.float32); rows.append(r)  # at 2^-100
    r = np.full(256, 1e30, np.float32); r[::2] *= -1; rows.append(r)    # huge, ties at amax
    r = np.full(256, -0.0, np.float32); r[7] = 1e-40; r[8] = 1.0; rows.append(r)  # -0 and a subnormal
    # row i, block b holds edge block (i + b) mod len(rows)
    out = np.zeros((len(rows), k), np.float32)
    for i in range(len(rows)):
        for b in range(k // 256):
            out[i, 256 * b:256 * (b + 1)] = rows[(i + b) % len(rows)]
    return out


@pytest.mark.parametrize("t,k", [(1, 256), (3, 4096), (37, 4096), (2, 16384), (5, 7168), (64, 2048)])
def test_quantize_bit_exact(tq, oracle, t, k):
    rng = np.random.default_rng(t * 1000 + k)
    x = rng.standard_normal((t, k)).astype(np.float32)
    x *= np.exp(rng.uniform(np.log(1e-3), np.log(1e3), (t, 1))).astype(np.float32)
    announce(f"quantize t={t} k={k}")
    q, d, b = gpu_quantize(tq, x)
    oq, od, ob = oracle.quantize(x)
    assert np.array_equal(q.cpu().numpy(), oq)
    assert np.array_equal(d.cpu().numpy().view(np.uint32), od.view(np.uint32))
    assert np.array_equal(b.cpu().numpy(), ob)


@pytest.mark.parametrize("k", [256, 2048, 4096])
def test_quantize_edge_blocks_bit_exact(tq, oracle, k):
    x = special_blocks(k)
    announce(f"quantize edge blocks k={k}")
    q, d, b = gpu_quantize(tq, x)
    oq, od, ob = oracle.quantize(x)
    assert np.array_equal(q.cpu().numpy(), oq)
    assert np.array_equal(d.cpu().numpy().view(np.uint32), od.view(np.uint32))
    assert np.array_equal(b.cpu().numpy(), ob)


def test_quantize_zero_tokens_is_noop(tq):
    x = torch.empty((0, 256), dtype=torch.float32, device="cuda")
    q = torch.empty((0, 256), dtype=torch.int8, device="cuda")
    d = torch.empty((0, 1), dtype=torch.float32, device="cuda")
    tq.tq_quantize_act(x, q, d, torch.empty((0, 1), dtype=torch.int32, device="cuda"))


@pytest.mark.parametrize("key,n,k", [(0, 3, 768), (0x1234567890ABCDEF, 17, 7168), (2 ** 64 - 5, 64, 256)])
def test_synth_weights_match_oracle_generator(tq, oracle, key, n, k):
    m = tq.TqMatrix.empty(n, k)
    announce(f"synth key={key:#x} n={n} k={k}")
    tq.tq_synth_weights(key, m)
    torch.cuda.synchronize()
    c_ref, s_ref = oracle.synth_codes(key, n, k)
    codes = m.codes.cpu().numpy()
    assert np.array_equal(tq.tq_unpack_host(codes, n, k), c_ref)
    assert np.array_equal(m.scales.cpu().numpy().view(np.uint16), s_ref)


def run_gemv(tq, m, x: np.ndarray, want_isum=True):
    t = x.shape[0]
    q, d, b = gpu_quantize(tq, x)
    y = torch.empty((t, m.n), dtype=torch.float32, device="cuda")
    isum = torch.empty((t, m.n, m.k // 256), dtype=torch.int32, device="cuda") if want_isum else None
    tq.tq_gemv(m, q, d, b, y, isum)
    torch.cuda.synchronize()
    return q, d, b, y, isum


def check_gemv(tq, oracle, m, c_ref, s_ref, x):
    q, d, b, y, isum = run_gemv(tq, m, x)
    oq, od, ob = oracle.quantize(x)
    assert np.array_equal(q.cpu().numpy(), oq)
    yr, ar, ir = oracle.gemv(c_ref, s_ref, oq, od, want_isum=True)
    assert np.array_equal(isum.cpu().numpy(), ir)
    return assert_close(y.cpu().numpy(), yr, ar, what="y")


@pytest.mark.parametrize("n,k,t", [(1, 256, 1), (5, 768, 3), (67, 2048, 9), (33, 4096, 2), (19, 7168, 5),
                                   (8, 16384, 4), (300, 3840, 1), (130, 1280, 6)])
def test_gemv_small_shapes(tq, oracle, n, k, t):
    rng = np.random.default_rng(n * 7 + k + t)
    t1 = rng.integers(-1, 2, (n, k)).astype(np.int8)
    t2 = rng.integers(-1, 2, (n, k)).astype(np.int8)
    s = np.asarray(np.exp(rng.uniform(np.log(1e-3), np.log(1e-1), (n, k // 256))), np.float16).view(np.uint16)
    m = tq.TqMatrix(n, k, torch.from_numpy(tq.tq_fold_pack_host(t1, t2)).cuda(), torch.from_numpy(s.view(np.int16)).cuda())
    x = rng.standard_normal((t, k)).astype(np.float32)
    announce(f"gemv n={n} k={k} t={t}")
    check_gemv(tq, oracle, m, oracle.fold(t1, t2), s, x)


def test_gemv_single_matrix_2048x4096(tq, oracle):
    """The single-GEMV workload: 2048 x 4096, one token, seed 0."""
    n, k = gen.CONFIGS[0]["n"], gen.CONFIGS[0]["k"]
    key = gen.single_matrix_key(gen.SEED)
    m = tq.TqMatrix.empty(n, k)
    announce("gemv 2048x4096 seed 0")
    tq.tq_synth_weights(key, m)
    c_ref, s_ref = oracle.synth_codes(key, n, k)
    x = gen.activations(gen.SEED, 0, 1, k)
    rel = check_gemv(tq, oracle, m, c_ref, s_ref, x)
    assert rel < 1e-5
    # bitwise reproducible across runs
    _, _, _, y1, i1 = run_gemv(tq, m, x)
    _, _, _, y2, i2 = run_gemv(tq, m, x)
    assert torch.equal(y1, y2) and torch.equal(i1, i2)


def test_gemv_without_debug_output_matches(tq):
    rng = np.random.default_rng(3)
    n, k = 96, 4096
    m = tq.TqMatrix.empty(n, k)
    tq.tq_synth_weights(99, m)
    x = rng.standard_normal((3, k)).astype(np.float32)
    announce("gemv debug vs no-debug")
    _, _, _, y1, _ = run_gemv(tq, m, x, want_isum=True)
    _, _, _, y2, _ = run_gemv(tq, m, x, want_isum=False)
    assert torch.equal(y1, y2)


def run_gemv_f32(tq, m, x: np.ndarray, want_isum=True):
    t, k = x.shape
    xd = torch.from_numpy(np.ascontiguousarray(x)).cuda()
    q = torch.full((t, k), 99, dtype=torch.int8, device="cuda")
    d = torch.full((t, k // 256), float("nan"), dtype=torch.float32, device="cuda")
    b = torch.full((t, k // 256), -7, dtype=torch.int32, device="cuda")
    y = torch.full((t, m.n), float("nan"), dtype=torch.float32, device="cuda")
    isum = torch.full((t, m.n, k // 256), -1, dtype=torch.int32, device="cuda") if want_isum else None
    tq.tq_gemv_f32(m, xd, y, q, d, b, isum)
    torch.cuda.synchronize()
    return q, d, b, y, isum


@pytest.mark.parametrize("n,k,t", [(1, 256, 1), (5, 768, 1), (67, 2048, 1), (2048, 4096, 1), (19, 7168, 1),
                                   (8, 16384, 1), (300, 3840, 1), (16384, 4096, 1), (16387, 512, 1), (130, 1280, 6)])
def test_gemv_f32_fused_quantization(tq, oracle, n, k, t):
    """tq_gemv_f32 (quantization fused into the dot-pass launch at one token): q, d, bsum
    and the block sums bit-exact against the oracle, y within 1e-5 of the absolute terms
    and bitwise equal to tq_quantize_act + tq_gemv (same rows per wave, same order);
    several tokens take the two-launch path with the same guarantees."""
    rng = np.random.default_rng(n * 11 + k + t)
    t1 = rng.integers(-1, 2, (n, k)).astype(np.int8)
    t2 = rng.integers(-1, 2, (n, k)).astype(np.int8)
    s = np.asarray(np.exp(rng.uniform(np.log(1e-3), np.log(1e-1), (n, k // 256))), np.float16).view(np.uint16)
    m = tq.TqMatrix(n, k, torch.from_numpy(tq.tq_fold_pack_host(t1, t2)).cuda(), torch.from_numpy(s.view(np.int16)).cuda())
    x = rng.standard_normal((t, k)).astype(np.float32) * np.float32(3.0)
    if k >= 1024:
        x[0, 256:512] = 0.0  # an all-zero block: d = 0, q = 0
    announce(f"gemv_f32 n={n} k={k} t={t}")
    q, d, b, y, isum = run_gemv_f32(tq, m, x)
    oq, od, ob = oracle.quantize(x)
    assert np.array_equal(q.cpu().numpy(), oq)
    assert np.array_equal(d.cpu().numpy().view(np.uint32), od.view(np.uint32))
    assert np.array_equal(b.cpu().numpy(), ob)
    yr, ar, ir = oracle.gemv(oracle.fold(t1, t2), s, oq, od, want_isum=True)
    assert np.array_equal(isum.cpu().numpy(), ir)
    assert_close(y.cpu().numpy(), yr, ar + 1e-30, what="y")
    _, _, _, y2, _ = run_gemv(tq, m, x, want_isum=False)
    assert torch.equal(y, y2), "fused quantization changes y"
    _, _, _, y3, _ = run_gemv_f32(tq, m, x, want_isum=False)
    assert torch.equal(y, y3), "debug output changes y"


def test_gemv_f32_single_matrix_2048x4096(tq, oracle):
    """The single-GEMV workload through the fused entry point: 2048 x 4096, one token,
    seed 0."""
    n, k = gen.CONFIGS[0]["n"], gen.CONFIGS[0]["k"]
    key = gen.single_matrix_key(gen.SEED)
    m = tq.TqMatrix.empty(n, k)
    announce("gemv_f32 2048x4096 seed 0")
    tq.tq_synth_weights(key, m)
    c_ref, s_ref = oracle.synth_codes(key, n, k)
    x = gen.activations(gen.SEED, 0, 1, k)
    q, d, b, y, isum = run_gemv_f32(tq, m, x)
    oq, od, ob = oracle.quantize(x)
    assert np.array_equal(q.cpu().numpy(), oq) and np.array_equal(b.cpu().numpy(), ob)
    yr, ar, ir = oracle.gemv(c_ref, s_ref, oq, od, want_isum=True)
    assert np.array_equal(isum.cpu().numpy(), ir)
    assert_close(y.cpu().numpy(), yr, ar, what="y")
