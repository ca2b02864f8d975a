"""GPU parity of the MXFP4 reference arm's integer pass (tq_gemv_mx) against the CPU
oracle.

Bar: the exact int32 sums of every 32-element block are bit-exact (they exercise the
kernel's table decode of all 16 e2m1 codes); fp32 outputs agree within 1e-5 of the sum
of the absolute block terms (the order of the fp32 sum is free on the GPU)."""
import numpy as np
import pytest
import torch

from gpu_util import announce, assert_close, device
from synth import gen
from test_gpu_gemv import gpu_quantize, special_blocks

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tq():
    device()
    from paper_2608_08910_amd import tq as _tq
    return _tq


def upload_mx(tq, c4, e8):
    n, k = c4.shape
    return tq.TqMatrixMx(n, k, torch.from_numpy(tq.tq_mx_pack_host(c4)).cuda(), torch.from_numpy(np.ascontiguousarray(e8)).cuda())


def run_mx(tq, m, q, d, want_isum=True):
    t = q.shape[0]
    y = torch.empty((t, m.n), dtype=torch.float32, device="cuda")
    isum = torch.empty((t, m.n, m.k // 32), dtype=torch.int32, device="cuda") if want_isum else None
    tq.tq_gemv_mx(m, q, d, y, isum)
    torch.cuda.synchronize()
    return y, isum


def check_mx(tq, oracle, m, c4, e8, x):
    q, d, _ = gpu_quantize(tq, x)
    oq, od, _ = oracle.quantize(x)
    assert np.array_equal(q.cpu().numpy(), oq)
    y, isum = run_mx(tq, m, q, d)
    yr, ar, ir = oracle.gemv_mx(c4, e8, oq, od, want_isum=True)
    assert np.array_equal(isum.cpu().numpy(), ir)
    return assert_close(y.cpu().numpy(), yr, ar, what="y"), (q, d, y)


def random_mx(rng, n, k):
    return rng.integers(0, 16, (n, k)).astype(np.uint8), rng.integers(112, 132, (n, k // 32)).astype(np.uint8)


@pytest.mark.parametrize("n,k,t", [(1, 256, 1), (5, 768, 3), (67, 2048, 9), (33, 4096, 2), (19, 7168, 5),
                                   (8, 16384, 4), (300, 3840, 1), (130, 1280, 6), (16387, 512, 3),
                                   (16390, 4096, 1)])
def test_gemv_mx_small_shapes(tq, oracle, n, k, t):
    rng = np.random.default_rng(n * 13 + k + t)
    c4, e8 = random_mx(rng, n, k)
    x = rng.standard_normal((t, k)).astype(np.float32)
    announce(f"gemv_mx n={n} k={k} t={t}")
    check_mx(tq, oracle, upload_mx(tq, c4, e8), c4, e8, x)


def test_gemv_mx_every_code_at_every_position(tq, oracle):
    # row r, element i holds code (r + i) mod 16 (each code at every lane position and
    # nibble), one-hot rows (a single nonzero code), block exponents spread over 64..190
    n, k, t = 48, 1024, 3
    c4 = ((np.arange(n)[:, None] + np.arange(k)[None, :]) % 16).astype(np.uint8)
    for r in range(32, 48):
        c4[r] = 0
        c4[r, (r * 37) % k] = r - 32
    e8 = (64 + (np.arange(n)[:, None] * 7 + np.arange(k // 32)[None, :] * 5) % 127).astype(np.uint8)
    x = np.random.default_rng(3).standard_normal((t, k)).astype(np.float32)
    announce("gemv_mx every code at every position")
    check_mx(tq, oracle, upload_mx(tq, c4, e8), c4, e8, x)


@pytest.mark.parametrize("k", [256, 2048])
def test_gemv_mx_edge_activation_blocks(tq, oracle, k):
    x = special_blocks(k)
    x[np.abs(x) > 1e20] = 1.0  # keep 2^(E-128) * d * isum within fp32 (documented precondition)
    rng = np.random.default_rng(k + 1)
    c4, e8 = random_mx(rng, 37, k)
    announce(f"gemv_mx edge activation blocks k={k}")
    check_mx(tq, oracle, upload_mx(tq, c4, e8), c4, e8, x)


def test_gemv_mx_full_size(tq, oracle):
    """The MXFP4 workload at full size in the benchmark's launch configuration: 32768 x 4096,
    one token; every output against the oracle, bitwise reproducible."""
    cfg = gen.MXFP4_CONFIG
    n, k = cfg["n"], cfg["k"]
    c4, e8 = gen.mxfp4_weights(gen.SEED, 0, n, k)
    x = gen.activations(gen.SEED, 0, 1, k)
    announce("gemv_mx 32768x4096 t=1 full size")
    m = upload_mx(tq, c4, e8)
    rel, (q, d, y) = check_mx(tq, oracle, m, c4, e8, x)
    assert rel < 1e-5
    y2, _ = run_mx(tq, m, q, d, want_isum=False)
    y3, _ = run_mx(tq, m, q, d, want_isum=False)
    assert torch.equal(y, y2) and torch.equal(y2, y3)
