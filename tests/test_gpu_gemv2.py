"""GPU parity of the free-scale two-plane pass (tq_gemv2) against the CPU oracle.

Bar: the exact int32 block sums of both planes are bit-exact; fp32 outputs agree within
1e-5 of the sum of the absolute block terms (both planes' terms; the order of the fp32
sum is free on the GPU). With tied scales alpha = (3s, s) the two-plane block sums must
meet the fold identity against the folded pass of the same planes on the GPU."""
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


def upload2(tq, t1, t2, a):
    n, k = t1.shape
    return tq.TqMatrix2(n, k, torch.from_numpy(tq.tq_pack2_host(t1, t2)).cuda(),
                        torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda())


def run_gemv2(tq, m, q, d, want_isum=True):
    t = q.shape[0]
    y = torch.empty((t, m.n), dtype=torch.float32, device="cuda")
    isum = torch.empty((t, m.n, m.k // 256, 2), dtype=torch.int32, device="cuda") if want_isum else None
    tq.tq_gemv2(m, q, d, y, isum)
    torch.cuda.synchronize()
    return y, isum


def check_gemv2(tq, oracle, m, t1, t2, a, x):
    q, d, _ = gpu_quantize(tq, x)
    oq, od, _ = oracle.quantize(x)
    assert np.array_equal(q.cpu().numpy(), oq)
    y, isum = run_gemv2(tq, m, q, d)
    yr, ar, ir = oracle.gemv2(t1, t2, a, oq, od, want_isum=True)
    assert np.array_equal(isum.cpu().numpy(), ir)
    return assert_close(y.cpu().numpy(), yr, ar, what="y"), (q, d, y, isum)


def random_two_plane(rng, n, k):
    t1 = rng.integers(-1, 2, (n, k)).astype(np.int8)
    t2 = rng.integers(-1, 2, (n, k)).astype(np.int8)
    a = np.asarray(np.exp(rng.uniform(np.log(1e-3), np.log(1e-1), (n, k // 256, 2))), np.float16).view(np.uint16)
    return t1, t2, a


# shapes: one block; ragged loads (kb % 8 != 0); several token chunks with a ragged
# tail (NT = 4); the largest k; row counts off the wave's; the four-rows-per-wave
# variant (n >= 16384, at most 2 loads per row) with a ragged last wave
@pytest.mark.parametrize("n,k,t", [(1, 256, 1), (5, 768, 3), (67, 2048, 9), (33, 4096, 2), (19, 7168, 5),
                                   (8, 16384, 4), (300, 3840, 1), (130, 1280, 6), (16387, 512, 3),
                                   (16390, 4096, 1)])
def test_gemv2_small_shapes(tq, oracle, n, k, t):
    rng = np.random.default_rng(n * 11 + k + t)
    t1, t2, a = random_two_plane(rng, n, k)
    x = rng.standard_normal((t, k)).astype(np.float32)
    announce(f"gemv2 n={n} k={k} t={t}")
    check_gemv2(tq, oracle, upload2(tq, t1, t2, a), t1, t2, a, x)


@pytest.mark.parametrize("k", [256, 2048])
def test_gemv2_edge_activation_blocks(tq, oracle, k):
    # zero blocks, blocks below the 2^-100 floor, unit-scale halves, huge values
    x = special_blocks(k)
    rng = np.random.default_rng(k)
    t1, t2, a = random_two_plane(rng, 37, k)
    announce(f"gemv2 edge activation blocks k={k}")
    check_gemv2(tq, oracle, upload2(tq, t1, t2, a), t1, t2, a, x)


def test_gemv2_edge_planes(tq, oracle):
    # all-zero planes, one plane empty, all -1 / all +1 rows, zero and negative scales,
    # f16 subnormal and largest-finite scales
    n, k, t = 12, 1024, 3
    rng = np.random.default_rng(7)
    t1, t2, a = random_two_plane(rng, n, k)
    t1[0] = 0; t2[0] = 0
    t2[1] = 0
    t1[2] = 0
    t1[3] = -1; t2[3] = -1
    t1[4] = 1; t2[4] = 1
    a[5] = 0
    a[6, :, 1] = 0
    a[7] ^= np.uint16(0x8000)
    a[8] = 0x0001  # smallest subnormal
    a[9] = 0x7BFF  # 65504
    x = rng.standard_normal((t, k)).astype(np.float32)
    announce("gemv2 edge planes and scales")
    check_gemv2(tq, oracle, upload2(tq, t1, t2, a), t1, t2, a, x)


def test_gemv2_tied_scales_meet_the_fold_identity_on_the_gpu(tq, oracle):
    # alpha = (3s, s) with 3s exact in f16: the two-plane block sums and the folded pass's
    # block sums of the same planes satisfy 3 * isum_1 + isum_2 = isum_folded exactly
    n, k, t = 96, 4096, 5
    rng = np.random.default_rng(13)
    t1 = rng.integers(-1, 2, (n, k)).astype(np.int8)
    t2 = rng.integers(-1, 2, (n, k)).astype(np.int8)
    s = (rng.integers(gen.SCALE_F16_LO, gen.SCALE_F16_HI, (n, k // 256)) & ~3).astype(np.uint16)
    s3 = np.asarray(3 * s.view(np.float16).astype(np.float64), np.float16).view(np.uint16)
    a = np.ascontiguousarray(np.stack([s3, s], axis=2))
    x = rng.standard_normal((t, k)).astype(np.float32)
    announce("gemv2 tied scales vs folded pass")
    _, (q, d, y2, isum2) = check_gemv2(tq, oracle, upload2(tq, t1, t2, a), t1, t2, a, x)
    mf = tq.TqMatrix(n, k, torch.from_numpy(tq.tq_fold_pack_host(t1, t2)).cuda(), torch.from_numpy(s.view(np.int16)).cuda())
    yf = torch.empty((t, n), dtype=torch.float32, device="cuda")
    isf = torch.empty((t, n, k // 256), dtype=torch.int32, device="cuda")
    tq.tq_gemv(mf, q, d, torch.zeros((t, k // 256), dtype=torch.int32, device="cuda"), yf, isf)
    torch.cuda.synchronize()
    i2 = isum2.cpu().numpy().astype(np.int64)
    assert np.array_equal(3 * i2[..., 0] + i2[..., 1], isf.cpu().numpy())
    yr, ar = oracle.gemv(oracle.fold(t1, t2), s, *oracle.quantize(x)[:2])
    assert_close(yf.cpu().numpy(), yr, ar, what="folded y")


def test_gemv2_decode_stack_full_size(tq, oracle):
    """The two-plane workload at full size and in the launch configuration the benchmark
    times: 32768 x 4096 (one decode step's routed gate and up rows), one token; every
    output against the oracle, and bitwise reproducible."""
    cfg = gen.TWO_PLANE_CONFIG
    n, k = cfg["n"], cfg["k"]
    t1, t2, a = gen.two_plane_weights(gen.SEED, 0, n, k)
    x = gen.activations(gen.SEED, 0, 1, k)
    announce("gemv2 32768x4096 t=1 full size")
    m = upload2(tq, t1, t2, a)
    rel, (q, d, y, isum) = check_gemv2(tq, oracle, m, t1, t2, a, x)
    assert rel < 1e-5
    y2, _ = run_gemv2(tq, m, q, d, want_isum=False)
    y3, _ = run_gemv2(tq, m, q, d, want_isum=False)
    assert torch.equal(y, y2) and torch.equal(y2, y3)
