"""GPU parity of the free-scale solver (tq_free_quantize) against the CPU oracle's
(Sec. 2.1: PTQTP's alternation with two free scales, started from the tied fit).

Bar: bit-exact. Both sides start from the same tied fit (the GPU's, itself bit-exact
with the oracle's) and take every decision in the same precision and order, so the
two planes, the f16 scale pairs and the plane steps per block must all match."""
import numpy as np
import pytest
import torch

from gpu_util import announce, assert_close, device
from synth import gen
from test_gpu_tied import edge_rows

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tq():
    device()
    from paper_2608_08910_amd import tq as _tq
    return _tq


def gpu_free(tq, w: np.ndarray, max_iter: int = 16):
    n, k = w.shape
    wd = torch.from_numpy(w).cuda()
    tied = tq.TqMatrix.empty(n, k)
    tq.tq_tied_quantize(wd, tied)
    out = tq.TqMatrix2.empty(n, k)
    it = torch.empty((n, k // 256), dtype=torch.uint8, device="cuda")
    tq.tq_free_quantize(wd, tied, out, it, max_iter=max_iter)
    torch.cuda.synchronize()
    t1, t2 = tq.tq_unpack2_host(out.codes.cpu().numpy(), n, k)
    return t1, t2, out.scales.cpu().numpy().view(np.uint16), it.cpu().numpy(), out


def check(tq, oracle, w, max_iter=16):
    t1, t2, a, it, out = gpu_free(tq, w, max_iter)
    oc, os_, _ = oracle.tied_quantize(w)
    o1, o2, oa, oit = oracle.free_quantize(w, oc, os_, max_iter)
    bad = np.argwhere(a != oa)
    assert not len(bad), f"scale pairs differ at {bad[:5].tolist()}"
    assert np.array_equal(it, oit), f"plane steps differ at {np.argwhere(it != oit)[:5].tolist()}"
    assert np.array_equal(t1, o1) and np.array_equal(t2, o2), "planes differ"
    return out, it


@pytest.mark.parametrize("n,k", [(7, 256), (16, 768), (33, 4096), (5, 7168)])
def test_free_random_shapes(tq, oracle, n, k):
    rng = np.random.default_rng(n * 977 + k)
    w = (rng.standard_normal((n, k)) * np.exp(rng.uniform(np.log(1e-3), np.log(10), (n, 1)))).astype(np.float32)
    announce(f"free n={n} k={k}")
    check(tq, oracle, w)


@pytest.mark.parametrize("max_iter", [1, 2, 16, 255])
def test_free_edge_blocks(tq, oracle, max_iter):
    # zero and sub-floor blocks, an exact tied grid, f16-subnormal and saturating scales,
    # blocks with exact ties at the start; and a negated copy of each
    w = edge_rows(1024)
    w = np.concatenate([w, -w])
    announce(f"free edge blocks max_iter={max_iter}")
    _, it = check(tq, oracle, w, max_iter)
    assert it[0].max() == 0 and it[1].max() == 0


def test_free_full_matrix_deterministic(tq, oracle):
    c = gen.QUANT_CONFIG
    w = gen.float_weights(gen.SEED, 0, c["n"], c["k"])
    announce("free 2048x4096 full matrix")
    out, it = check(tq, oracle, w)
    _, _, _, it2, out2 = gpu_free(tq, w)
    assert torch.equal(out.codes, out2.codes) and torch.equal(out.scales, out2.scales) and np.array_equal(it, it2)


def test_free_output_feeds_the_two_plane_pass(tq, oracle):
    rng = np.random.default_rng(5)
    n, k = 64, 1024
    w = (rng.standard_normal((n, k)) * 0.02).astype(np.float32)
    x = rng.standard_normal((2, k)).astype(np.float32)
    t1, t2, a, _, out = gpu_free(tq, w)
    q = torch.empty((2, k), dtype=torch.int8, device="cuda")
    d = torch.empty((2, k // 256), dtype=torch.float32, device="cuda")
    b = torch.empty((2, k // 256), dtype=torch.int32, device="cuda")
    tq.tq_quantize_act(torch.from_numpy(x).cuda(), q, d, b)
    y = torch.empty((2, n), dtype=torch.float32, device="cuda")
    announce("free -> gemv2")
    tq.tq_gemv2(out, q, d, y)
    torch.cuda.synchronize()
    oc, os_, _ = oracle.tied_quantize(w)
    o1, o2, oa, _ = oracle.free_quantize(w, oc, os_)
    oq, od, _ = oracle.quantize(x)
    ref, absref = oracle.gemv2(o1, o2, oa, oq, od)
    assert_close(y.cpu().numpy(), ref, absref, what="y")
