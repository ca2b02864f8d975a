"""GPU parity of the tied quantizer (tq_tied_quantize) against the CPU oracle's tied
solver (Sec. 2.1: alternating code and scale steps against one scale per block).

Bar: bit-exact. Every decision (the fp32 code step, the fp64 pairwise-halving scale
step, the f16 rounding) is taken in the same precision and order on both sides, so the
packed codes, the f16 scales and the number of code steps per block must all match."""
import numpy as np
import pytest
import torch

from gpu_util import announce, device
from synth import gen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tq():
    device()
    from paper_2608_08910_amd import tq as _tq
    return _tq


def gpu_tied(tq, w: np.ndarray, max_iter: int = 16):
    n, k = w.shape
    m = tq.TqMatrix.empty(n, k)
    it = torch.empty((n, k // 256), dtype=torch.uint8, device="cuda")
    tq.tq_tied_quantize(torch.from_numpy(w).cuda(), m, it, max_iter=max_iter)
    torch.cuda.synchronize()
    codes = m.codes.cpu().numpy()
    return tq.tq_unpack_host(codes, n, k), m.scales.cpu().numpy().view(np.uint16), it.cpu().numpy(), codes


def check(tq, oracle, w, max_iter=16):
    c, s, it, packed = gpu_tied(tq, w, max_iter)
    oc, os_, oit = oracle.tied_quantize(w, max_iter)
    bad = np.argwhere(s != os_)
    assert not len(bad), f"scales differ at {bad[:5].tolist()}: gpu {s[tuple(bad[0])]:#06x} oracle {os_[tuple(bad[0])]:#06x}"
    assert np.array_equal(it, oit), f"code steps differ at {np.argwhere(it != oit)[:5].tolist()}"
    assert np.array_equal(c, oc), f"codes differ at {np.argwhere(c != oc)[:5].tolist()}"
    return packed, it


def edge_rows(k: int) -> np.ndarray:
    """Hand-built blocks, tiled to width k: zero, below the 2^-100 floor, an exact f16
    grid, a scale in the f16 subnormal range, one past the f16 range (saturates), and
    blocks whose start scale lands codes on exact halves (w / s = k + 0.5 exactly)."""
    rng = np.random.default_rng(7)
    rows = [np.zeros(256, np.float32), np.full(256, 2.0 ** -110, np.float32)]
    c = rng.integers(-4, 5, 256); c[3] = -4
    rows.append((np.float32(np.float16(0.0123)) * c).astype(np.float32))
    rows.append((rng.standard_normal(256) * 3e-7).astype(np.float32))
    rows.append((rng.standard_normal(256) * 1e5).astype(np.float32))
    h = np.array([4, 0.5, 1.5, 2.5, -2.5, -3.5, -0.5, 3.5] * 32, np.float32)
    rows.append(h * np.float32(0.25))
    rows.append(h * np.float32(0.1875))  # ties again at a start scale that is no power of two
    rows.append(h * np.float32(np.float16(0.0123)))
    out = np.stack(rows)
    return np.tile(out, (1, k // 256))


@pytest.mark.parametrize("n,k", [(7, 256), (16, 768), (33, 4096), (5, 7168)])
def test_tied_random_shapes(tq, oracle, n, k):
    rng = np.random.default_rng(n * 1000 + k)
    w = (rng.standard_normal((n, k)) * np.exp(rng.uniform(np.log(1e-3), np.log(10), (n, 1)))).astype(np.float32)
    announce(f"tied n={n} k={k}")
    check(tq, oracle, w)


@pytest.mark.parametrize("max_iter", [1, 2, 16, 255])
def test_tied_edge_blocks(tq, oracle, max_iter):
    w = edge_rows(1024)
    announce(f"tied edge blocks max_iter={max_iter}")
    _, it = check(tq, oracle, w, max_iter)
    assert it[0].max() == 0 and it[1].max() == 0  # zero and sub-floor blocks take no step


def test_tied_full_matrix_deterministic(tq, oracle):
    c = gen.QUANT_CONFIG
    w = gen.float_weights(gen.SEED, 0, c["n"], c["k"])
    announce("tied 2048x4096 full matrix")
    packed, it = check(tq, oracle, w)
    _, _, it2, packed2 = gpu_tied(tq, w)
    assert np.array_equal(packed, packed2) and np.array_equal(it, it2)
    assert it.max() <= 16 and it.min() >= 2


def test_tied_output_feeds_the_dot_pass(tq, oracle):
    # the quantizer's bytes are the serving bytes: tq_gemv on them matches the oracle's
    # dot pass on the oracle's own codes and scales
    rng = np.random.default_rng(3)
    n, k = 64, 1024
    w = (rng.standard_normal((n, k)) * 0.02).astype(np.float32)
    x = rng.standard_normal((2, k)).astype(np.float32)
    m = tq.TqMatrix.empty(n, k)
    tq.tq_tied_quantize(torch.from_numpy(w).cuda(), m)
    q = torch.empty((2, k), dtype=torch.int8, device="cuda")
    d = torch.empty((2, k // 256), dtype=torch.float32, device="cuda")
    b = torch.empty((2, k // 256), dtype=torch.int32, device="cuda")
    tq.tq_quantize_act(torch.from_numpy(x).cuda(), q, d, b)
    y = torch.empty((2, n), dtype=torch.float32, device="cuda")
    announce("tied -> gemv")
    tq.tq_gemv(m, q, d, b, y)
    torch.cuda.synchronize()
    oc, os_, _ = oracle.tied_quantize(w)
    oq, od, _ = oracle.quantize(x)
    ref, absref = oracle.gemv(oc, os_, oq, od)
    err = np.abs(y.cpu().numpy().astype(np.float64) - ref)
    assert np.all(err <= 1e-5 * absref)
