"""A seeded sweep of routed-expert layer shapes against the CPU oracle, every path
(automatic choice, forced grouped VALU, forced MFMA): expert counts, hidden and
intermediate widths with 1 to 12 blocks per row (ragged last loads), 1 to 130 tokens,
top-1 to top-8, uniform and skewed routing with duplicated ids in a token's list.
Same bar as test_gpu_moe.py (staged parity bit-exact where integer, the gate, up and
down block sums included, 1e-5 of the absolute terms where fp32)."""
import numpy as np
import pytest
import torch

from gpu_util import announce, check_moe, host_experts, run_moe

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tq():
    from gpu_util import device
    device()
    from paper_2608_08910_amd import tq as _tq
    return _tq


def _cases():
    rng = np.random.default_rng(2026)
    cases = []
    for i in range(12):
        E = int(rng.integers(2, 12))
        H = 256 * int(rng.integers(1, 13))
        I = 256 * int(rng.integers(1, 13))
        T = int(rng.choice([1, 2, 3, 7, 16, 33, 64, 130]))
        topk = int(rng.integers(1, min(E, 8) + 1))
        flags = int(rng.choice([0, 1, 2]))
        skew = bool(rng.integers(0, 2))
        cases.append((i, E, H, I, T, topk, flags, skew))
    return cases


@pytest.mark.parametrize("i,E,H,I,T,topk,flags,skew", _cases())
def test_moe_sweep(tq, oracle, i, E, H, I, T, topk, flags, skew):
    ex, logical = host_experts(tq, oracle, E, H, I, seed=500 + i)
    rng = np.random.default_rng(600 + i)
    x = (rng.standard_normal((T, H)) * np.exp(rng.uniform(-1, 1, (T, 1)))).astype(np.float32)
    p = None
    if skew:
        p = np.arange(1, E + 1, dtype=np.float64) ** -1.5
        p /= p.sum()
    idx = np.stack([rng.choice(E, topk, replace=False, p=p) for _ in range(T)]).astype(np.int32)
    if topk >= 2 and T >= 2:
        idx[1, 1] = idx[1, 0]  # a duplicated expert in one token's list
    w = rng.uniform(0.05, 1.0, (T, topk)).astype(np.float32)
    announce(f"moe sweep {i}: E={E} H={H} I={I} T={T} topk={topk} flags={flags} skew={skew}")
    out, ws = run_moe(tq, ex, x, idx, w, flags=flags)
    tokens = sorted(set([0, T // 2, T - 1]))
    check_moe(tq, oracle, ex, lambda e: logical[e], x, idx, w, out, ws, tokens)
    assert tq.tq_moe_status(ws, ex, T, topk) == 0
    # the production kernels (no debug dump: on the mixed path one launch per projection)
    # give bitwise the checked outputs
    plain, _ = run_moe(tq, ex, x, idx, w, flags=flags, debug=False)
    assert torch.equal(plain, out), "output changes with TQ_MOE_DEBUG_STAGES"
