"""The no-allocation variant of the routed-expert layer (tq_moe_grouped_noalloc, whose
workspace is the library's fixed per-device scratch array) against tq_moe_grouped on a
caller workspace: two calls in a row on each path, the second with fewer tokens, give
bitwise the same outputs; a call whose workspace exceeds the array is refused before
any launch."""
import numpy as np
import pytest
import torch

from gpu_util import announce, device, host_experts

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tq():
    device()
    from paper_2608_08910_amd import tq as _tq
    return _tq


def _inputs(rng, E, H, T, topk):
    x = torch.from_numpy((rng.standard_normal((T, H)) * 2).astype(np.float32)).cuda()
    idx = torch.from_numpy(np.stack([rng.choice(E, topk, replace=False) for _ in range(T)]).astype(np.int32)).cuda()
    w = torch.from_numpy(rng.uniform(0.1, 1.0, (T, topk)).astype(np.float32)).cuda()
    return x, idx, w


@pytest.mark.parametrize("E,H,I,topk,flags,T1,T2", [
    (12, 1024, 512, 4, 0, 24, 1),      # grouped VALU, then the single-token path
    (10, 768, 1280, 3, 2, 70, 33),     # forced MFMA, two sizes
    (16, 4096, 2048, 8, 0, 32, 5),     # the decode shape, grouped VALU twice
    (16, 4096, 2048, 8, 0, 1, 1),      # the single-token decode shape, twice
])
def test_noalloc_matches_grouped(tq, oracle, E, H, I, topk, flags, T1, T2):
    ex, _ = host_experts(tq, oracle, E, H, I, seed=3000 + E + topk)
    rng = np.random.default_rng(3100 + T1)
    for call, T in enumerate((T1, T2)):
        x, idx, w = _inputs(rng, E, H, T, topk)
        announce(f"noalloc call {call}: E={E} H={H} I={I} T={T} topk={topk} flags={flags}")
        ref = torch.empty((T, H), dtype=torch.float32, device="cuda")
        ws = tq.moe_workspace(ex, T, topk)
        tq.tq_moe_grouped(ex, x, idx, w, ref, ws, flags)
        got = torch.full((T, H), float("nan"), dtype=torch.float32, device="cuda")
        tq.tq_moe_grouped_noalloc(ex, x, idx, w, got, flags)
        torch.cuda.synchronize()
        assert torch.equal(got, ref), f"call {call} (T={T}): no-alloc output differs from tq_moe_grouped"


def test_noalloc_refuses_a_workspace_beyond_the_array(tq, oracle):
    E, H, I, topk = 8, 4096, 2048, 8
    ex, _ = host_experts(tq, oracle, E, H, I, seed=3200)
    need = tq.tq_moe_workspace_bytes(ex, 256, topk)
    assert need > tq.tq_moe_noalloc_max_bytes() == 16 << 20
    x = torch.zeros((256, H), dtype=torch.float32, device="cuda")
    idx = torch.zeros((256, topk), dtype=torch.int32, device="cuda")
    w = torch.zeros((256, topk), dtype=torch.float32, device="cuda")
    out = torch.full((256, H), 7.0, dtype=torch.float32, device="cuda")
    with pytest.raises(tq.TqError) as ei:
        tq.tq_moe_grouped_noalloc(ex, x, idx, w, out)
    assert ei.value.status == tq.TQ_ERR_WORKSPACE and "scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())  # nothing was launched
