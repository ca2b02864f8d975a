"""Host-tier expert streaming on the GPU: a step served from an LRU pool of expert slots
in HBM, filled from pinned host memory, must give bitwise the same output as the same
step served from resident experts (the same bytes and kernels, only the addresses
differ), for the single-token, grouped VALU and MFMA paths. The first and the last
streamed step of each case are also checked against the oracle (staged, with the gate,
up and down block sums bit-exact, and end to end), the slot ids mapped back to expert
ids; and two streamed steps queued without a synchronization between them (each with
its own pinned slot-id buffer) give the resident outputs."""
import numpy as np
import pytest
import torch

import oracle as oracle_pkg
from gpu_util import announce, check_moe, device, synth_experts
from synth import gen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tq():
    device()
    from paper_2608_08910_amd import tq as _tq
    return _tq


def records_from_stack(tq, ex):
    """The stacked experts' bytes rewritten as contiguous records (device)."""
    rec = tq.TqExpertRecords.empty(ex.n_experts, ex.hidden, ex.inter)
    base = 1 << 20
    d = tq.tq_experts_from_records(base, 1, ex.hidden, ex.inter)
    code_offs = [d.gate_codes - base, d.up_codes - base, d.down_codes - base]
    scale_offs = [d.gate_scales - base, d.up_scales - base, d.down_scales - base]
    for p in range(3):
        c = ex.codes[p].reshape(ex.n_experts, -1)
        s = ex.scales[p].reshape(ex.n_experts, -1).view(torch.uint8)
        rec.data[:, code_offs[p]:code_offs[p] + c.shape[1]] = c
        rec.data[:, scale_offs[p]:scale_offs[p] + s.shape[1]] = s
    torch.cuda.synchronize()
    return rec


def run_resident(tq, ex, x, idx, w, flags):
    T, H = x.shape
    out = torch.empty((T, H), dtype=torch.float32, device="cuda")
    ws = tq.moe_workspace(ex, T, idx.shape[1])
    tq.tq_moe_grouped(ex, x, idx, w, out, ws, flags)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("E,H,I,S,T,topk,flags,steps", [
    (12, 512, 512, 4, 1, 2, 0, 10),       # single-token path, small
    (12, 512, 768, 5, 3, 2, 0, 10),       # grouped VALU path
    (12, 512, 512, 8, 4, 2, 2, 6),        # forced MFMA path
    (32, 4096, 2048, 10, 1, 8, 0, 6),     # decode batch 1 at the model's shape
    (48, 4096, 2048, 32, 4, 8, 0, 4),     # grouped decode at the model's shape
])
def test_streamed_equals_resident_bitwise(tq, oracle, E, H, I, S, T, topk, flags, steps):
    announce(f"stream E={E} H={H} I={I} S={S} T={T} topk={topk} flags={flags}")
    ex = synth_experts(tq, 7, 0, E, H, I)
    resident = records_from_stack(tq, ex)
    store = tq.TqExpertRecords.empty(E, H, I, device="cpu", pin_memory=True)
    store.data.copy_(resident.data)
    pool = tq.TqExpertRecords.empty(S, H, I)
    cache = tq.TqCache(E, S)
    ws_pool = tq.moe_workspace(pool, T, topk, debug=True)
    get = oracle_pkg.expert_getter(7, 0, H, I, oracle)
    rng = np.random.default_rng(E * 100 + T)
    total_misses = 0
    served = []
    for step in range(steps):
        ids = np.stack([rng.choice(E, size=topk, replace=False) for _ in range(T)]).astype(np.int32)
        if len(np.unique(ids)) > S:
            continue
        w = rng.random((T, topk)).astype(np.float32)
        xh = rng.standard_normal((T, H)).astype(np.float32)
        x = torch.from_numpy(xh).cuda()
        idx_dev = torch.from_numpy(ids).cuda()
        w_dev = torch.from_numpy(w).cuda()
        slots_host = torch.empty((T, topk), dtype=torch.int32).pin_memory()
        slots, misses = cache.map(ids, slots_host.numpy())
        total_misses += len(misses)
        slots_dev = torch.empty((T, topk), dtype=torch.int32, device="cuda")
        cache.fetch(store, pool, misses, slots_host, slots_dev)
        out_s = torch.empty((T, H), dtype=torch.float32, device="cuda")
        tq.tq_moe_grouped(pool, x, slots_dev, w_dev, out_s, ws_pool, flags | tq.TQ_MOE_DEBUG_STAGES)
        torch.cuda.synchronize()
        out_r = run_resident(tq, resident, x, idx_dev, w_dev, flags)
        out_k = run_resident(tq, ex, x, idx_dev, w_dev, flags)
        assert torch.equal(out_s, out_r), f"step {step}: streamed != resident records"
        assert torch.equal(out_r, out_k), f"step {step}: records != stacked layout"
        for e, s in zip(ids.ravel().tolist(), slots.ravel().tolist()):
            assert torch.equal(pool.data[s], resident.data[e])
        served.append(step)
        if len(served) == 1 or step == steps - 1:
            # the streamed step against the oracle: its stage buffers are per slot position,
            # so the expert ids themselves name what each slot ran
            announce(f"stream step {step}: oracle")
            check_moe(tq, oracle, pool, get, xh, ids, w, out_s, ws_pool, list(range(T)), n_ids=E)
    assert total_misses > 0


@pytest.mark.parametrize("E,H,I,S,T,topk,flags", [(12, 512, 768, 5, 3, 2, 0), (16, 1024, 512, 6, 1, 4, 0),
                                                 (12, 512, 512, 8, 4, 2, 2)])
def test_two_streamed_steps_queued_without_sync(tq, E, H, I, S, T, topk, flags):
    """Two steps planned, fetched and run back to back on one stream with no host
    synchronization between them, each with its own pinned slot-id buffer: both outputs
    equal the resident ones (the second step's copies, queued behind the first step's
    kernels, may overwrite slots the first step reads only after it has read them)."""
    announce(f"stream queued E={E} H={H} I={I} S={S} T={T} topk={topk} flags={flags}")
    ex = synth_experts(tq, 9, 0, E, H, I)
    resident = records_from_stack(tq, ex)
    store = tq.TqExpertRecords.empty(E, H, I, device="cpu", pin_memory=True)
    store.data.copy_(resident.data)
    pool = tq.TqExpertRecords.empty(S, H, I)
    cache = tq.TqCache(E, S)
    rng = np.random.default_rng(E * 10 + S)
    for rnd in range(3):
        steps = []
        for k in range(2):
            while True:
                ids = np.stack([rng.choice(E, size=topk, replace=False) for _ in range(T)]).astype(np.int32)
                if len(np.unique(ids)) <= S:
                    break
            x = torch.from_numpy(rng.standard_normal((T, H)).astype(np.float32)).cuda()
            w = torch.from_numpy(rng.random((T, topk)).astype(np.float32)).cuda()
            slots_host = torch.empty((T, topk), dtype=torch.int32).pin_memory()
            _, misses = cache.map(ids, slots_host.numpy())
            slots_dev = torch.empty((T, topk), dtype=torch.int32, device="cuda")
            out = torch.empty((T, H), dtype=torch.float32, device="cuda")
            ws = tq.moe_workspace(pool, T, topk)
            cache.fetch(store, pool, misses, slots_host, slots_dev)
            tq.tq_moe_grouped(pool, x, slots_dev, w, out, ws, flags)
            steps.append((ids, x, w, out, slots_host))
        torch.cuda.synchronize()
        for k, (ids, x, w, out, _) in enumerate(steps):
            ref = run_resident(tq, resident, x, torch.from_numpy(ids).cuda(), w, flags)
            assert torch.equal(out, ref), f"round {rnd} step {k}: queued streamed step != resident"
