"""GPU parity of the routed-expert MoE layer (tq_moe_grouped) against the CPU oracle.

Every parity call runs with TQ_MOE_DEBUG_STAGES, so that the exact int32 block sums of
the gate, up and down dot passes of every checked slot are compared bit for bit with the
oracle's; the staged and end-to-end bars are those of gpu_util.check_moe / check_slots.
The flag's outputs are checked to be bitwise those of the same call without it, on every
path (single token, grouped VALU, grouped MFMA)."""
import numpy as np
import pytest
import torch

import oracle as oracle_pkg
from gpu_util import (announce, assert_close, check_moe, check_slots, device, host_experts, run_moe,
                      synth_experts, ws_views)
from synth import gen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tq():
    device()
    from paper_2608_08910_amd import tq as _tq
    return _tq


@pytest.fixture(scope="module")
def experts_h4096(tq):
    """The 256 routed experts (hidden 4096, inter 2048) of the decode workloads, seed 0."""
    announce("synth 256 experts h4096 i2048")
    ex = synth_experts(tq, gen.SEED, 0, 256, 4096, 2048)
    torch.cuda.synchronize()
    return ex


def test_moe_small_host_packed(tq, oracle):
    E, H, I, T, topk = 6, 512, 768, 7, 3
    ex, logical = host_experts(tq, oracle, E, H, I, seed=5)
    rng = np.random.default_rng(6)
    x = (rng.standard_normal((T, H)) * 2).astype(np.float32)
    idx = np.stack([rng.choice(E, topk, replace=False) for _ in range(T)]).astype(np.int32)
    idx[3] = [2, 2, 5]  # a duplicated expert in one token's list: two separate slots
    w = rng.uniform(0.1, 1.0, (T, topk)).astype(np.float32)
    announce("moe small host-packed")
    out, ws = run_moe(tq, ex, x, idx, w)
    check_moe(tq, oracle, ex, lambda e: logical[e], x, idx, w, out, ws, list(range(T)))
    assert tq.tq_moe_status(ws, ex, T, topk) == 0


def test_moe_invalid_expert_ids_flagged_and_skipped(tq, oracle):
    E, H, I, T, topk = 4, 256, 256, 3, 2
    ex, logical = host_experts(tq, oracle, E, H, I, seed=8)
    rng = np.random.default_rng(9)
    x = rng.standard_normal((T, H)).astype(np.float32)
    idx = np.array([[0, 1], [-1, 2], [3, E]], np.int32)
    w = np.full((T, topk), 0.5, np.float32)
    announce("moe invalid ids")
    out, ws = run_moe(tq, ex, x, idx, w)
    assert tq.tq_moe_status(ws, ex, T, topk) & 1
    # the routed slots staged and end to end; the unrouted ones add nothing
    check_moe(tq, oracle, ex, lambda e: logical[e], x, idx, w, out, ws, [0, 1, 2])


def test_moe_zero_tokens_and_top1(tq, oracle):
    E, H, I = 3, 256, 512
    ex, logical = host_experts(tq, oracle, E, H, I, seed=11)
    x = np.zeros((0, H), np.float32)
    run_moe(tq, ex, x, np.zeros((0, 1), np.int32), np.zeros((0, 1), np.float32))
    rng = np.random.default_rng(12)
    x = rng.standard_normal((2, H)).astype(np.float32)
    idx = np.array([[1], [2]], np.int32)
    w = np.ones((2, 1), np.float32)
    announce("moe top-1")
    out, ws = run_moe(tq, ex, x, idx, w)
    check_moe(tq, oracle, ex, lambda e: logical[e], x, idx, w, out, ws, [0, 1])


def assert_debug_flag_neutral(tq, ex, x, idx, w, out, flags=0):
    """The call without TQ_MOE_DEBUG_STAGES gives bitwise the debug call's output."""
    plain, _ = run_moe(tq, ex, x, idx, w, flags=flags, debug=False)
    assert torch.equal(plain, out), "output changes with TQ_MOE_DEBUG_STAGES"


def test_moe_decode_batch1_uniform(tq, oracle, experts_h4096):
    """One MoE layer at decode, batch 1: 256 experts, hidden 4096, inter 2048, top-8
    uniform without replacement, softmax weights over N(0,1) logits, seed 0. All 8 slots'
    gate, up and down block sums bit-exact."""
    c = gen.CONFIGS[1]
    x = gen.activations(gen.SEED, 0, c["tokens"], c["hidden"])
    idx, w = gen.routing(gen.SEED, 0, c["tokens"], c["experts"], c["topk"], c["routing"])
    assert tq.tq_moe_path(experts_h4096, 1, c["topk"]) == tq.TQ_MOE_PATH_T1
    announce("moe decode t=1 top-8 uniform")
    out, ws = run_moe(tq, experts_h4096, x, idx, w)
    get = oracle_pkg.expert_getter(gen.SEED, 0, c["hidden"], c["inter"], oracle)
    check_moe(tq, oracle, experts_h4096, get, x, idx, w, out, ws, [0])
    assert tq.tq_moe_status(ws, experts_h4096, 1, c["topk"]) == 0
    out2, _ = run_moe(tq, experts_h4096, x, idx, w)
    assert torch.equal(out, out2)  # bitwise reproducible
    assert_debug_flag_neutral(tq, experts_h4096, x, idx, w, out)


def test_moe_decode_batch32_zipf(tq, oracle, experts_h4096):
    """Batched decode: 32 tokens, top-8 with Zipf(1.1) expert popularity, seed 0, on the
    mixed path (the experts of 3 to 32 slots on the 32-token MFMA kernel, the others on
    the grouped VALU kernel). Every slot's block sums bit-exact."""
    c = gen.CONFIGS[2]
    x = gen.activations(gen.SEED, 0, c["tokens"], c["hidden"])
    idx, w = gen.routing(gen.SEED, 0, c["tokens"], c["experts"], c["topk"], c["routing"])
    assert tq.tq_moe_path(experts_h4096, c["tokens"], c["topk"]) == tq.TQ_MOE_PATH_MIXED
    counts = np.bincount(idx.ravel(), minlength=c["experts"])
    assert (counts > 2).any() and ((counts > 0) & (counts <= 2)).any()  # both kernels have experts
    announce("moe decode t=32 top-8 zipf")
    out, ws = run_moe(tq, experts_h4096, x, idx, w)
    get = oracle_pkg.expert_getter(gen.SEED, 0, c["hidden"], c["inter"], oracle)
    check_moe(tq, oracle, experts_h4096, get, x, idx, w, out, ws, list(range(c["tokens"])))
    assert_debug_flag_neutral(tq, experts_h4096, x, idx, w, out)


def test_moe_prefill_2048(tq, oracle, experts_h4096):
    """Prefill: 2048 tokens, Zipf top-8, activations scaled per token by a log-uniform
    factor in [0.1, 10]; the expert contraction runs on int8 MFMA in tiles of 128 tokens.
      - every token's quantized input, bit-exact;
      - every token's out against sum_j w_j * yd_j of its own slots (GPU data, fp64);
      - the dispatch lists: each expert's slot count, and the hottest expert first;
      - staged parity, block sums bit-exact, for two slots of every 128-token tile of the
        three hottest experts (a position that moves across the tile, and the tile's last
        token), and end to end for a spread of tokens."""
    c = gen.CONFIGS[3]
    T, topk, H = c["tokens"], c["topk"], c["hidden"]
    x = gen.activations(gen.SEED, 0, T, H) * gen.token_factors(gen.SEED, T)[:, None]
    idx, w = gen.routing(gen.SEED, 0, T, c["experts"], topk, c["routing"])
    assert tq.tq_moe_path(experts_h4096, T, topk) == tq.TQ_MOE_PATH_MFMA
    announce("moe prefill t=2048 (debug dump)")
    out, ws = run_moe(tq, experts_h4096, x, idx, w)
    V = ws_views(tq, experts_h4096, ws, T, topk)
    oq, od, ob = oracle.quantize(x)
    assert np.array_equal(V["xq"].cpu().numpy(), oq)
    assert np.array_equal(V["xd"].cpu().numpy().view(np.uint32), od.view(np.uint32))
    assert np.array_equal(V["xb"].cpu().numpy(), ob)
    # every token, staged: out[t] against its slots' yd, ascending j, in fp64 on the device
    yd = V["yd"].view(T, topk, H).double()
    wd = torch.from_numpy(w).cuda().double()
    staged = torch.zeros((T, H), dtype=torch.float64, device="cuda")
    staged_abs = torch.zeros_like(staged)
    for j in range(topk):
        staged += wd[:, j:j + 1] * yd[:, j]
        staged_abs += wd[:, j:j + 1].abs() * yd[:, j].abs()
    ratio = ((out.double() - staged).abs() / (staged_abs + 1e-30)).max().item()
    assert ratio <= 1e-5, f"out vs its slots' yd: worst {ratio:.3g} of the absolute terms"
    del yd, staged, staged_abs
    # dispatch lists
    counts = np.bincount(idx.ravel(), minlength=c["experts"])
    n_active = int(V["n_active"].item())
    active = V["active"][:n_active].cpu().numpy()
    off = V["act_off"][:n_active + 1].cpu().numpy()
    slot_list = V["slot_list"].cpu().numpy()
    assert n_active == int((counts > 0).sum()) and active[0] == int(np.argmax(counts))
    assert np.array_equal(np.diff(off), counts[active])
    for a in range(n_active):
        sl = slot_list[off[a]:off[a + 1]]
        assert np.array_equal(np.sort(sl), np.where(idx.ravel() == active[a])[0])
    # two slots of every 128-token tile of the three hottest experts
    slots = []
    for a in range(3):
        cnt = off[a + 1] - off[a]
        for k0 in range(0, cnt, 128):
            n_in = min(128, cnt - k0)
            for p in sorted({k0 + (37 * (k0 // 128) + 5) % n_in, k0 + n_in - 1}):
                slots.append(int(slot_list[off[a] + p]))
    get = oracle_pkg.expert_getter(gen.SEED, 0, c["hidden"], c["inter"], oracle)
    announce(f"moe prefill: staged parity of {len(slots)} slots")
    _, flips, codes = check_slots(tq, oracle, experts_h4096, get, x, idx, ws, slots, V)
    assert sum(flips.values()) <= max(2, 1e-3 * codes)
    # end to end on a spread of tokens (the hottest expert's first, the coldest used one's)
    cold = int(np.where(counts > 0)[0][np.argmin(counts[counts > 0])])
    tokens = sorted(set([int(np.where((idx == 0).any(1))[0][0]), int(np.where((idx == cold).any(1))[0][0]), 0, 777,
                         2047]))
    check_moe(tq, oracle, experts_h4096, get, x, idx, w, out, ws, tokens)
    del V
    torch.cuda.empty_cache()
    assert_debug_flag_neutral(tq, experts_h4096, x, idx, w, out)


def test_moe_prefill_2048_paths_agree(tq, experts_h4096):
    """Every slot and output of the 2048-token prefill layer, MFMA path (the production
    instances, no debug dump) against the grouped VALU path, which the sampled oracle
    checks cover on their own: a tile the MFMA task order leaves out, repeats or places on
    the wrong rows shows up here whichever tokens it holds, as an error of the size of the
    values themselves. The int32 block dots are exact on both paths, which differ only in
    the fp32 order of the block-scaled sums:
      - h of every slot within 1e-5 of the slot's largest |h| (gate/up tiles);
      - the requantized codes of h equal but for rare one-step flips near a rounding
        boundary (at most one code in 1e4), with block scales within 1e-6;
      - yd of every slot whose codes of h came out identical within 1e-5 of the slot's
        largest |yd| (down tiles); every slot's within 1e-2, since one flip moves a slot's
        whole row by about a thousandth of its size;
      - out of every token within 1e-2 of the token's largest output."""
    c = gen.CONFIGS[3]
    T, topk, H = c["tokens"], c["topk"], c["hidden"]
    x = gen.activations(gen.SEED, 0, T, H) * gen.token_factors(gen.SEED, T)[:, None]
    idx, w = gen.routing(gen.SEED, 0, T, c["experts"], topk, c["routing"])
    announce("moe prefill t=2048: MFMA path against VALU path, every slot and output")

    def rel(a, b, dim=1):
        return ((a - b).abs() / b.abs().amax(dim=dim, keepdim=True).clamp_min(1e-30)).amax(dim=dim)

    out_m, ws_m = run_moe(tq, experts_h4096, x, idx, w, debug=False)
    out_v, ws_v = run_moe(tq, experts_h4096, x, idx, w, flags=tq.TQ_MOE_FORCE_VALU, debug=False)
    Vm, Vv = ws_views(tq, experts_h4096, ws_m, T, topk), ws_views(tq, experts_h4096, ws_v, T, topk)
    assert torch.isfinite(out_m).all() and torch.isfinite(Vm["h"]).all()
    h_rel = rel(Vm["h"], Vv["h"]).max().item()
    dq = Vm["hq"].int() - Vv["hq"].int()
    n_flip = int((dq != 0).sum().item())
    hd_rel = ((Vm["hd"] - Vv["hd"]).abs() / Vv["hd"].abs().clamp_min(1e-30)).max().item()
    clean = (dq != 0).sum(dim=1).eq(0)
    yd_rel = rel(Vm["yd"], Vv["yd"])
    yd_clean, yd_all = yd_rel[clean].max().item(), yd_rel.max().item()
    out_rel = rel(out_m, out_v).max().item()
    msg = (f"MFMA vs VALU path: h {h_rel:.3g}; {n_flip} code flips (max step {dq.abs().max().item()}), "
           f"hd {hd_rel:.3g}; yd {yd_clean:.3g} on {int(clean.sum())} clean slots of {clean.numel()}, "
           f"{yd_all:.3g} on all; out {out_rel:.3g}")
    print(msg)
    assert h_rel <= 1e-5, msg
    assert dq.abs().max().item() <= 1 and n_flip <= 1e-4 * dq.numel(), msg
    assert hd_rel <= 1e-6, msg
    assert yd_clean <= 1e-5 and yd_all <= 1e-2, msg
    assert out_rel <= 1e-2, msg
    del out_m, out_v, ws_m, ws_v, Vm, Vv, dq, yd_rel
    torch.cuda.empty_cache()


def test_moe_mixed_all_rank_ranges(tq, oracle):
    """The mixed path with both roles populated: expert 0 in all 40 tokens (more than 32
    slots: two 32-token tiles of the MFMA role), experts 1-5 with 16 slots each (one tile
    each), experts 6 and 7 with one slot each (VALU role); hidden 17 blocks (loads per lane
    rounded up from 3 to 4, ragged) and inter 9 blocks (ragged). Every token staged
    against the oracle (debug run), and the one-launch production kernels bitwise equal
    to it."""
    E, H, I, T, topk = 8, 256 * 17, 256 * 9, 40, 3
    ex, logical = host_experts(tq, oracle, E, H, I, seed=71)
    rng = np.random.default_rng(72)
    x = rng.standard_normal((T, H)).astype(np.float32)
    idx = np.array([[0, 1 + t % 5, 6 + t if t < 2 else 1 + (t + 2) % 5] for t in range(T)], np.int32)
    counts = np.bincount(idx.ravel(), minlength=E)
    assert counts[0] > 32 and (counts[1:6] > 2).all() and (counts[1:6] <= 32).all() and counts[6] == counts[7] == 1
    w = rng.uniform(0.1, 1.0, (T, topk)).astype(np.float32)
    assert tq.tq_moe_path(ex, T, topk) == tq.TQ_MOE_PATH_MIXED
    announce("moe mixed path, all rank ranges")
    out, ws = run_moe(tq, ex, x, idx, w)
    check_moe(tq, oracle, ex, lambda e: logical[e], x, idx, w, out, ws, list(range(T)))
    assert_debug_flag_neutral(tq, ex, x, idx, w, out)


@pytest.mark.parametrize("T,flags", [(1, 0), (24, 1), (40, 0), (40, 2)])
def test_moe_timed_matches_untimed(tq, oracle, T, flags):
    """tq_moe_grouped_timed on every path (single token, forced VALU, mixed, forced MFMA
    with its two launches on two streams): the output is bitwise that of tq_moe_grouped,
    every kernel stage of the path takes a positive time, the empty ones none below zero,
    and the stages follow one another."""
    E, H, I, topk = 16, 1024, 512, 4
    ex, _ = host_experts(tq, oracle, E, H, I, seed=95)
    rng = np.random.default_rng(96)
    x = torch.from_numpy(rng.standard_normal((T, H)).astype(np.float32)).cuda()
    idx = torch.from_numpy(np.stack([rng.choice(E, topk, replace=False) for _ in range(T)]).astype(np.int32)).cuda()
    w = torch.from_numpy(rng.uniform(0.1, 1.0, (T, topk)).astype(np.float32)).cuda()
    path = tq.tq_moe_path(ex, T, topk, flags)
    assert path == {(1, 0): tq.TQ_MOE_PATH_T1, (24, 1): tq.TQ_MOE_PATH_VALU, (40, 0): tq.TQ_MOE_PATH_MIXED,
                    (40, 2): tq.TQ_MOE_PATH_MFMA}[(T, flags)]
    ws = tq.moe_workspace(ex, T, topk)
    announce(f"moe timed entry point T={T} flags={flags}")
    ref = torch.empty((T, H), dtype=torch.float32, device="cuda")
    tq.tq_moe_grouped(ex, x, idx, w, ref, ws, flags)
    n = tq.tq_moe_stage_count()
    names = [tq.tq_moe_stage_name(i) for i in range(n)]
    for rep in range(2):  # (the second call reuses the events)
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(2 * n)]
        out = torch.full((T, H), float("nan"), device="cuda")
        tq.tq_moe_grouped_timed(ex, x, idx, w, out, ws, evs, flags)
        torch.cuda.synchronize()
        assert torch.equal(out, ref), f"call {rep}"
        kernel_stages = {"gate_up", "down"} if path == tq.TQ_MOE_PATH_T1 else set(names)
        for i, name in enumerate(names):
            ms = evs[2 * i].elapsed_time(evs[2 * i + 1])
            assert (ms > 0) if name in kernel_stages else (ms >= 0), (name, ms)
            if i > 0:
                assert evs[2 * (i - 1) + 1].elapsed_time(evs[2 * i]) >= 0, f"stage {name} starts before its predecessor ends"


def test_moe_mixed_boundary_counts(tq, oracle):
    """The mixed path's roles at their bounds: experts of exactly 33 slots (two 32-token
    tiles, the second with one token), 32, 28 and 3 (one tile) on the MFMA role, 2 and 1
    on the VALU role; ragged rows (3 and 5 blocks). Every token staged against the oracle,
    and the production kernels bitwise equal to the debug run."""
    E, H, I, T, topk = 8, 256 * 3, 256 * 5, 33, 3
    ex, logical = host_experts(tq, oracle, E, H, I, seed=81)
    rng = np.random.default_rng(82)
    x = rng.standard_normal((T, H)).astype(np.float32)
    col1 = [1 if t < 32 else 2 for t in range(T)]
    col2 = [2 if t < 2 else (3 if t < 4 else (4 if t == 4 else 5)) for t in range(T)]
    idx = np.array([[0, col1[t], col2[t]] for t in range(T)], np.int32)
    assert all(len(set(r)) == topk for r in idx.tolist())
    assert np.bincount(idx.ravel(), minlength=E).tolist() == [33, 32, 3, 2, 1, 28, 0, 0]
    w = rng.uniform(0.1, 1.0, (T, topk)).astype(np.float32)
    assert tq.tq_moe_path(ex, T, topk) == tq.TQ_MOE_PATH_MIXED
    announce("moe mixed path, boundary counts")
    out, ws = run_moe(tq, ex, x, idx, w)
    check_moe(tq, oracle, ex, lambda e: logical[e], x, idx, w, out, ws, list(range(T)))
    assert_debug_flag_neutral(tq, ex, x, idx, w, out)


@pytest.mark.parametrize("E,H,I,T,topk", [(5, 512, 768, 150, 3), (4, 1280, 256, 70, 2)])
def test_moe_mfma_forced_small(tq, oracle, E, H, I, T, topk):
    """The int8 MFMA expert path on host-packed experts: one expert spans several
    128-token tiles, hidden/inter give ragged row tiles and odd block counts (1 to 5)."""
    ex, logical = host_experts(tq, oracle, E, H, I, seed=21)
    rng = np.random.default_rng(22)
    x = (rng.standard_normal((T, H)) * np.exp(rng.uniform(-2, 2, (T, 1)))).astype(np.float32)
    idx = np.stack([np.concatenate([[0], rng.choice(np.arange(1, E), topk - 1, replace=False)]) for _ in range(T)]).astype(np.int32)
    w = rng.uniform(0.1, 1.0, (T, topk)).astype(np.float32)
    announce(f"moe mfma E={E} H={H} I={I} T={T}")
    out, ws = run_moe(tq, ex, x, idx, w, flags=tq.TQ_MOE_FORCE_MFMA)
    check_moe(tq, oracle, ex, lambda e: logical[e], x, idx, w, out, ws, [0, 1, 63, 64, 65, T - 1])
    out2, _ = run_moe(tq, ex, x, idx, w, flags=tq.TQ_MOE_FORCE_MFMA)
    assert torch.equal(out, out2)
    assert_debug_flag_neutral(tq, ex, x, idx, w, out, flags=tq.TQ_MOE_FORCE_MFMA)


def test_moe_mfma_forced_batch32(tq, oracle, experts_h4096):
    """The batched-decode workload forced onto the MFMA path (all tokens checked)."""
    c = gen.CONFIGS[2]
    x = gen.activations(gen.SEED, 0, c["tokens"], c["hidden"])
    idx, w = gen.routing(gen.SEED, 0, c["tokens"], c["experts"], c["topk"], c["routing"])
    announce("moe mfma forced t=32")
    out, ws = run_moe(tq, experts_h4096, x, idx, w, flags=tq.TQ_MOE_FORCE_MFMA)
    get = oracle_pkg.expert_getter(gen.SEED, 0, c["hidden"], c["inter"], oracle)
    check_moe(tq, oracle, experts_h4096, get, x, idx, w, out, ws, list(range(c["tokens"])))
    assert_debug_flag_neutral(tq, experts_h4096, x, idx, w, out, flags=tq.TQ_MOE_FORCE_MFMA)


@pytest.mark.parametrize("E,H,I,topk", [(4, 512, 768, 3), (3, 7168, 2048, 2), (9, 2304, 1280, 8), (2, 256, 256, 1),
                                        (5, 4096, 4096, 4), (10, 7168, 2048, 8), (12, 8192, 512, 8),
                                        (8, 1024, 1792, 8), (9, 256, 2048, 8), (3, 512, 8192, 2),
                                        (3, 256, 6400, 2), (2, 256, 16384, 1)])
def test_moe_single_token_shapes(tq, oracle, E, H, I, topk):
    """The single-token path (gate/up, then down with the requant and combine fused) at
    block counts of 1 to 64 per row: ragged last loads, every slot count up to 8, a
    duplicated expert, and down rows of 4 and 8 loads per lane (long intermediate rows at
    one or two slots)."""
    ex, logical = host_experts(tq, oracle, E, H, I, seed=31 + topk)
    rng = np.random.default_rng(32 + topk)
    x = (rng.standard_normal((1, H)) * 3).astype(np.float32)
    idx = rng.choice(E, topk, replace=False).astype(np.int32)[None, :]
    if topk >= 3:
        idx[0, 2] = idx[0, 0]
    w = rng.uniform(0.1, 1.0, (1, topk)).astype(np.float32)
    announce(f"moe t=1 E={E} H={H} I={I} topk={topk}")
    out, ws = run_moe(tq, ex, x, idx, w)
    check_moe(tq, oracle, ex, lambda e: logical[e], x, idx, w, out, ws, [0])
    assert tq.tq_moe_status(ws, ex, 1, topk) == 0


@pytest.mark.parametrize("E,H,I,T,topk", [(3, 1024, 512, 40, 2), (4, 7168, 512, 9, 3)])
def test_moe_grouped_valu_long_lists(tq, oracle, E, H, I, T, topk):
    """The grouped VALU path with many tokens per expert (several token chunks plus a
    remainder) and a ragged 28-block hidden size."""
    ex, logical = host_experts(tq, oracle, E, H, I, seed=41)
    rng = np.random.default_rng(42)
    x = rng.standard_normal((T, H)).astype(np.float32)
    idx = np.stack([rng.choice(E, topk, replace=False) for _ in range(T)]).astype(np.int32)
    w = rng.uniform(0.1, 1.0, (T, topk)).astype(np.float32)
    announce(f"moe valu E={E} H={H} I={I} T={T}")
    out, ws = run_moe(tq, ex, x, idx, w, flags=tq.TQ_MOE_FORCE_VALU)
    check_moe(tq, oracle, ex, lambda e: logical[e], x, idx, w, out, ws, list(range(T)))
    assert_debug_flag_neutral(tq, ex, x, idx, w, out, flags=tq.TQ_MOE_FORCE_VALU)


def test_moe_workspace_shared_across_paths(tq, experts_h4096):
    """One prepared workspace serves single-token and grouped calls in any order (the
    grouped call pinned to the VALU kernels, whose per-row arithmetic is the single-token
    kernels' own, so that token 0's output agrees bitwise; the mixed path's MFMA tiles
    sum the block terms in another fp32 order and are checked against the oracle in the
    32-token test)."""
    c = gen.CONFIGS[2]
    ws = tq.moe_workspace(experts_h4096, c["tokens"], c["topk"])
    x = gen.activations(gen.SEED, 60, c["tokens"], c["hidden"])
    idx, w = gen.routing(gen.SEED, 60, c["tokens"], c["experts"], c["topk"], c["routing"])
    xd, idd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(idx).cuda(), torch.from_numpy(w).cuda()
    outs = []
    announce("moe workspace shared: t=1, t=32, t=1")
    for t in (1, c["tokens"], 1):
        out = torch.empty((t, c["hidden"]), dtype=torch.float32, device="cuda")
        tq.tq_moe_grouped(experts_h4096, xd[:t], idd[:t], wd[:t], out, ws, tq.TQ_MOE_FORCE_VALU)
        outs.append(out)
        assert tq.tq_moe_status(ws, experts_h4096, t, c["topk"]) == 0
    assert torch.equal(outs[0], outs[2]) and torch.equal(outs[0], outs[1][:1])


def test_t1_repeated_calls_share_one_workspace(tq, oracle):
    """Forty single-token calls in a row on one workspace, routing and x changing every
    call: each output is bitwise the output of the same call on a fresh workspace, and
    the last call's stages match the oracle."""
    E, H, I, topk = 16, 1024, 512, 8
    ex, logical = host_experts(tq, oracle, E, H, I, seed=71)
    rng = np.random.default_rng(72)
    n = 40
    xs = rng.standard_normal((n, 1, H)).astype(np.float32)
    idx = np.stack([rng.choice(E, topk, replace=False)[None, :] for _ in range(n)]).astype(np.int32)
    w = rng.uniform(0.1, 1.0, (n, 1, topk)).astype(np.float32)
    announce(f"moe t=1 repeated x{n} E={E} H={H} I={I}")
    ws = tq.moe_workspace(ex, 1, topk)
    outs = []
    for i in range(n):
        out = torch.empty((1, H), dtype=torch.float32, device="cuda")
        tq.tq_moe_grouped(ex, torch.from_numpy(xs[i]).cuda(), torch.from_numpy(idx[i]).cuda(),
                          torch.from_numpy(w[i]).cuda(), out, ws)
        outs.append(out)
    torch.cuda.synchronize()
    assert tq.tq_moe_status(ws, ex, 1, topk) == 0
    for i in (0, 17, n - 1):
        fresh, _ = run_moe(tq, ex, xs[i], idx[i], w[i])
        assert torch.equal(fresh, outs[i]), f"call {i}"
    # the last call's stages against the oracle
    check_moe(tq, oracle, ex, lambda e: logical[e], xs[-1], idx[-1], w[-1], outs[-1], ws, [0])


def test_t1_unrouted_slots(tq, oracle):
    """Out-of-range expert ids on the single-token path: flagged, and they contribute
    nothing (the routed slots staged, block sums bit-exact, and end to end at 1e-5)."""
    E, H, I, topk = 5, 768, 512, 4
    ex, logical = host_experts(tq, oracle, E, H, I, seed=81)
    rng = np.random.default_rng(82)
    x = rng.standard_normal((1, H)).astype(np.float32)
    idx = np.array([[3, -2, 0, E]], np.int32)
    w = np.array([[0.4, 0.3, 0.2, 0.1]], np.float32)
    announce("moe t=1 unrouted slots")
    out, ws = run_moe(tq, ex, x, idx, w)
    assert tq.tq_moe_status(ws, ex, 1, topk) & 1
    check_moe(tq, oracle, ex, lambda e: logical[e], x, idx, w, out, ws, [0])
    assert_debug_flag_neutral(tq, ex, x, idx, w, out)


def test_t1_graph_replays_match_eager(tq, oracle):
    """Single-token calls captured in a HIP graph: every replay (with eager calls on the
    same workspace between replays) gives bitwise the eager outputs."""
    E, H, I, topk = 12, 4096, 2048, 8
    ex, _ = host_experts(tq, oracle, E, H, I, seed=91)
    rng = np.random.default_rng(92)
    n = 4
    xs = torch.from_numpy(rng.standard_normal((n, 1, H)).astype(np.float32)).cuda()
    idx = torch.from_numpy(np.stack([rng.choice(E, topk, replace=False)[None, :] for _ in range(n)]).astype(np.int32)).cuda()
    w = torch.from_numpy(rng.uniform(0.1, 1.0, (n, 1, topk)).astype(np.float32)).cuda()
    ws = tq.moe_workspace(ex, 1, topk)
    announce("moe t=1 graph capture")
    eager = [torch.empty((1, H), dtype=torch.float32, device="cuda") for _ in range(n)]
    for i in range(n):
        tq.tq_moe_grouped(ex, xs[i], idx[i], w[i], eager[i], ws)
    torch.cuda.synchronize()
    outs = [torch.empty((1, H), dtype=torch.float32, device="cuda") for _ in range(n)]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for i in range(n):
                tq.tq_moe_grouped(ex, xs[i], idx[i], w[i], outs[i], ws, stream=s)
    torch.cuda.synchronize()
    for rep in range(3):
        for o in outs:
            o.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        for i in range(n):
            assert torch.equal(outs[i], eager[i]), f"replay {rep} call {i}"
        tmp = torch.empty((1, H), dtype=torch.float32, device="cuda")
        tq.tq_moe_grouped(ex, xs[rep], idx[rep], w[rep], tmp, ws)  # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(tmp, eager[rep])
    assert tq.tq_moe_status(ws, ex, 1, topk) == 0


@pytest.mark.parametrize("flags,T", [(1, 24), (2, 40), (0, 40)])
def test_grouped_graph_replays_match_eager(tq, oracle, flags, T):
    """Grouped calls (forced VALU, forced MFMA, automatic: the mixed path) captured in a
    HIP graph, each call with its own routing: every replay (with eager calls on the same
    workspace between replays) gives bitwise the eager outputs, so the dispatch's counters
    and lists are rebuilt on every replay."""
    E, H, I, topk = 16, 1024, 512, 4
    ex, _ = host_experts(tq, oracle, E, H, I, seed=93 + flags)
    rng = np.random.default_rng(94 + flags)
    n = 3
    xs = torch.from_numpy(rng.standard_normal((n, T, H)).astype(np.float32)).cuda()
    idx = torch.from_numpy(np.stack([np.stack([rng.choice(E, topk, replace=False) for _ in range(T)])
                                     for _ in range(n)]).astype(np.int32)).cuda()
    w = torch.from_numpy(rng.uniform(0.1, 1.0, (n, T, topk)).astype(np.float32)).cuda()
    ws = tq.moe_workspace(ex, T, topk)
    announce(f"moe grouped graph capture flags={flags} T={T}")
    eager = [torch.empty((T, H), dtype=torch.float32, device="cuda") for _ in range(n)]
    for i in range(n):
        tq.tq_moe_grouped(ex, xs[i], idx[i], w[i], eager[i], ws, flags=flags)
    torch.cuda.synchronize()
    outs = [torch.empty((T, H), dtype=torch.float32, device="cuda") for _ in range(n)]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for i in range(n):
                tq.tq_moe_grouped(ex, xs[i], idx[i], w[i], outs[i], ws, flags=flags, stream=s)
    torch.cuda.synchronize()
    for rep in range(3):
        for o in outs:
            o.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        for i in range(n):
            assert torch.equal(outs[i], eager[i]), f"replay {rep} call {i}"
        tmp = torch.empty((T, H), dtype=torch.float32, device="cuda")
        tq.tq_moe_grouped(ex, xs[rep], idx[rep], w[rep], tmp, ws, flags=flags)  # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(tmp, eager[rep])
    assert tq.tq_moe_status(ws, ex, T, topk) == 0
    assert tq.tq_moe_path(ex, T, topk, flags) == {1: tq.TQ_MOE_PATH_VALU, 2: tq.TQ_MOE_PATH_MFMA,
                                                   0: tq.TQ_MOE_PATH_MIXED}[flags]
