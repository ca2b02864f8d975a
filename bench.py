"""Benchmark of the tied-trit-plane expert dot pass on one MI355X.

Workload (one step = one pass of the whole hot path): one routed-expert MoE layer at
decode, batch 1 -- 256 experts resident in HBM (hidden 4096, expert intermediate 2048,
gate/up/down in the folded 4.0625 bit/weight format, 3.27 GB), one token, top-8 experts
uniform without replacement with softmax weights: quantize x, dispatch, gate/up dot pass
with SiLU(gate)*up, requantize, down dot pass, weighted combine.

Every step routes to experts not used in the previous 3 steps (a reuse distance above
the 256 MB last-level cache), each with its own token; all inputs are resident in HBM
before timing. Steps are captured in HIP graphs (W warmup steps, then exactly K timed
steps) and timed by wall clock between device synchronizations.

`value` = algorithmic bytes moved per step (the routed experts' codes and scales, x in,
out) x K / time, in GB/s; `tokens_per_s` = tokens x K / time.

The roofline object covers the dominant kernel (gate_up): its algorithmic bytes per
launch divided by its mean duration, measured here with HIP events recorded on the
launch stream around that kernel over a second run of the same steps.

The CPU baseline times the oracle (single-threaded C) on a bounded sample of the same
layer on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "achieved HBM GB/s (% of peak) for tq expert GEMV; MoE-layer tokens/sec"
HBM_PEAK_GBS = 8000.0


def recorded_traffic(kernel: str):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter summary, or
    None if no record exists or the kernel's sources changed since it was taken."""
    import glob
    import hashlib
    for path in glob.glob(os.path.join(ROOT, "profiles", "*traffic*.md")):
        for line in open(path):
            line = line.strip()
            if not line.startswith('{"kernel"'):
                continue
            rec = json.loads(line)
            if rec["kernel"] != kernel:
                continue
            h = hashlib.sha256()
            for f in rec["sources"]:
                h.update(open(os.path.join(ROOT, f), "rb").read())
            if h.hexdigest() == rec["sources_sha256"]:
                return rec["traffic_bytes_per_launch"]
    return None


def matrix_bytes(n: int, k: int) -> int:
    return n * k // 2 + n * (k // 256) * 2


def cpu_baseline(seed: int, hidden: int, inter: int, topk: int, target_s: float = 12.0) -> dict:
    """Oracle (plain single-threaded C + numpy glue) on a bounded sample of the same layer."""
    import oracle as oracle_pkg
    from synth import gen

    o = oracle_pkg.get()
    experts = {}
    for e in range(topk):  # the sample's experts, generated before timing
        experts[e] = {
            "gate": o.synth_codes(gen.matrix_key(seed, 0, e, gen.PROJ_GATE), inter, hidden),
            "up": o.synth_codes(gen.matrix_key(seed, 0, e, gen.PROJ_UP), inter, hidden),
            "down": o.synth_codes(gen.matrix_key(seed, 0, e, gen.PROJ_DOWN), hidden, inter),
        }
    idx = np.arange(topk, dtype=np.int32)[None, :]
    w = np.full((1, topk), 1.0 / topk, np.float32)
    x0 = gen.activations(seed, 0, 1, hidden)
    t0 = time.perf_counter()
    o.moe(x0, idx, w, experts.__getitem__)
    one = time.perf_counter() - t0
    n_tok = int(max(1, min(200, target_s / max(one, 1e-3))))
    xs = gen.activations(seed, 1, n_tok, hidden)
    t0 = time.perf_counter()
    for i in range(n_tok):
        o.moe(xs[i:i + 1], idx, w, experts.__getitem__)
    el = time.perf_counter() - t0
    per_tok = topk * (2 * matrix_bytes(inter, hidden) + matrix_bytes(hidden, inter)) + 2 * hidden * 4
    return {
        "value": round(per_tok * n_tok / el / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
        "tokens_per_s": round(n_tok / el, 3),
        "sample": f"{n_tok} tokens of the batch-1 decode layer, each routed to the same {topk} pre-generated "
                  f"experts (hidden {hidden}, inter {inter}); oracle compute only, weight generation excluded; "
                  f"{el:.1f} s on 1 host thread",
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-steps", type=int, default=256, help="steps of the per-kernel event pass")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (to scale HBM byte counters)")
    args = ap.parse_args()
    if args.calibrate_copy:
        import torch
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda:0")  # 1 GiB
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(10):
            dst.copy_(src)
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
        print(json.dumps({"calibrate_copy_bytes": src.numel() * 4, "copies": 13,
                          "copy_GBps_read_plus_write": round(10 * 2 * src.numel() * 4 / el / 1e9, 1)}))
        return
    if args.gpus != 1:
        print(f"bench.py: this build measures one GPU only (--gpus {args.gpus} requested); "
              "the expert-parallel multi-GPU path is not built", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_08910_amd import tq
    from synth import gen

    cfg = gen.CONFIGS[1]
    E, H, I, T, topk, seed = cfg["experts"], cfg["hidden"], cfg["inter"], cfg["tokens"], cfg["topk"], gen.SEED
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    # resident experts, generated on the device
    ex = tq.TqExperts.empty(E, H, I, device=dev)
    for e in range(E):
        for p in range(3):
            tq.tq_synth_weights(gen.matrix_key(seed, 0, e, p), ex.matrix(e, p))
    torch.cuda.synchronize()

    K, W, P = args.steps, args.warmup, args.profile_steps
    total = W + K
    sched = gen.bench_routing_schedule(seed, total, T, E, topk, cfg["routing"])
    idx_all = torch.from_numpy(np.stack([s[0] for s in sched])).to(dev)          # [steps][T][topk]
    w_all = torch.from_numpy(np.stack([s[1] for s in sched])).to(dev)
    x_all = torch.from_numpy(gen.activations(seed, 1000, total * T, H).reshape(total, T, H)).to(dev)
    out = torch.empty((T, H), dtype=torch.float32, device=dev)
    ws = torch.empty(tq.tq_moe_workspace_bytes(ex, T, topk), dtype=torch.uint8, device=dev)

    def step(i):
        tq.tq_moe_grouped(ex, x_all[i], idx_all[i], w_all[i], out, ws)

    # eager sanity pass (also loads the code objects)
    for i in range(min(W, 8)):
        step(i)
    torch.cuda.synchronize()

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g_warm, g_time = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g_warm, stream=s):
            for i in range(W):
                step(i)
        with torch.cuda.graph(g_time, stream=s):
            for i in range(W, W + K):
                step(i)
    torch.cuda.synchronize()

    g_warm.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    g_time.replay()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    bytes_expert = 2 * matrix_bytes(I, H) + matrix_bytes(H, I)
    distinct = [len(np.unique(sched[i][0])) for i in range(W, W + K)]
    alg_bytes = sum(d * bytes_expert for d in distinct) + K * (T * H * 4 * 2 + T * topk * 8)
    gbs = alg_bytes / elapsed / 1e9

    # per-kernel pass: events around every stage, eager launches queued behind a spin
    # kernel so the GPU runs the stages back to back
    nst = tq.tq_moe_stage_count()
    names = [tq.tq_moe_stage_name(i) for i in range(nst)]
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2 * nst)] for _ in range(P)]
    torch.cuda.synchronize()
    torch.cuda._sleep(int(2.4e9 * 0.05))  # ~50 ms of queue head-room
    for j in range(P):
        i = W + (j % K)
        tq.tq_moe_grouped_timed(ex, x_all[i], idx_all[i], w_all[i], out, ws, evs[j])
    torch.cuda.synchronize()
    stage_ms = {n: float(np.mean([evs[j][2 * si].elapsed_time(evs[j][2 * si + 1]) for j in range(P)]))
                for si, n in enumerate(names)}
    gu = names.index("gate_up")
    gu_ms = stage_ms["gate_up"]
    # gate_up moves the routed experts' gate and up codes + scales, reads x (fp32) and
    # writes h (fp32, one row per slot)
    gu_bytes = float(np.mean([len(np.unique(sched[W + (j % K)][0])) for j in range(P)])) * 2 * matrix_bytes(I, H) \
        + T * H * 4 + T * topk * I * 4
    achieved = gu_bytes / (gu_ms * 1e-3) / 1e9
    # the single-token step's gate/up kernel (hidden 4096: two 16-byte loads per row and lane)
    gu_kernel = "k_t1_gateup<2, 4, 4, false>"
    traffic = recorded_traffic(gu_kernel)

    res = {
        "metric": METRIC,
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(elapsed * 1e3 / K, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": cfg["name"], "experts": E, "hidden": H, "inter": I, "tokens_per_step": T,
                   "topk": topk, "routing": "uniform top-8, no expert reused within 3 steps",
                   "bits_per_weight": 4.0625, "resident_expert_bytes": E * bytes_expert},
        "pct_of_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
        "tokens_per_s": round(K * T / elapsed, 1),
        "stage_ms": {k: round(v, 5) for k, v in stage_ms.items()},
        "roofline": {"kernel": "gate_up", "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "bytes_per_launch": round(gu_bytes), "mean_ms": round(gu_ms, 5),
                     "kernel_symbol": gu_kernel},
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(seed, H, I, topk)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
