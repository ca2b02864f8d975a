"""Benchmark of the tied-trit-plane expert dot pass on one MI355X.

Default workload (one step = one pass of the whole hot path): one routed-expert MoE
layer at decode, batch 1 -- 256 experts resident in HBM (hidden 4096, expert
intermediate 2048, gate/up/down in the folded 4.0625 bit/weight format, 3.27 GB), one
token, top-8 experts uniform without replacement with softmax weights: quantize x,
dispatch, gate/up dot pass with SiLU(gate)*up, requantize, down dot pass, weighted
combine.

Other workloads (--workload): `decode32` (32 tokens, Zipf top-8), `prefill2048` (2048
tokens, Zipf top-8, per-token log-uniform factors; the expert contraction runs on int8
MFMA), `stack43` (a decode step through 43 such layers at hidden 7168, 8 tokens,
Zipf top-8: 246 GB of experts resident), `gemv` (the single 2048 x 4096 matrix, one
token: quantize + dot pass), `tiedquant` (the tied quantizer that produces the code
plane: one 2048 x 4096 fp32 matrix per step, rotating over 32), `twoplane` (the
free-scale two-plane variant, 4.125 bits/weight: one decode step's routed gate and up
rows as one 32768 x 4096 matrix, one token, rotating over 8 copies; the folded pass over
the same trit planes is timed beside it, and both kernels at 1, 4 and 16 tokens),
`mxfp4` (the MXFP4 reference arm, 4.25 bits/weight, same shape and protocol, the folded
pass over a folded matrix of that shape beside it), `stream` (the batch-1 decode layer
with every expert in pinned host memory and an LRU pool of --slots expert slots in HBM:
misses copied over the host link each step, eager steps), `freequant` (the free-scale
solver refining each matrix's tied fit, same matrices as `tiedquant`).

Cache hygiene: every step touches bytes that cannot still sit in the 256 MB last-level
cache. Batch-1 steps route to experts not used in the previous 3 steps (reuse distance
above the cache); the larger steps move 1-37 GB each; the GEMV rotates over 128
distinct copies of its matrix (545 MB). All inputs are resident in HBM before timing.
Steps are captured in HIP graphs (W warmup steps, then exactly K timed steps) and
timed by wall clock between device synchronizations.

`value` = algorithmic bytes moved per step (the routed experts' codes and scales, or
the matrix; activations in, outputs out) x K / time, in GB/s.

The roofline object covers the dominant kernel: its algorithmic bytes (or int8 ops, on
the MFMA path) per launch divided by its mean duration, measured here with HIP events
recorded on the launch stream around that kernel over a second run of the same steps.

The CPU baseline (default workload only) times the oracle (single-threaded C) on a
bounded sample of the same layer on this host.
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
MFMA_I8_PEAK_TOPS = 5000.0
# VALU issue: each of a CU's 4 SIMDs starts one wave64 VALU instruction every 4 cycles
# (16 lanes a cycle); 256 CUs at 2.4 GHz
VALU_PEAK_GINST = 256 * 4 * 2.4 / 4


def _recorded(kernel: str, field: str, kind: str = "traffic"):
    """`field` of the committed rocprofv3 counter record of `kernel` (profiles/*<kind>*.md),
    or None if no record exists or the kernel's sources changed since it was taken."""
    import glob
    import hashlib
    for path in glob.glob(os.path.join(ROOT, "profiles", f"*{kind}*.md")):
        for line in open(path):
            line = line.strip()
            if not line.startswith('{"kernel"'):
                continue
            rec = json.loads(line)
            if rec["kernel"] != kernel or field not in rec:
                continue
            h = hashlib.sha256()
            for f in rec["sources"]:
                h.update(open(os.path.join(ROOT, f), "rb").read())
            if h.hexdigest() == rec["sources_sha256"]:
                return rec[field]
    return None


def recorded_traffic(kernel: str):
    """HBM bytes per launch of `kernel` (FETCH_SIZE + WRITE_SIZE, calibrated)."""
    return _recorded(kernel, "traffic_bytes_per_launch")


def matrix_bytes(n: int, k: int) -> int:
    return n * k // 2 + n * (k // 256) * 2


def host_info() -> dict:
    """The host the CPU legs ran on: logical CPUs, the ones this process may use, the model."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "usable_cpus": len(os.sched_getaffinity(0)), "cpu_model": model}


def cpu_baseline(seed: int, hidden: int, inter: int, topk: int, target_s: float = 8.0) -> dict:
    """The oracle (plain C, its dot pass row-parallel under OpenMP, + numpy glue) on a
    bounded sample of the same layer, on all usable host cores and on one."""
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
    per_tok = topk * (2 * matrix_bytes(inter, hidden) + matrix_bytes(hidden, inter)) + 2 * hidden * 4
    info = host_info()

    def leg(threads: int, salt: int):
        used = o.set_threads(threads)
        x0 = gen.activations(seed, salt, 1, hidden)
        t0 = time.perf_counter()
        o.moe(x0, idx, w, experts.__getitem__)
        one = time.perf_counter() - t0
        n_tok = int(max(1, min(400, target_s / max(one, 1e-3))))
        xs = gen.activations(seed, salt + 1, n_tok, hidden)
        t0 = time.perf_counter()
        for i in range(n_tok):
            o.moe(xs[i:i + 1], idx, w, experts.__getitem__)
        el = time.perf_counter() - t0
        return used, n_tok, el

    used_all, n_all, el_all = leg(info["usable_cpus"], 1)
    _, n_one, el_one = leg(1, 3)
    o.set_threads(info["usable_cpus"])
    return {
        "value": round(per_tok * n_all / el_all / 1e9, 4), "unit": "GB/s", "cores": used_all, "kind": "oracle",
        "tokens_per_s": round(n_all / el_all, 3),
        "one_core": {"value": round(per_tok * n_one / el_one / 1e9, 4), "unit": "GB/s", "cores": 1,
                     "tokens_per_s": round(n_one / el_one, 3)},
        **info,
        "sample": f"{n_all} tokens ({el_all:.1f} s on {used_all} OpenMP threads) and {n_one} tokens ({el_one:.1f} s "
                  f"on 1 thread) of the batch-1 decode layer, each routed to the same {topk} pre-generated experts "
                  f"(hidden {hidden}, inter {inter}); oracle compute only, weight generation excluded",
    }


WORKLOADS = {
    "decode1": dict(cfg=1, steps=2000, warmup=200, profile=256),
    "decode32": dict(cfg=2, steps=300, warmup=30, profile=64),
    # (a graph's first replay carries about 1 ms of one-time launch cost: enough steps that
    # it stays near 1% of the timed region)
    "prefill2048": dict(cfg=3, steps=100, warmup=10, profile=4),
    "stack43": dict(cfg=4, steps=20, warmup=3, profile=2),
    "gemv": dict(cfg=0, steps=4000, warmup=400, profile=512),
    "tiedquant": dict(cfg="quant", steps=64, warmup=8, profile=32),
    "twoplane": dict(cfg="twoplane", steps=2000, warmup=200, profile=256),
    "mxfp4": dict(cfg="mxfp4", steps=2000, warmup=200, profile=256),
    "stream": dict(cfg=1, steps=200, warmup=20, profile=0, stream=True),
    "freequant": dict(cfg="quant", steps=64, warmup=8, profile=32, free=True),
}


REPLAYS = 20  # repeats of the timed graph for the median and min-max band
USE_GRAPH = True  # --no-graph: eager launches (for profiler counter passes, which only need the dispatches)


def time_graph(step, W: int, K: int):
    """Capture W warmup and K timed steps in two HIP graphs; replay the warmup graph,
    then time the K-step graph between device synchronizations (seconds). Then replay
    the K-step graph REPLAYS more times, each bracketed by HIP events on its stream, for
    the band (seconds per replay). Without graphs (USE_GRAPH false): the same steps
    launched eagerly, timed by wall clock, no band."""
    import torch
    if not USE_GRAPH:
        for i in range(W):
            step(i)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(W, W + K):
            step(i)
        torch.cuda.synchronize()
        return time.perf_counter() - t0, None
    for i in range(min(W, 4)):  # eager sanity pass (also loads the code objects)
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
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(REPLAYS)]
    with torch.cuda.stream(s):
        for a, b in evs:
            a.record(s)
            g_time.replay()
            b.record(s)
    torch.cuda.synchronize()
    return elapsed, [a.elapsed_time(b) * 1e-3 for a, b in evs]


def hbm_roof(kernel, nbytes, ms, symbol):
    """The dominant kernel against the HBM roof. `frac` uses `mean_ms`: the mean of the
    kernel's own start/stop timestamps (HIP events of hipExtLaunchKernelGGL) over the eager
    launches of the per-kernel pass. Beside it, the committed rocprofv3 record of the same
    kernel (its AverageNs), while the kernel's sources are unchanged since it was taken."""
    achieved = nbytes / (ms * 1e-3) / 1e9
    r = {"kernel": kernel, "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
         "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": recorded_traffic(symbol),
         "bytes_per_launch": round(nbytes), "mean_ms": round(ms, 5), "kernel_symbol": symbol,
         "frac_timing": "hip events: the kernel's own start/stop timestamps, mean over the per-kernel pass"}
    avg_ns = _recorded(symbol, "average_ns", kind="kernel_stats")
    if avg_ns is not None:
        r["rocprof_mean_ms"] = round(avg_ns * 1e-6, 5)
        r["frac_rocprof"] = round(nbytes / (avg_ns * 1e-9) / 1e9 / HBM_PEAK_GBS, 4)
    return r


def stream_ceiling(nbytes: float, launches: int) -> dict:
    """A plain streaming read of nbytes in one launch (tq_stream_read_timed), from a
    device buffer at rotating offsets (each read's bytes last touched at least 1 GiB of
    reads earlier, beyond the 256 MB last-level cache); the launches queued back to back
    behind a spin kernel, each timed by its own start/stop timestamps. Median over the
    launches."""
    import torch
    from paper_2608_08910_amd import tq
    nb = int(nbytes + 255) // 256 * 256
    span = max(1 << 30, 3 * nb) // 256 * 256
    buf = torch.empty(span + nb, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(launches)]
    torch.cuda.synchronize()
    torch.cuda._sleep(int(2.4e9 * 0.02))
    for i in range(launches):
        off = (i * nb) % span
        tq.tq_stream_read_timed(buf[off:], nb, sink, ev[i])
    torch.cuda.synchronize()
    ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    del buf
    return {"bytes": nb, "ms": round(ms, 5), "GBps": round(nb / (ms * 1e-3) / 1e9, 1)}


def run_gemv(args, wl, cfg):
    import torch
    from paper_2608_08910_amd import tq
    from synth import gen

    n, k, seed = cfg["n"], cfg["k"], gen.SEED
    K = args.steps if args.steps is not None else wl["steps"]
    W = args.warmup if args.warmup is not None else wl["warmup"]
    P = args.profile_steps if args.profile_steps is not None else wl["profile"]
    copies = 128  # 128 x 4.26 MB = 545 MB > the 256 MB last-level cache
    mats = [tq.TqMatrix.empty(n, k) for _ in range(copies)]
    for i, m in enumerate(mats):
        tq.tq_synth_weights(gen.matrix_key(seed, 0xFFFF, i, 0), m)  # copy 0 is the workload's matrix
    total = W + K
    x_all = torch.from_numpy(gen.activations(seed, 1000, total, k)).cuda()
    q = torch.empty((1, k), dtype=torch.int8, device="cuda")
    d = torch.empty((1, k // 256), dtype=torch.float32, device="cuda")
    b = torch.empty((1, k // 256), dtype=torch.int32, device="cuda")
    y = torch.empty((1, n), dtype=torch.float32, device="cuda")

    def step(i):
        # fp32 activations in, quantized inside the dot-pass launch
        tq.tq_gemv_f32(mats[i % copies], x_all[i:i + 1], y, q, d, b)

    elapsed, reps = time_graph(step, W, K)
    per_step = matrix_bytes(n, k) + k * 4 + n * 4
    gbs = per_step * K / elapsed / 1e9
    # per-kernel pass: each launch with its own start/stop events (the kernel's
    # timestamps), eager launches queued behind a spin kernel
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(P)]
    torch.cuda.synchronize()
    torch.cuda._sleep(int(2.4e9 * 0.02))
    for j in range(P):
        tq.tq_gemv_f32_timed(mats[j % copies], x_all[j:j + 1], y, q, d, b, ev[j])
    torch.cuda.synchronize()
    ms = float(np.mean([a.elapsed_time(c) for a, c in ev]))
    # the kernel reads the codes, scales and x (fp32) and writes y (and q, d, bsum once)
    roof = hbm_roof("gemv", per_step, ms, "k_gemv_x<2, 1, 4, false>")
    ceil = stream_ceiling(per_step, 64)
    step_ms = elapsed * 1e3 / K
    return dict(value=gbs, K=K, W=W, elapsed=elapsed, reps=reps, tokens=K, roof=roof,
                config={"workload": cfg["name"], "n": n, "k": k, "tokens_per_step": 1, "bits_per_weight": 4.0625,
                        "rotating_copies": copies, "path": "valu, quantization fused (tq_gemv_f32)"},
                extra={"stream_ceiling": {"step_bytes": ceil["bytes"], "stream_read_GBps": ceil["GBps"],
                                          "stream_read_ms": ceil["ms"],
                                          "step_frac_of_stream_read": round(ceil["ms"] / step_ms, 4)}})


def cpu_baseline_quant(cfg, target_s: float = 10.0) -> dict:
    """The oracle's tied solver (plain single-threaded C) on the workload's first matrix,
    repeated to about target_s seconds."""
    import oracle as oracle_pkg
    from synth import gen

    o = oracle_pkg.get()
    w = gen.float_weights(gen.SEED, 0, cfg["n"], cfg["k"])
    t0 = time.perf_counter()
    o.tied_quantize(w[:64])
    per_row = (time.perf_counter() - t0) / 64
    reps = int(max(1, min(64, round(target_s / max(per_row * cfg["n"], 1e-6)))))
    t0 = time.perf_counter()
    for _ in range(reps):
        o.tied_quantize(w)
    el = time.perf_counter() - t0
    nbytes = reps * (cfg["n"] * cfg["k"] * 4 + matrix_bytes(cfg["n"], cfg["k"]))
    return {"value": round(nbytes / el / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "weights_per_s": round(reps * cfg["n"] * cfg["k"] / el, 1),
            "sample": f"the workload's first {cfg['n']} x {cfg['k']} matrix, {reps} times; {el:.1f} s on 1 host thread"}


def run_quant(args, wl, cfg):
    import torch
    from paper_2608_08910_amd import tq
    from synth import gen

    M, n, k = cfg["matrices"], cfg["n"], cfg["k"]
    K = args.steps if args.steps is not None else wl["steps"]
    W = args.warmup if args.warmup is not None else wl["warmup"]
    P = args.profile_steps if args.profile_steps is not None else wl["profile"]
    # 32 x 33.5 MB of fp32 weights (1.07 GB, beyond the 256 MB last-level cache), one
    # matrix per step in rotation
    free = wl.get("free", False)
    ws = [torch.from_numpy(gen.float_weights(gen.SEED, i, n, k)).cuda() for i in range(M)]
    outs = [tq.TqMatrix.empty(n, k) for _ in range(M)]
    iters = torch.empty((n, k // 256), dtype=torch.uint8, device="cuda")
    if free:
        # the free-scale solver refines each matrix's tied fit (computed once, untimed)
        for i in range(M):
            tq.tq_tied_quantize(ws[i], outs[i])
        outs2 = [tq.TqMatrix2.empty(n, k) for _ in range(M)]
    torch.cuda.synchronize()

    def run(i, it=None):
        if free:
            tq.tq_free_quantize(ws[i % M], outs[i % M], outs2[i % M], it)
        else:
            tq.tq_tied_quantize(ws[i % M], outs[i % M], it)

    def step(i):
        run(i)

    elapsed, reps = time_graph(step, W, K)
    # bytes: fp32 weights in, the format out (and the tied fit in, for the free solver)
    per_step = n * k * 4 + (matrix_bytes(n, k) + n * k // 2 + n * (k // 256) * 4 if free else matrix_bytes(n, k))
    gbs = per_step * K / elapsed / 1e9
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(P)]
    torch.cuda.synchronize()
    for j in range(P):
        ev[j][0].record()
        run(j)
        ev[j][1].record()
    torch.cuda.synchronize()
    ms = float(np.mean([a.elapsed_time(c) for a, c in ev]))
    run(0, iters)
    torch.cuda.synchronize()
    steps = iters.to(torch.float32)
    sym = "k_free_quantize" if free else "k_tied_quantize"
    fit = {}
    if free:
        # relative Frobenius reconstruction error of both fits of matrix 0 (host, fp64)
        w0 = ws[0].cpu().numpy().astype(np.float64).reshape(n, k // 256, 256)
        tc = tq.tq_unpack_host(outs[0].codes.cpu().numpy(), n, k).astype(np.float64).reshape(n, k // 256, 256)
        ts = outs[0].scales.cpu().numpy().view(np.float16).astype(np.float64)
        p1, p2 = tq.tq_unpack2_host(outs2[0].codes.cpu().numpy(), n, k)
        fa = outs2[0].scales.cpu().numpy().view(np.float16).astype(np.float64)
        rt = tc * ts[:, :, None]
        rf = p1.reshape(n, k // 256, 256) * fa[:, :, 0, None] + p2.reshape(n, k // 256, 256) * fa[:, :, 1, None]
        nw = np.sqrt((w0 ** 2).sum())
        fit = {"tied_rel_frobenius_error": round(float(np.sqrt(((w0 - rt) ** 2).sum()) / nw), 5),
               "free_rel_frobenius_error": round(float(np.sqrt(((w0 - rf) ** 2).sum()) / nw), 5)}
    valu = _recorded(sym, "valu_insts_per_launch", "valu")
    if valu is None:  # no current instruction count: fall back to the bytes
        roof = hbm_roof("free_quantize" if free else "tied_quantize", per_step, ms, sym)
    else:
        # the kernel is bound by VALU issue: its wave64 VALU instructions per launch
        # (SQ_INSTS_VALU, rocprofv3, committed record) over its mean duration
        achieved = valu / (ms * 1e-3) / 1e9
        roof = {"kernel": "free_quantize" if free else "tied_quantize", "bound": "alu", "achieved": round(achieved, 1), "peak": VALU_PEAK_GINST,
                "unit": "G VALU wave64 instructions/s", "frac": round(achieved / VALU_PEAK_GINST, 4),
                "traffic": recorded_traffic(sym), "valu_insts_per_launch": valu, "bytes_per_launch": per_step,
                "hbm_GBps": round(per_step / (ms * 1e-3) / 1e9, 1), "mean_ms": round(ms, 5), "kernel_symbol": sym}
    return dict(value=gbs, K=K, W=W, elapsed=elapsed, reps=reps, tokens=K, roof=roof,
                config={"workload": cfg["name"].replace("tied", "free") if free else cfg["name"], "matrices": M,
                        "n": n, "k": k, "max_iter": 16,
                        "weights": "N(0,1) x per-row spread log-uniform [0.005, 0.05], fp32"},
                extra={"weights_per_s": round(n * k * K / elapsed, 1),
                       ("mean_plane_steps_per_block" if free else "mean_code_steps_per_block"): round(float(steps.mean()), 3),
                       ("max_plane_steps_per_block" if free else "max_code_steps_per_block"): int(steps.max()), **fit})


def cpu_baseline_twoplane(cfg, target_s: float = 10.0) -> dict:
    """The oracle's two-plane pass (plain single-threaded C) over the workload's matrix,
    one token per call, repeated to about target_s seconds."""
    import oracle as oracle_pkg
    from synth import gen

    o = oracle_pkg.get()
    n, k = cfg["n"], cfg["k"]
    t1, t2, a = gen.two_plane_weights(gen.SEED, 0, n, k)
    xs = gen.activations(gen.SEED, 1000, 64, k)
    q, d, _ = o.quantize(xs)
    t0 = time.perf_counter()
    o.gemv2(t1, t2, a, q[:1], d[:1])
    one = time.perf_counter() - t0
    reps = int(max(1, min(64, round(target_s / max(one, 1e-6)))))
    t0 = time.perf_counter()
    for i in range(reps):
        o.gemv2(t1, t2, a, q[i:i + 1], d[i:i + 1])
    el = time.perf_counter() - t0
    nbytes = reps * (two_plane_bytes(n, k) + k * 4 + n * 4)
    return {"value": round(nbytes / el / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"the workload's {n} x {k} two-plane matrix, {reps} single-token passes (quantized "
                      f"activations precomputed); {el:.1f} s on 1 host thread"}


def two_plane_bytes(n: int, k: int) -> int:
    return n * k // 2 + n * (k // 256) * 4


def run_twoplane(args, wl, cfg):
    """The free-scale two-plane pass on one decode step's routed gate and up rows, with
    the folded pass over the same trit planes timed beside it."""
    import torch
    from paper_2608_08910_amd import tq
    from synth import gen

    n, k, seed = cfg["n"], cfg["k"], gen.SEED
    kb = k // 256
    K = args.steps if args.steps is not None else wl["steps"]
    W = args.warmup if args.warmup is not None else wl["warmup"]
    P = args.profile_steps if args.profile_steps is not None else wl["profile"]
    copies = 8  # 8 x 69 MB per format > the 256 MB last-level cache
    t1, t2, a = gen.two_plane_weights(seed, 0, n, k)
    c2 = torch.from_numpy(tq.tq_pack2_host(t1, t2)).cuda()
    s2 = torch.from_numpy(a.view(np.int16)).cuda()
    cf = torch.from_numpy(tq.tq_fold_pack_host(t1, t2)).cuda()
    sf = s2[:, :, 1].contiguous()
    del t1, t2
    mats2 = [tq.TqMatrix2(n, k, c2.clone(), s2.clone()) for _ in range(copies)]
    matsf = [tq.TqMatrix(n, k, cf.clone(), sf.clone()) for _ in range(copies)]
    total = W + K
    x_all = torch.from_numpy(gen.activations(seed, 1000, total + 16, k)).cuda()
    T_MAX = 16
    q = torch.empty((T_MAX, k), dtype=torch.int8, device="cuda")
    d = torch.empty((T_MAX, kb), dtype=torch.float32, device="cuda")
    b = torch.empty((T_MAX, kb), dtype=torch.int32, device="cuda")
    y = torch.empty((T_MAX, n), dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()

    def step2(i):
        tq.tq_quantize_act(x_all[i:i + 1], q[:1], d[:1], b[:1])
        tq.tq_gemv2(mats2[i % copies], q[:1], d[:1], y[:1])

    def stepf(i):
        tq.tq_quantize_act(x_all[i:i + 1], q[:1], d[:1], b[:1])
        tq.tq_gemv(matsf[i % copies], q[:1], d[:1], b[:1], y[:1])

    elapsed, reps = time_graph(step2, W, K)
    elapsed_f, _ = time_graph(stepf, W, K)
    io = k * 4 + n * 4
    gbs = (two_plane_bytes(n, k) + io) * K / elapsed / 1e9
    gbs_f = (matrix_bytes(n, k) + io) * K / elapsed_f / 1e9

    def kernel_ms(fn, t):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(P)]
        torch.cuda.synchronize()
        torch.cuda._sleep(int(2.4e9 * 0.02))
        for j in range(P):
            tq.tq_quantize_act(x_all[j:j + t], q[:t], d[:t], b[:t])
            fn(j, t, ev[j])
        torch.cuda.synchronize()
        return float(np.mean([s.elapsed_time(e) for s, e in ev]))

    def k2(j, t, ev):
        tq.tq_gemv2_timed(mats2[j % copies], q[:t], d[:t], y[:t], ev)

    def kf(j, t, ev):
        tq.tq_gemv_timed(matsf[j % copies], q[:t], d[:t], b[:t], y[:t], ev)

    by_tokens = {}
    for t in (1, 4, 16):
        m2, mf = kernel_ms(k2, t), kernel_ms(kf, t)
        by_tokens[str(t)] = {"two_plane_ms": round(m2, 5), "folded_ms": round(mf, 5),
                             "two_plane_GBps": round((two_plane_bytes(n, k) + t * (k + kb * 4 + n * 4)) / (m2 * 1e-3) / 1e9, 1),
                             "folded_GBps": round((matrix_bytes(n, k) + t * (k + kb * 4 + n * 4)) / (mf * 1e-3) / 1e9, 1)}
    ms = by_tokens["1"]["two_plane_ms"]
    roof = hbm_roof("gemv2", two_plane_bytes(n, k) + k + kb * 4 + n * 4, ms, "k_gemv2<2, 1, 4, false>")
    return dict(value=gbs, K=K, W=W, elapsed=elapsed, reps=reps, tokens=K, roof=roof,
                config={"workload": cfg["name"], "n": n, "k": k, "tokens_per_step": 1, "bits_per_weight": 4.125,
                        "rotating_copies": copies, "format": "free-scale two-plane (2 x 2-bit trit planes, 2 f16 scales "
                                                             "per 256 weights)"},
                extra={"folded_same_planes": {"value": round(gbs_f, 2), "ms_per_step": round(elapsed_f * 1e3 / K, 5),
                                              "bits_per_weight": 4.0625},
                       "kernel_ms_by_tokens": by_tokens})


def mx_bytes(n: int, k: int) -> int:
    return n * k // 2 + n * (k // 32)


def cpu_baseline_mx(cfg, target_s: float = 10.0) -> dict:
    """The oracle's MXFP4 pass (plain single-threaded C) over the workload's matrix, one
    token per call, repeated to about target_s seconds."""
    import oracle as oracle_pkg
    from synth import gen

    o = oracle_pkg.get()
    n, k = cfg["n"], cfg["k"]
    c4, e8 = gen.mxfp4_weights(gen.SEED, 0, n, k)
    q, d, _ = o.quantize(gen.activations(gen.SEED, 1000, 64, k))
    t0 = time.perf_counter()
    o.gemv_mx(c4, e8, q[:1], d[:1])
    one = time.perf_counter() - t0
    reps = int(max(1, min(64, round(target_s / max(one, 1e-6)))))
    t0 = time.perf_counter()
    for i in range(reps):
        o.gemv_mx(c4, e8, q[i:i + 1], d[i:i + 1])
    el = time.perf_counter() - t0
    nbytes = reps * (mx_bytes(n, k) + k * 4 + n * 4)
    return {"value": round(nbytes / el / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"the workload's {n} x {k} MXFP4 matrix, {reps} single-token passes (quantized activations "
                      f"precomputed); {el:.1f} s on 1 host thread"}


def run_mxfp4(args, wl, cfg):
    """The MXFP4 reference arm's integer pass on one decode step's routed gate and up rows,
    with the folded pass over a folded matrix of the same shape timed beside it."""
    import torch
    from paper_2608_08910_amd import tq
    from synth import gen

    n, k, seed = cfg["n"], cfg["k"], gen.SEED
    kb = k // 256
    K = args.steps if args.steps is not None else wl["steps"]
    W = args.warmup if args.warmup is not None else wl["warmup"]
    P = args.profile_steps if args.profile_steps is not None else wl["profile"]
    copies = 8  # 8 x 71 MB per format > the 256 MB last-level cache
    c4, e8 = gen.mxfp4_weights(seed, 0, n, k)
    cm = torch.from_numpy(tq.tq_mx_pack_host(c4)).cuda()
    sm = torch.from_numpy(e8).cuda()
    del c4, e8
    mats = [tq.TqMatrixMx(n, k, cm.clone(), sm.clone()) for _ in range(copies)]
    matsf = [tq.TqMatrix.empty(n, k) for _ in range(copies)]
    for i, m in enumerate(matsf):
        tq.tq_synth_weights(gen.matrix_key(seed, 0xFFFE, i, 0), m)
    total = W + K
    x_all = torch.from_numpy(gen.activations(seed, 1000, total + 16, k)).cuda()
    T_MAX = 16
    q = torch.empty((T_MAX, k), dtype=torch.int8, device="cuda")
    d = torch.empty((T_MAX, kb), dtype=torch.float32, device="cuda")
    b = torch.empty((T_MAX, kb), dtype=torch.int32, device="cuda")
    y = torch.empty((T_MAX, n), dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()

    def step(i):
        tq.tq_quantize_act(x_all[i:i + 1], q[:1], d[:1], b[:1])
        tq.tq_gemv_mx(mats[i % copies], q[:1], d[:1], y[:1])

    def stepf(i):
        tq.tq_quantize_act(x_all[i:i + 1], q[:1], d[:1], b[:1])
        tq.tq_gemv(matsf[i % copies], q[:1], d[:1], b[:1], y[:1])

    elapsed, reps = time_graph(step, W, K)
    elapsed_f, _ = time_graph(stepf, W, K)
    io = k * 4 + n * 4
    gbs = (mx_bytes(n, k) + io) * K / elapsed / 1e9
    gbs_f = (matrix_bytes(n, k) + io) * K / elapsed_f / 1e9

    def kernel_ms(fn, t):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(P)]
        torch.cuda.synchronize()
        torch.cuda._sleep(int(2.4e9 * 0.02))
        for j in range(P):
            tq.tq_quantize_act(x_all[j:j + t], q[:t], d[:t], b[:t])
            fn(j, t, ev[j])
        torch.cuda.synchronize()
        return float(np.mean([s.elapsed_time(e) for s, e in ev]))

    def km(j, t, ev):
        tq.tq_gemv_mx_timed(mats[j % copies], q[:t], d[:t], y[:t], ev)

    def kf(j, t, ev):
        tq.tq_gemv_timed(matsf[j % copies], q[:t], d[:t], b[:t], y[:t], ev)

    by_tokens = {}
    for t in (1, 4, 16):
        m1, mf = kernel_ms(km, t), kernel_ms(kf, t)
        by_tokens[str(t)] = {"mxfp4_ms": round(m1, 5), "folded_ms": round(mf, 5),
                             "mxfp4_GBps": round((mx_bytes(n, k) + t * (k + kb * 4 + n * 4)) / (m1 * 1e-3) / 1e9, 1),
                             "folded_GBps": round((matrix_bytes(n, k) + t * (k + kb * 4 + n * 4)) / (mf * 1e-3) / 1e9, 1)}
    ms = by_tokens["1"]["mxfp4_ms"]
    roof = hbm_roof("gemv_mx", mx_bytes(n, k) + k + kb * 4 + n * 4, ms, "k_gemv_mx<2, 1, 2, false>")
    return dict(value=gbs, K=K, W=W, elapsed=elapsed, reps=reps, tokens=K, roof=roof,
                config={"workload": cfg["name"], "n": n, "k": k, "tokens_per_step": 1, "bits_per_weight": 4.25,
                        "rotating_copies": copies, "format": "MXFP4 (e2m1 codes, e8m0 scale per 32), doubled-e2m1 "
                                                             "integer dot"},
                extra={"folded_same_shape": {"value": round(gbs_f, 2), "ms_per_step": round(elapsed_f * 1e3 / K, 5),
                                             "bits_per_weight": 4.0625},
                       "kernel_ms_by_tokens": by_tokens})


PCIE5_X16_GBS = 63.0  # PCIe 5.0 x16, one direction: 32 GT/s x 16 lanes x 128/130


def run_stream(args, wl, cfg):
    """The batch-1 decode layer with its experts streamed: all 256 experts in pinned host
    memory as contiguous records, an LRU pool of expert slots in HBM; per step the host
    maps the routing to slots, the misses are copied host-to-device, and the same MoE
    kernels run on the pool. Steps run eagerly (the host plans each step)."""
    import torch
    from paper_2608_08910_amd import tq
    from synth import gen

    E, H, I, T, topk, seed = cfg["experts"], cfg["hidden"], cfg["inter"], cfg["tokens"], cfg["topk"], gen.SEED
    K = args.steps if args.steps is not None else wl["steps"]
    W = args.warmup if args.warmup is not None else wl["warmup"]
    S = args.slots
    total = W + K
    rb = tq.tq_expert_record_bytes(H, I)
    store = tq.TqExpertRecords.empty(E, H, I, device="cpu", pin_memory=True)
    # the host store: every expert generated on the device, rewritten as a record, copied out
    tmp = tq.TqExperts.empty(1, H, I)
    rec = tq.TqExpertRecords.empty(1, H, I)
    d0 = tq.tq_experts_from_records(1 << 20, 1, H, I)
    code_offs = [d0.gate_codes - (1 << 20), d0.up_codes - (1 << 20), d0.down_codes - (1 << 20)]
    scale_offs = [d0.gate_scales - (1 << 20), d0.up_scales - (1 << 20), d0.down_scales - (1 << 20)]
    for e in range(E):
        for p in range(3):
            tq.tq_synth_weights(gen.matrix_key(seed, 0, e, p), tmp.matrix(0, p))
            c = tmp.codes[p].reshape(-1)
            sc = tmp.scales[p].reshape(-1).view(torch.uint8)
            rec.data[0, code_offs[p]:code_offs[p] + c.numel()] = c
            rec.data[0, scale_offs[p]:scale_offs[p] + sc.numel()] = sc
        store.data[e].copy_(rec.data[0])
    torch.cuda.synchronize()
    pool = tq.TqExpertRecords.empty(S, H, I)
    cache = tq.TqCache(E, S)
    sched = gen.bench_routing_schedule(seed, total, T, E, topk, cfg["routing"])
    x_all = torch.from_numpy(gen.activations(seed, 1000, total * T, H).reshape(total, T, H)).cuda()
    w_all = torch.from_numpy(np.stack([s_[1] for s_ in sched])).cuda()
    slots_host = [torch.empty((T, topk), dtype=torch.int32, pin_memory=True) for _ in range(total)]
    slots_dev = [torch.empty((T, topk), dtype=torch.int32, device="cuda") for _ in range(total)]
    out = torch.empty((T, H), dtype=torch.float32, device="cuda")
    ws = tq.moe_workspace(pool, T, topk)
    misses_per_step = []

    def step(i):
        _, misses = cache.map(sched[i][0], slots_host[i].numpy())
        misses_per_step.append(len(misses))
        cache.fetch(store, pool, misses, slots_host[i], slots_dev[i])
        tq.tq_moe_grouped(pool, x_all[i], slots_dev[i], w_all[i], out, ws)

    for i in range(W):
        step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(W, W + K):
        step(i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    copied = sum(misses_per_step[W:]) * rb
    bytes_expert = 2 * matrix_bytes(I, H) + matrix_bytes(H, I)
    distinct = [len(np.unique(sched[i][0])) for i in range(W, W + K)]
    alg_bytes = sum(d_ * bytes_expert for d_ in distinct) + K * (T * H * 4 * 2 + T * topk * 8)
    link = copied / elapsed / 1e9
    roof = {"kernel": "host_to_device_copies", "bound": "pcie", "achieved": round(link, 2), "peak": PCIE5_X16_GBS,
            "unit": "GB/s", "frac": round(link / PCIE5_X16_GBS, 4), "traffic": None,
            "bytes_per_step": round(copied / K), "note": "expert records copied per step over the host link "
                                                        "(pinned host -> HBM); peak = PCIe 5.0 x16 one direction"}
    return dict(value=alg_bytes / elapsed / 1e9, K=K, W=W, elapsed=elapsed, reps=None, tokens=K * T, roof=roof,
                config={"workload": cfg["name"] + f"_streamed_{S}slots", "experts": E, "hidden": H, "inter": I,
                        "tokens_per_step": T, "topk": topk, "routing": "uniform top-8, no expert reused within 3 steps",
                        "bits_per_weight": 4.0625, "host_store_bytes": E * rb, "hbm_slots": S,
                        "hbm_pool_bytes": S * rb, "path": "single_token (eager steps)"},
                extra={"misses_per_step": round(float(np.mean(misses_per_step[W:])), 3),
                       "hit_rate": round(1.0 - sum(misses_per_step[W:]) / max(1, sum(distinct)), 4),
                       "copied_GBps": round(link, 2)})


def mixed_kernel(nmat: int, kb: int) -> str:
    """The mixed path's one-launch kernel for a projection of kb blocks per row (NL rounded
    up to 1, 2, 4 or 8; the VALU role's tile as the grouped VALU kernel's)."""
    nl = (kb + 7) // 8
    nl4 = nl if nl <= 2 else (4 if nl <= 4 else 8)
    if nmat == 2:
        rpw = 8 if nl4 == 1 else (4 if nl4 == 2 else (2 if nl4 <= 4 else 1))
    else:
        rpw = 8 if nl4 <= 2 else (4 if nl4 <= 4 else 2)
    nt = 2 if nl4 <= 2 else 1
    return f"k_mixed<{nmat}, {nl4}, {rpw}, {nt}, {nt}, {'true' if kb != 8 * nl4 else 'false'}>"


def run_moe(args, wl, cfg):
    import torch
    from paper_2608_08910_amd import tq
    from synth import gen

    E, H, I, T, topk, seed = cfg["experts"], cfg["hidden"], cfg["inter"], cfg["tokens"], cfg["topk"], gen.SEED
    L = cfg.get("layers", 1)
    K = args.steps if args.steps is not None else wl["steps"]
    W = args.warmup if args.warmup is not None else wl["warmup"]
    P = args.profile_steps if args.profile_steps is not None else wl["profile"]
    total = W + K

    # resident experts, generated on the device (one set per layer)
    layers = []
    for l in range(L):
        ex = tq.TqExperts.empty(E, H, I)
        for e in range(E):
            for p in range(3):
                tq.tq_synth_weights(gen.matrix_key(seed, l, e, p), ex.matrix(e, p))
        layers.append(ex)
    torch.cuda.synchronize()

    if T == 1:
        # every step avoids the experts of the previous 3 steps (last-level-cache reuse),
        # and the last timed steps those of the first ones (the timed graph is replayed)
        sched = [gen.bench_routing_schedule(seed, total, T, E, topk, cfg["routing"], wrap_from=W)]
    else:
        # many tokens per step: a step's expert union is 0.9-3.3 GB per layer, far beyond the cache
        sched = [[gen.routing(seed, 1000 + 97 * l + i, T, E, topk, cfg["routing"]) for i in range(total)]
                 for l in range(L)]
    idx_all = [torch.from_numpy(np.stack([s[0] for s in sl])).cuda() for sl in sched]  # [layer][step][T][topk]
    w_all = [torch.from_numpy(np.stack([s[1] for s in sl])).cuda() for sl in sched]
    x_all = []
    for l in range(L):
        xs = gen.activations(seed, 1000 + l, total * T, H).reshape(total, T, H)
        if cfg.get("token_factor"):
            xs = xs * np.stack([gen.token_factors(seed + 1 + i, T) for i in range(total)])[:, :, None]
        x_all.append(torch.from_numpy(np.ascontiguousarray(xs, dtype=np.float32)).cuda())
    out = torch.empty((T, H), dtype=torch.float32, device="cuda")
    ws = tq.moe_workspace(layers[0], T, topk)

    def step(i):
        for l in range(L):
            tq.tq_moe_grouped(layers[l], x_all[l][i], idx_all[l][i], w_all[l][i], out, ws, args.flags)

    elapsed, reps = time_graph(step, W, K)
    bytes_expert = 2 * matrix_bytes(I, H) + matrix_bytes(H, I)
    distinct = [len(np.unique(sched[l][i][0])) for l in range(L) for i in range(W, W + K)]
    alg_bytes = sum(d * bytes_expert for d in distinct) + K * L * (T * H * 4 * 2 + T * topk * 8)
    gbs = alg_bytes / elapsed / 1e9

    # per-kernel pass: every stage's kernel launched with its own start/stop events,
    # eager launches queued behind a spin kernel so the GPU runs them back to back
    nst = tq.tq_moe_stage_count()
    names = [tq.tq_moe_stage_name(i) for i in range(nst)]
    runs = [(W + (j % K), l) for j in range(P) for l in range(L)]
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2 * nst)] for _ in runs]
    torch.cuda.synchronize()
    torch.cuda._sleep(int(2.4e9 * 0.05))  # ~50 ms of queue head-room
    # about 30 ms of the same steps untimed first: the first launches after the idle spin
    # run up to a third slower than back-to-back work, so the timed ones follow warm work
    # as the graph's replays do
    for j in range(max(1, int(0.03 / (elapsed / K)))):
        for l in range(L):
            i = W + (j % K)
            tq.tq_moe_grouped(layers[l], x_all[l][i], idx_all[l][i], w_all[l][i], out, ws, args.flags)
    for (i, l), ev in zip(runs, evs):
        tq.tq_moe_grouped_timed(layers[l], x_all[l][i], idx_all[l][i], w_all[l][i], out, ws, ev, args.flags)
    torch.cuda.synchronize()
    path = tq.tq_moe_path(layers[0], T, topk, args.flags)
    # stages with no kernel on the path taken (their event pairs are recorded back to
    # back) are reported as null: the single-token path runs gate_up and down only
    kernel_stages = {"gate_up", "down"} if path == tq.TQ_MOE_PATH_T1 else set(names)
    stage_ms = {n: (float(np.mean([ev[2 * si].elapsed_time(ev[2 * si + 1]) for ev in evs])) if n in kernel_stages
                    else None) for si, n in enumerate(names)}
    gu_ms = stage_ms["gate_up"]
    n_distinct = float(np.mean([len(np.unique(sched[l][i][0])) for i, l in runs]))
    mfma = path == tq.TQ_MOE_PATH_MFMA
    nl_gu, nl_dn = (H // 256 + 7) // 8, (I // 256 + 7) // 8
    ragged = "true" if (H // 256) % 8 else "false"
    if path == tq.TQ_MOE_PATH_T1:
        # the single-token gate/up kernel moves the routed experts' gate and up codes +
        # scales, reads x (fp32) and writes h (fp32, one row per slot)
        gu_bytes = n_distinct * 2 * matrix_bytes(I, H) + T * H * 4 + T * topk * I * 4
        gu_kernel = f"k_t1_gateup<{nl_gu}, {4 if nl_gu <= 2 else (2 if nl_gu <= 4 else 1)}, 4, {ragged}>"
        kname = "gate_up"
    else:
        # the grouped gate/up kernels read the routed experts' gate and up planes and the
        # quantized tokens (int8 + scale per block), and write h per slot
        gu_bytes = n_distinct * 2 * matrix_bytes(I, H) + T * (H + (H // 256) * 4) + T * topk * I * 4
        rpw = 8 if nl_gu == 1 else (4 if nl_gu == 2 else (2 if nl_gu <= 4 else 1))
        nt = 2 if nl_gu <= 2 else 1  # tokens per group of the grouped VALU kernel (first, later)
        # the MFMA stage is two launches: 128-token tiles, then the experts of at most 32 slots
        gu_kernel = ("k_moe_mfma<2, 128, 8, false, false, false, false> + k_moe_mfma<2, 32, 4, true, false, false, false>" if mfma
                     else f"k_tb<2, {nl_gu}, {rpw}, {nt}, {nt}, 4, {ragged}>")
        if path == tq.TQ_MOE_PATH_MIXED:  # one launch: the VALU tasks and the 32-token MFMA tiles
            gu_kernel = mixed_kernel(2, H // 256)
        kname = "gate_up"
    if mfma:
        gu_ops = 2.0 * T * topk * (2 * I * H)  # int8 multiply-adds of gate and up, 2 ops each
        achieved = gu_ops / (gu_ms * 1e-3) / 1e12
        roof = {"kernel": kname, "bound": "mfma", "achieved": round(achieved, 1), "peak": MFMA_I8_PEAK_TOPS,
                "unit": "TOP/s", "frac": round(achieved / MFMA_I8_PEAK_TOPS, 4), "traffic": recorded_traffic(gu_kernel),
                "ops_per_launch": gu_ops, "bytes_per_launch": round(gu_bytes), "mean_ms": round(gu_ms, 5),
                "hbm_GBps": round(gu_bytes / (gu_ms * 1e-3) / 1e9, 1), "kernel_symbol": gu_kernel,
                "frac_timing": "hip events recorded on the stream before the fork and after the join of the "
                               "stage's two launches, which run side by side on two streams (the span of both, "
                               "event commands included); mean over the per-kernel pass"}
        avg_ns = _recorded(gu_kernel, "average_ns", kind="kernel_stats")
        if avg_ns is not None:
            roof["rocprof_mean_ms"] = round(avg_ns * 1e-6, 5)
            roof["frac_rocprof"] = round(gu_ops / (avg_ns * 1e-9) / 1e12 / MFMA_I8_PEAK_TOPS, 4)
    else:
        roof = hbm_roof(kname, gu_bytes, gu_ms, gu_kernel)
    # the down kernel beside it: the routed experts' down planes, h in (fp32 per slot on the
    # single-token path, which requantizes it itself; int8 + scale per block otherwise),
    # the output (or the per-slot rows) out
    if path == tq.TQ_MOE_PATH_T1:
        dn_bytes = n_distinct * matrix_bytes(H, I) + T * topk * I * 4 + T * H * 4
        nl4 = nl_dn if nl_dn <= 2 else (4 if nl_dn <= 4 else 8)
        r = (16 // nl4) * min(topk, 4) // 4
        rows = 1 if r < 1 else 1 << (r.bit_length() - 1)
        dn_kernel = f"k_t1_down<{nl4}, {rows}, {topk}, {'true' if (I // 256) % 8 or nl4 * 8 != I // 256 else 'false'}>"
    else:
        dn_bytes = n_distinct * matrix_bytes(H, I) + T * topk * (I + (I // 256) * 4) + T * topk * H * 4
        # (down: two 16-row tiles per wave, run as the kernel's two-matrix path)
        dn_kernel = ("k_moe_mfma<2, 128, 8, false, false, true, false> + k_moe_mfma<2, 32, 4, true, false, true, false>" if mfma
                     else "k_tb<1, ...>")
        if path == tq.TQ_MOE_PATH_MIXED:
            dn_kernel = mixed_kernel(1, I // 256)
    dn_ms = stage_ms["down"]
    down = {
        "kernel_symbol": dn_kernel, "bytes_per_launch": round(dn_bytes), "mean_ms": round(dn_ms, 5),
        "GBps": round(dn_bytes / (dn_ms * 1e-3) / 1e9, 1),
        "frac_of_hbm_peak": round(dn_bytes / (dn_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    # second ceiling: a plain streaming read of the step's bytes (per layer) and of the
    # dominant kernel's, measured here
    step_bytes = alg_bytes / (K * L)
    ceil_step = stream_ceiling(step_bytes, 32 if step_bytes < 4e8 else 6)
    ceil_gu = stream_ceiling(gu_bytes, 32 if gu_bytes < 4e8 else 6)
    layer_ms = elapsed * 1e3 / (K * L)
    ceiling = {"step_bytes": ceil_step["bytes"], "stream_read_GBps": ceil_step["GBps"],
               "stream_read_ms": ceil_step["ms"], "layer_GBps": round(step_bytes / (layer_ms * 1e-3) / 1e9, 1),
               "layer_frac_of_stream_read": round(ceil_step["ms"] / layer_ms, 4),
               "dominant_kernel_bytes": ceil_gu["bytes"], "dominant_stream_read_GBps": ceil_gu["GBps"],
               "dominant_kernel_frac_of_stream_read": round(ceil_gu["ms"] / gu_ms, 4)}
    routing_desc = ("uniform top-8, no expert reused within 3 steps" if T == 1 else
                    f"{cfg['routing']} top-{topk}, fresh draw per step")
    config = {"workload": cfg["name"], "layers": L, "experts": E, "hidden": H, "inter": I, "tokens_per_step": T,
              "topk": topk, "routing": routing_desc, "bits_per_weight": 4.0625,
              "resident_expert_bytes": L * E * bytes_expert,
              "path": {0: "single_token", 1: "valu", 2: "mfma", 3: "mixed_valu_mfma"}[path]}
    extra = {"stage_ms": {k: (None if v is None else round(v, 5)) for k, v in stage_ms.items()},
             "down_kernel": down, "stream_ceiling": ceiling,
             "bytes_per_token": round(alg_bytes / (K * T)),
             "mean_distinct_experts_per_layer": round(float(np.mean(distinct)), 2)}
    if T > 1:
        # the routing actually timed: per-expert slot counts of each timed step and layer
        counts = [np.bincount(sched[l][i][0].ravel(), minlength=E) for l in range(L) for i in range(W, W + K)]
        first = np.sort(counts[0])[::-1]
        vals, nexp = np.unique(counts[0][counts[0] > 0], return_counts=True)
        extra["routing_histogram"] = {
            "steps_x_layers": len(counts),
            "active_experts_mean": round(float(np.mean([(c > 0).sum() for c in counts])), 2),
            "max_slots_per_expert_mean": round(float(np.mean([c.max() for c in counts])), 2),
            "first_timed_step_top16_counts": first[:16].tolist(),
            "first_timed_step_experts_by_count": {int(v): int(n) for v, n in zip(vals, nexp)}}
    return dict(value=gbs, K=K, W=W, elapsed=elapsed, reps=reps, tokens=K * T, roof=roof, config=config, extra=extra)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--workload", choices=sorted(WORKLOADS), default="decode1")
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-steps", type=int, default=None, help="steps of the per-kernel event pass")
    ap.add_argument("--flags", type=int, default=0, help="tq_moe_grouped flags (1 force VALU, 2 force MFMA)")
    ap.add_argument("--slots", type=int, default=64, help="HBM expert slots of the stream workload")
    ap.add_argument("--no-graph", action="store_true",
                    help="launch the steps eagerly instead of in HIP graphs, and skip the replay band (for "
                         "profiler counter passes, which only need the kernels' dispatches)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy (to scale HBM byte counters)")
    args = ap.parse_args()
    global USE_GRAPH
    USE_GRAPH = not args.no_graph
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
    from synth import gen

    torch.cuda.set_device(0)
    wl = WORKLOADS[args.workload]
    cfg = {"quant": gen.QUANT_CONFIG, "twoplane": gen.TWO_PLANE_CONFIG,
           "mxfp4": gen.MXFP4_CONFIG}.get(wl["cfg"]) or gen.CONFIGS[wl["cfg"]]
    run = {"gemv": run_gemv, "moe": run_moe, "quant": run_quant, "twoplane": run_twoplane,
           "mxfp4": run_mxfp4}[cfg["kind"]]
    if wl.get("stream"):
        run = run_stream
    r = run(args, wl, cfg)
    K, W, elapsed = r["K"], r["W"], r["elapsed"]
    res = {
        "metric": METRIC,
        "value": round(r["value"], 2),
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
        "config": r["config"],
        "pct_of_hbm_peak": round(100 * r["value"] / HBM_PEAK_GBS, 2),
        "tokens_per_s": round(r["tokens"] / elapsed, 1),
        **r["extra"],
        "roofline": r["roof"],
    }
    if not USE_GRAPH:
        res["timing_note"] = "eager launches (--no-graph): not the graph-timed figure"
    if r.get("reps"):
        per_step = np.array(r["reps"]) * 1e3 / K
        vals = r["value"] * (elapsed / np.array(r["reps"]))
        res["band"] = {"replays": len(per_step), "of": f"the {K}-step timed graph, each replay bracketed by HIP events",
                       "ms_per_step": {"median": round(float(np.median(per_step)), 5),
                                       "min": round(float(per_step.min()), 5), "max": round(float(per_step.max()), 5)},
                       "value": {"median": round(float(np.median(vals)), 2), "min": round(float(vals.min()), 2),
                                 "max": round(float(vals.max()), 2)}}
    if not args.no_cpu_baseline and args.workload == "decode1":
        res["cpu_baseline"] = cpu_baseline(gen.SEED, cfg["hidden"], cfg["inter"], cfg["topk"])
    if not args.no_cpu_baseline and args.workload == "tiedquant":
        res["cpu_baseline"] = cpu_baseline_quant(cfg)
    if not args.no_cpu_baseline and args.workload == "twoplane":
        res["cpu_baseline"] = cpu_baseline_twoplane(cfg)
    if not args.no_cpu_baseline and args.workload == "mxfp4":
        res["cpu_baseline"] = cpu_baseline_mx(cfg)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
