"""The grouped MFMA path runs each projection as two launches that write disjoint outputs,
the second on a stream the library owns (one per device), forked from the caller's
stream and joined back to it by events. Its results must not depend on how the calls
are issued: eagerly, captured in a graph before the side stream exists (the process's
first MFMA call made under capture runs both launches on the caller's stream), captured
after it (the fork and join become graph edges), or from two host threads at once, each
on its own stream (they share the side stream and its two events)."""
import os
import subprocess
import sys
import threading

import numpy as np
import pytest
import torch

from gpu_util import announce, device, synth_experts
from synth import gen

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# Zipf routing over 16 experts at 256 tokens x top-4: the hottest experts take several
# 128-token tiles (the first launch), the coldest at most 32 slots (the second).
E, H, I, T, TOPK = 16, 1024, 512, 256, 4


@pytest.fixture(scope="module")
def tq():
    device()
    from paper_2608_08910_amd import tq as _tq
    return _tq


def make_inputs(seed: int, n: int):
    xs, idx, w = [], [], []
    for i in range(n):
        xs.append(torch.from_numpy(gen.activations(seed, i, T, H)).cuda())
        ii, ww = gen.routing(seed, i, T, E, TOPK, "zipf")
        idx.append(torch.from_numpy(ii).cuda())
        w.append(torch.from_numpy(ww).cuda())
    return xs, idx, w


def both_launches_busy(idx) -> bool:
    counts = np.bincount(idx.cpu().numpy().ravel(), minlength=E)
    return counts.max() > 128 and 0 < counts[counts > 0].min() <= 32


CHILD = r"""
import sys
sys.path.insert(0, sys.argv[1]); sys.path.insert(0, sys.argv[1] + "/tests")
import torch
from paper_2608_08910_amd import tq
from gpu_util import synth_experts
from test_gpu_moe_streams import E, H, I, T, TOPK, make_inputs
F = tq.TQ_MOE_FORCE_MFMA
ex = synth_experts(tq, 31, 0, E, H, I)
xs, idx, w = make_inputs(32, 3)
torch.cuda.synchronize()

def capture(ws, outs):
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for i in range(3):
                tq.tq_moe_grouped(ex, xs[i], idx[i], w[i], outs[i], ws, flags=F, stream=s)
    torch.cuda.synchronize()
    return g

def check(outs, ref, what):
    for i in range(3):
        assert torch.equal(outs[i], ref[i]), f"{what}: call {i} differs from the eager call"

# the process's first MFMA calls, made under capture
ws_g = tq.moe_workspace(ex, T, TOPK)
outs = [torch.full((T, H), float("nan"), device="cuda") for _ in range(3)]
g1 = capture(ws_g, outs)
print("captured before the side stream exists", flush=True)
g1.replay()
torch.cuda.synchronize()
# eager calls: the first one creates the side stream
ws_e = tq.moe_workspace(ex, T, TOPK)
ref = [torch.empty((T, H), device="cuda") for _ in range(3)]
for i in range(3):
    tq.tq_moe_grouped(ex, xs[i], idx[i], w[i], ref[i], ws_e, flags=F)
torch.cuda.synchronize()
assert all(torch.isfinite(r).all() for r in ref)
check(outs, ref, "graph captured before the side stream")
# captured again: now forked to the side stream and joined back
outs2 = [torch.full((T, H), float("nan"), device="cuda") for _ in range(3)]
g2 = capture(ws_g, outs2)
for rep in range(3):
    for o in outs2:
        o.fill_(float("nan"))
    g2.replay()
    torch.cuda.synchronize()
    check(outs2, ref, f"graph with the fork and join, replay {rep}")
    g1.replay()  # the first graph still replays alongside
    torch.cuda.synchronize()
    check(outs, ref, f"first graph, replay {rep}")
print("OK", flush=True)
"""


def test_first_mfma_call_under_capture_then_forked(tq):
    """A fresh process whose first MFMA calls are captured (both launches on the capture
    stream), then eager calls (the side stream is created), then a second capture with
    the fork and join: every replay of both graphs equals the eager outputs bitwise."""
    device()
    xs, idx, w = make_inputs(32, 3)
    assert all(both_launches_busy(i) for i in idx)
    announce("moe side stream: first MFMA call under capture (child process)")
    r = subprocess.run([sys.executable, "-u", "-c", CHILD, ROOT], capture_output=True, text=True, timeout=240)
    assert r.returncode == 0 and r.stdout.strip().endswith("OK"), (r.stdout[-2000:], r.stderr[-3000:])


def test_two_host_threads_own_streams(tq):
    """Two host threads, each calling the MFMA path repeatedly on its own stream with its
    own workspace and inputs while the other does: every output equals the same call made
    alone, bitwise."""
    device()
    ex = synth_experts(tq, 41, 0, E, H, I)
    n = 3
    data = [make_inputs(42 + k, n) for k in range(2)]
    F = tq.TQ_MOE_FORCE_MFMA
    assert tq.tq_moe_path(ex, T, TOPK, F) == tq.TQ_MOE_PATH_MFMA
    ws0 = tq.moe_workspace(ex, T, TOPK)
    ref = []
    for k in range(2):
        xs, idx, w = data[k]
        ref.append([torch.empty((T, H), device="cuda") for _ in range(n)])
        for i in range(n):
            tq.tq_moe_grouped(ex, xs[i], idx[i], w[i], ref[k][i], ws0, flags=F)
    torch.cuda.synchronize()
    announce("moe side stream: two host threads, own streams")
    results, errors = {}, []

    def run(k):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                ws = tq.moe_workspace(ex, T, TOPK)
                outs = [torch.full((T, H), float("nan"), device="cuda") for _ in range(n)]
                xs, idx, w = data[k]
                for _ in range(4):
                    for i in range(n):
                        tq.tq_moe_grouped(ex, xs[i], idx[i], w[i], outs[i], ws, flags=F, stream=s)
            s.synchronize()
            results[k] = outs
        except Exception as exc:  # reported below, on the main thread
            errors.append(exc)

    threads = [threading.Thread(target=run, args=(k,)) for k in range(2)]
    for th in threads:
        th.start()
    for th in threads:
        th.join(timeout=120)
    assert not errors, errors
    assert set(results) == {0, 1}
    for k in range(2):
        for i in range(n):
            assert torch.equal(results[k][i], ref[k][i]), f"thread {k} call {i}"
