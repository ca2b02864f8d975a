"""Helpers for the GPU parity tests (HIP path through the C-ABI vs the CPU oracle)."""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

from synth import gen


def device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def announce(msg: str):
    """Name the case before a GPU step (flushed, so a crash still shows it)."""
    print(f"[gpu-case] {msg}", file=sys.stderr, flush=True)


def assert_close(got, ref, absref, rtol=1e-5, what="value"):
    """|got - ref| <= rtol * absref elementwise, where absref is the sum of the absolute
    terms of the reference sum (a relative bound that survives cancellation)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    absref = np.asarray(absref, dtype=np.float64)
    err = np.abs(got - ref)
    bound = rtol * absref
    bad = err > bound
    if bad.any():
        i = np.unravel_index(np.argmax(err / np.maximum(absref, 1e-300)), err.shape)
        raise AssertionError(f"{what}: {int(bad.sum())}/{bad.size} elements exceed {rtol} * absref; worst at {i}: "
                             f"got {got[i]!r} ref {ref[i]!r} absref {absref[i]!r}")
    return float((err / np.maximum(absref, 1e-300)).max()) if err.size else 0.0


def synth_experts(tq, seed: int, layer: int, E: int, H: int, I: int):
    ex = tq.TqExperts.empty(E, H, I)
    for e in range(E):
        for p in range(3):
            tq.tq_synth_weights(gen.matrix_key(seed, layer, e, p), ex.matrix(e, p))
    return ex


def host_experts(tq, oracle, E: int, H: int, I: int, seed: int):
    """Small experts from host trit planes: packed by the library on the host, and the
    oracle's logical codes from the oracle's own fold of the same planes."""
    rng = np.random.default_rng(seed)
    ex = tq.TqExperts.empty(E, H, I)
    logical = {}
    for e in range(E):
        logical[e] = {}
        for p, name in enumerate(("gate", "up", "down")):
            n, k = ex.shape(p)
            t1 = rng.integers(-1, 2, (n, k)).astype(np.int8)
            t2 = rng.integers(-1, 2, (n, k)).astype(np.int8)
            s = np.asarray(np.exp(rng.uniform(np.log(1e-3), np.log(1e-1), (n, k // 256))), dtype=np.float16).view(np.uint16)
            ex.codes[p][e].copy_(torch.from_numpy(tq.tq_fold_pack_host(t1, t2)))
            ex.scales[p][e].copy_(torch.from_numpy(s.view(np.int16)))
            logical[e][name] = (oracle.fold(t1, t2), s)
    return ex, logical


def ws_views(tq, ex, ws: torch.Tensor, t: int, topk: int) -> dict:
    """Typed views of the stage buffers the MoE call leaves in its workspace."""
    lay = tq.tq_moe_workspace_layout(ex, t, topk)
    S, H, I = t * topk, ex.hidden, ex.inter

    def view(name, dtype, shape):
        n = int(np.prod(shape)) * torch.tensor([], dtype=dtype).element_size()
        return ws[lay[name]:lay[name] + n].view(dtype).reshape(shape)

    return dict(xq=view("xq", torch.int8, (t, H)), xd=view("xd", torch.float32, (t, H // 256)),
                xb=view("xb", torch.int32, (t, H // 256)), h=view("h", torch.float32, (S, I)),
                hq=view("hq", torch.int8, (S, I)), hd=view("hd", torch.float32, (S, I // 256)),
                hb=view("hb", torch.int32, (S, I // 256)), yd=view("yd", torch.float32, (S, H)),
                flags=view("flags", torch.int32, (1,)))
