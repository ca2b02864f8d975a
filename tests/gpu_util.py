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
    """Typed views of the stage buffers the MoE call leaves in its workspace (and of the
    debug dump, when the workspace has room for it)."""
    lay = tq.tq_moe_workspace_layout(ex, t, topk)
    S, H, I, E = t * topk, ex.hidden, ex.inter, ex.n_experts

    def view(name, dtype, shape):
        n = int(np.prod(shape)) * torch.tensor([], dtype=dtype).element_size()
        return ws[lay[name]:lay[name] + n].view(dtype).reshape(shape)

    v = dict(xq=view("xq", torch.int8, (t, H)), xd=view("xd", torch.float32, (t, H // 256)),
             xb=view("xb", torch.int32, (t, H // 256)), h=view("h", torch.float32, (S, I)),
             hq=view("hq", torch.int8, (S, I)), hd=view("hd", torch.float32, (S, I // 256)),
             hb=view("hb", torch.int32, (S, I // 256)), yd=view("yd", torch.float32, (S, H)),
             flags=view("flags", torch.int32, (1,)), n_active=view("n_active", torch.int32, (1,)),
             active=view("active", torch.int32, (E,)), act_off=view("act_off", torch.int32, (E + 1,)),
             slot_list=view("slot_list", torch.int32, (S,)))
    if ws.numel() >= lay["total_debug"]:
        v.update(g=view("g", torch.float32, (S, I)), u=view("u", torch.float32, (S, I)),
                 gsum=view("gsum", torch.int32, (S, I, H // 256)), usum=view("usum", torch.int32, (S, I, H // 256)),
                 dsum=view("dsum", torch.int32, (S, H, I // 256)))
    return v


def run_moe(tq, ex, x, idx, w, flags=0, debug=True):
    """One tq_moe_grouped call on host inputs; with debug (the default for parity tests)
    the workspace holds the debug dump and the call takes TQ_MOE_DEBUG_STAGES."""
    t, topk = idx.shape
    xd = torch.from_numpy(np.ascontiguousarray(x)).cuda()
    idd = torch.from_numpy(np.ascontiguousarray(idx)).cuda()
    wd = torch.from_numpy(np.ascontiguousarray(w)).cuda()
    out = torch.empty((t, ex.hidden), dtype=torch.float32, device="cuda")
    ws = tq.moe_workspace(ex, t, topk, debug=debug)
    tq.tq_moe_grouped(ex, xd, idd, wd, out, ws, flags | (tq.TQ_MOE_DEBUG_STAGES if debug else 0))
    torch.cuda.synchronize()
    return out, ws


def _rows(t: torch.Tensor, ix) -> np.ndarray:
    """Rows ix of a device tensor, gathered on the device, as a host array."""
    return t[torch.as_tensor(np.asarray(ix, dtype=np.int64), device=t.device)].cpu().numpy()


def check_slots(tq, o, ex, get_expert, x, idx, ws, slots, V=None, n_ids=None):
    """Staged parity of the listed slots (s = token * topk + j) of one tq_moe_grouped call,
    each GPU stage against the oracle applied to the GPU's previous stage:
      gsum, usum == the oracle's gate/up block sums on xq            (bit-exact, debug dump)
      g, u       ~= oracle (1e-5 of the absolute terms)               (debug dump)
      h          ~= oracle SiLU(g) * u                                (bound from 1e-5 on g, u)
      hq, hd, hb == oracle.quantize(GPU h)                           (bit-exact)
      dsum       == the oracle's down block sums on GPU hq          (bit-exact, debug dump)
      yd         ~= oracle dot pass of W_down on GPU (hq, hd)        (1e-5 of abs terms)
    (xq itself is checked by check_moe.) Slots whose expert id is outside [0, n_ids)
    (default: the experts of `ex`) are skipped; idx holds the ids get_expert takes (for a
    streamed step, the expert ids, while the call ran on their slots). Returns ({slot: (oracle yd, its absolute terms, GPU yd)}, {slot: requantized codes that
    differ from the oracle's own}, codes compared)."""
    t, topk = idx.shape
    E = n_ids or ex.n_experts
    V = V or ws_views(tq, ex, ws, t, topk)
    dbg = "gsum" in V
    slots = [int(s) for s in slots if 0 <= idx[s // topk, s % topk] < E]
    G = {n: _rows(V[n], slots) for n in ("h", "hq", "hd", "hb", "yd")}
    if dbg:
        G.update({n: _rows(V[n], slots) for n in ("g", "u", "gsum", "usum", "dsum")})
    by_expert: dict[int, list] = {}
    for r, s in enumerate(slots):
        by_expert.setdefault(int(idx[s // topk, s % topk]), []).append((r, s))
    ref_yd, flips, codes = {}, {}, 0
    for e in sorted(by_expert):
        ee = get_expert(e)
        for r, s in by_expert[e]:
            st = o.expert_slot(ee, x[s // topk], want_isum=dbg)
            if dbg:
                assert np.array_equal(G["gsum"][r], st["g_isum"]), f"gate block sums slot {s}"
                assert np.array_equal(G["usum"][r], st["u_isum"]), f"up block sums slot {s}"
                assert_close(G["g"][r], st["g"], st["g_abs"] + 1e-30, what=f"g slot {s}")
                assert_close(G["u"][r], st["u"], st["u_abs"] + 1e-30, what=f"u slot {s}")
            g, u, ga, ua = st["g"], st["u"], st["g_abs"], st["u_abs"]
            tol_h = 1e-5 * (1.1 * ga * np.abs(u) + np.abs(o.silu(g)) * ua) + 2e-6 * np.abs(st["h"]) + 1e-30
            err = np.abs(G["h"][r].astype(np.float64) - st["h"])
            assert (err <= tol_h).all(), f"h slot {s}: worst {(err / tol_h).max()}"
            hq, hd, hb = o.quantize(G["h"][r])
            assert np.array_equal(G["hq"][r], hq[0]), f"hq slot {s}"
            assert np.array_equal(G["hd"][r].view(np.uint32), hd[0].view(np.uint32)), f"hd slot {s}"
            assert np.array_equal(G["hb"][r], hb[0]), f"hb slot {s}"
            yr, ya, yi = o.gemv(*ee["down"], G["hq"][r], G["hd"][r], want_isum=True)
            if dbg:
                assert np.array_equal(G["dsum"][r], yi[0]), f"down block sums slot {s}"
            assert_close(G["yd"][r], yr[0], ya[0] + 1e-30, what=f"yd slot {s}")
            diff = int((G["hq"][r] != st["qh"]).sum())
            codes += G["hq"][r].size
            if diff:
                flips[s] = diff
                assert np.abs(G["hq"][r].astype(int) - st["qh"].astype(int)).max() <= 1
            ref_yd[s] = (st["yd"], st["yd_abs"], G["yd"][r].astype(np.float64))
    return ref_yd, flips, codes


def check_moe(tq, o, ex, get_expert, x, idx, w, out, ws, tokens, n_ids=None):
    """Staged + end-to-end parity of one tq_moe_grouped call on the listed tokens: xq, xd,
    xb bit-exact against oracle.quantize(x); every routed slot of the tokens staged as in
    check_slots; out ~= sum_j w_j * GPU yd_j over routed j in ascending j (1e-5 of the
    absolute terms). End to end: the fully independent oracle output (fp64), for every
    token whose requantized hidden codes agree with the oracle's own (a fp32 ulp of g or u
    can move an h value across a rounding boundary: one code then differs by 1; the rate
    is bounded and each such token is covered by the staged checks). Slots whose expert id
    is out of range contribute nothing (n_ids as in check_slots). Returns the flip count."""
    t, topk = idx.shape
    H, E = ex.hidden, n_ids or ex.n_experts
    V = ws_views(tq, ex, ws, t, topk)
    tokens = [int(tk) for tk in tokens]
    xq, xd, xb = (_rows(V[n], tokens) for n in ("xq", "xd", "xb"))
    oq, od, ob = o.quantize(x[tokens])
    assert np.array_equal(xq, oq), "xq"
    assert np.array_equal(xd.view(np.uint32), od.view(np.uint32)), "xd"
    assert np.array_equal(xb, ob), "xb"
    ref_yd, flips, codes = check_slots(tq, o, ex, get_expert, x, idx, ws,
                                       [tk * topk + j for tk in tokens for j in range(topk)], V, n_ids)
    outh = _rows(out, tokens).astype(np.float64)
    for n_t, tk in enumerate(tokens):
        staged, staged_abs, ref, ref_abs = (np.zeros(H) for _ in range(4))
        flipped = False
        for j in range(topk):  # ascending j, as the layer defines the sum
            s = tk * topk + j
            if not 0 <= idx[tk, j] < E:
                continue
            wj = float(w[tk, j])
            yr, ya, yg = ref_yd[s]
            staged += wj * yg
            staged_abs += abs(wj) * np.abs(yg)
            ref += wj * yr
            ref_abs += abs(wj) * ya
            flipped |= s in flips
        assert_close(outh[n_t], staged, staged_abs + 1e-30, what=f"out token {tk} (staged)")
        if not flipped:
            assert_close(outh[n_t], ref, ref_abs + 1e-30, what=f"out token {tk}")
    n_flips = sum(flips.values())
    assert n_flips <= max(2, 1e-3 * codes), f"{n_flips} requantized codes differ from the oracle's"
    return n_flips
