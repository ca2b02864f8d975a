"""GPU parity of the deep MoE stack: 43 routed-expert layers of 256 experts at hidden
7168, expert intermediate 2048 (the paper's model shape: 43 x 3 x 256 expert matrices,
Sec. 2.1), all 246 GB of folded codes and scales resident in HBM at once, 8 tokens per
step with Zipf(1.1) top-8 routing and independent N(0,1) inputs per layer.

One step runs all 43 layers on the GPU, each on its own experts, input and routing.
The oracle regenerates the routed experts of the first and the last layer from the
counter-based generator and checks sampled tokens there (every stage, staged and end
to end; those two layers run with the debug stage dump, so their gate, up and down
block sums are compared bit for bit); every layer's quantized input is checked
bit-exactly for all tokens, and every layer's output, for all tokens, against the
routing-weighted sum of its own slots' down outputs."""
import numpy as np
import pytest
import torch

import oracle as oracle_pkg
from gpu_util import announce, check_moe, synth_experts, ws_views
from synth import gen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tq():
    from gpu_util import device
    device()
    from paper_2608_08910_amd import tq as _tq
    return _tq


def test_stack_43_layers_h7168_full_size(tq, oracle):
    c = gen.CONFIGS[4]
    L, E, H, I, T, topk = c["layers"], c["experts"], c["hidden"], c["inter"], c["tokens"], c["topk"]
    torch.cuda.empty_cache()
    per_layer = 3 * (I * H // 2 + I * (H // 256) * 2)
    free, _ = torch.cuda.mem_get_info()
    if free < L * E * per_layer + (2 << 30):
        pytest.skip(f"needs {L * E * per_layer / 1e9:.1f} GB of free device memory, {free / 1e9:.1f} GB free")
    announce(f"stack synth {L} layers x {E} experts h{H} i{I} ({L * E * per_layer / 1e9:.1f} GB)")
    layers = [synth_experts(tq, gen.SEED, l, E, H, I) for l in range(L)]
    torch.cuda.synchronize()
    xs, idxs, ws_, outs, wts = [], [], [], [], []
    for l in range(L):
        x = gen.activations(gen.SEED, l, T, H)
        idx, w = gen.routing(gen.SEED, l, T, E, topk, c["routing"])
        xs.append(x); idxs.append(idx); wts.append(w)
        ws_.append(tq.moe_workspace(layers[l], T, topk, debug=l in (0, L - 1)))
        outs.append(torch.empty((T, H), dtype=torch.float32, device="cuda"))
    xd = [torch.from_numpy(x).cuda() for x in xs]
    idd = [torch.from_numpy(i).cuda() for i in idxs]
    wd = [torch.from_numpy(w).cuda() for w in wts]
    announce("stack step: 43 layers")
    for l in range(L):
        tq.tq_moe_grouped(layers[l], xd[l], idd[l], wd[l], outs[l], ws_[l],
                          tq.TQ_MOE_DEBUG_STAGES if l in (0, L - 1) else 0)
    torch.cuda.synchronize()
    for l in range(L):
        V = ws_views(tq, layers[l], ws_[l], T, topk)
        oq, od, ob = oracle.quantize(xs[l])
        assert np.array_equal(V["xq"].cpu().numpy(), oq), f"layer {l}: quantized input"
        assert np.array_equal(V["xd"].cpu().numpy().view(np.uint32), od.view(np.uint32))
        assert tq.tq_moe_status(ws_[l], layers[l], T, topk) == 0
        assert torch.isfinite(outs[l]).all()
        yd = V["yd"].view(T, topk, H).double()
        w64 = wd[l].double()
        staged = (w64[:, :, None] * yd).sum(1)
        staged_abs = (w64[:, :, None].abs() * yd.abs()).sum(1)
        ratio = ((outs[l].double() - staged).abs() / (staged_abs + 1e-30)).max().item()
        assert ratio <= 1e-5, f"layer {l}: out vs its slots' yd, worst {ratio:.3g} of the absolute terms"
    # the first and last layers again without the debug dump: the one-launch mixed kernels
    # (hidden 7168: 28 blocks a row, four loads per lane, the last partly past the row
    # end) give bitwise the outputs of the debug run's separate VALU and MFMA kernels,
    # which the oracle checks below
    assert tq.tq_moe_path(layers[0], T, topk) == tq.TQ_MOE_PATH_MIXED
    for l in (0, L - 1):
        assert (np.bincount(idxs[l].ravel(), minlength=E) > 2).any()  # the MFMA role has experts
        plain = torch.empty_like(outs[l])
        tq.tq_moe_grouped(layers[l], xd[l], idd[l], wd[l], plain, tq.moe_workspace(layers[l], T, topk))
        torch.cuda.synchronize()
        assert torch.equal(plain, outs[l]), f"layer {l}: output changes with TQ_MOE_DEBUG_STAGES"
    for l, tokens in ((0, [0, 5]), (L - 1, [3, 7])):
        announce(f"stack oracle layer {l} tokens {tokens}")
        get = oracle_pkg.expert_getter(gen.SEED, l, H, I, oracle)
        check_moe(tq, oracle, layers[l], get, xs[l], idxs[l], wts[l], outs[l], ws_[l], tokens)
