"""Seeded synthetic inputs for the tied-trit-plane expert dot pass.

This module holds random draws only: activations, per-token scale factors, routing
indices and routing weights, fp32 weights for the tied quantizer, trit planes and scale
pairs for the free-scale two-plane variant, e2m1 codes and e8m0 exponents for the MXFP4
arm, and the 64-bit keys
that name each weight matrix's counter-based stream. None of the method's arithmetic (fold, pack, quantize, integer
dot, scale combine, SiLU, weighted combine) lives here; both the CPU oracle and the
HIP path consume these draws, and each implements the method on its own.

Weight matrices are too large to draw on the host for the big workloads (the 43-layer
stack holds ~246 GB of packed codes), so they are defined by a counter-based
generator that each side implements from its published definition (SplitMix64,
Steele, Lea & Flood, OOPSLA 2014). The recipe, for a matrix with key ``key``, ``n``
rows, ``k`` columns (k a multiple of 256):

* ``word(key, i) = mix64(key + (i + 1) * 0x9E3779B97F4A7C15)`` (the i-th SplitMix64
  output of a generator whose state starts at ``key``), where ``mix64`` is
  SplitMix64's finaliser: ``z ^= z >> 30; z *= 0xBF58476D1CE4E5B9; z ^= z >> 27;
  z *= 0x94D049BB133111EB; z ^= z >> 31`` (all mod 2**64).
* Weight element ``e = row * k + col`` (row-major logical index) takes word
  ``word(key, e >> 1)``; its four 16-bit fields f0..f3 (f0 least significant) give
  the trits: an even ``e`` takes t1 from f0 and t2 from f1, an odd ``e`` takes t1 from
  f2 and t2 from f3. A field maps to a trit by ``((f * 3) >> 16) - 1`` (a 16-bit
  multiply-shift range reduction, Lemire 2019; P(-1) = 21846/65536, P(0) = P(1) =
  21845/65536).
* Scale ``j = row * (k // 256) + block`` takes word ``word(key, n * k // 2 + j)`` and
  maps its high 32 bits ``h`` to the fp16 bit pattern
  ``SCALE_F16_LO + ((h * SCALE_F16_SPAN) >> 32)``: uniform over the fp16 values in
  [1e-3, 1e-1], which is log-uniform at binade granularity (every binade holds the
  same 1024 patterns).
"""

from __future__ import annotations

import numpy as np

# SplitMix64 constants (Steele, Lea & Flood 2014; finaliser "mix64" variant 13).
SPLITMIX_GAMMA = 0x9E3779B97F4A7C15
SPLITMIX_M1 = 0xBF58476D1CE4E5B9
SPLITMIX_M2 = 0x94D049BB133111EB

# fp16 bit patterns bracketing the scale range [1e-3, 1e-1]:
# 0x1419 = 1.0244e-3 is the smallest fp16 >= 1e-3, 0x2E66 = 0.099976 the largest <= 0.1.
SCALE_F16_LO = 0x1419
SCALE_F16_HI = 0x2E66
SCALE_F16_SPAN = SCALE_F16_HI - SCALE_F16_LO + 1

SEED = 0

# Named sub-streams for the numpy draws.
_TAG_ACT = 1
_TAG_ROUTE = 2
_TAG_LOGIT = 3
_TAG_FACTOR = 4
_TAG_KEY = 5
_TAG_BENCH = 6
_TAG_FWEIGHT = 7
_TAG_TWOPLANE = 8
_TAG_MXFP4 = 9

PROJ_GATE, PROJ_UP, PROJ_DOWN = 0, 1, 2

# The five workloads: expert-matrix shapes of the paper's model (hidden 4096, expert
# intermediate 2048, 256 routed experts per layer; 43 MoE layers at hidden 7168 for
# the deep stack).
CONFIGS = {
    0: dict(name="tq_gemv_2048x4096_t1", kind="gemv", n=2048, k=4096, tokens=1),
    1: dict(name="moe_decode_e256_h4096_i2048_t1_top8_uniform", kind="moe",
            experts=256, hidden=4096, inter=2048, tokens=1, topk=8, routing="uniform",
            layers=1),
    2: dict(name="moe_decode_e256_h4096_i2048_t32_top8_zipf1.1", kind="moe",
            experts=256, hidden=4096, inter=2048, tokens=32, topk=8, routing="zipf",
            layers=1),
    3: dict(name="moe_prefill_e256_h4096_i2048_t2048_top8_zipf1.1_logfactor", kind="moe",
            experts=256, hidden=4096, inter=2048, tokens=2048, topk=8, routing="zipf",
            token_factor=True, layers=1),
    4: dict(name="moe_stack_l43_e256_h7168_i2048_t8_top8_zipf1.1", kind="moe",
            experts=256, hidden=7168, inter=2048, tokens=8, topk=8, routing="zipf",
            layers=43),
}


# The tied quantizer's workload (the producer of the persistent bytes): fp32 weights of
# 32 expert projections at the paper model's 2048 x 4096 expert shape.
QUANT_CONFIG = dict(name="tied_quantize_m32_2048x4096", kind="quant", matrices=32, n=2048, k=4096)


# The free-scale two-plane variant's workload: one decode step's routed gate and up rows
# (8 experts x 2 x 2048 rows of 4096 inputs) as one stacked matrix, one token, served
# from the two-plane layout; the folded layout of the same planes is timed beside it.
TWO_PLANE_CONFIG = dict(name="twoplane_gemv_32768x4096_t1", kind="twoplane", n=32768, k=4096, tokens=1)


# The MXFP4 reference arm's workload: the same stacked decode rows in the released-bytes
# format (e2m1 codes, one e8m0 scale per 32), one token.
MXFP4_CONFIG = dict(name="mxfp4_gemv_32768x4096_t1", kind="mxfp4", n=32768, k=4096, tokens=1)


def _rng(*key: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence(entropy=int(key[0]), spawn_key=tuple(int(v) for v in key[1:])))


def matrix_key(seed: int, layer: int, expert: int, proj: int) -> int:
    """64-bit stream key of one weight matrix (proj: 0 gate, 1 up, 2 down)."""
    w = np.random.SeedSequence(entropy=int(seed), spawn_key=(_TAG_KEY, int(layer), int(expert), int(proj))).generate_state(2, np.uint32)
    return int(w[0]) | (int(w[1]) << 32)


def single_matrix_key(seed: int = SEED) -> int:
    """Key of the lone matrix of the single-GEMV workload."""
    return matrix_key(seed, 0xFFFF, 0, 0)


def activations(seed: int, layer: int, tokens: int, width: int) -> np.ndarray:
    """N(0,1) fp32 activations [tokens][width]."""
    return _rng(seed, _TAG_ACT, layer).standard_normal((tokens, width), dtype=np.float32)


def float_weights(seed: int, index: int, n: int, k: int) -> np.ndarray:
    """fp32 weights [n][k] for the tied quantizer: N(0,1) times a per-row spread drawn
    log-uniform on [0.005, 0.05] (the magnitude range of transformer projection weights)."""
    r = _rng(seed, _TAG_FWEIGHT, index)
    sigma = np.exp(np.log(0.005) + r.random((n, 1)) * (np.log(0.05) - np.log(0.005)))
    return (r.standard_normal((n, k), dtype=np.float32) * sigma.astype(np.float32)).astype(np.float32)


def two_plane_weights(seed: int, index: int, n: int, k: int):
    """A free-scale two-plane matrix: trit planes t1, t2 [n][k] (int8, uniform on
    {-1, 0, 1}) and scale pairs [n][k/256][2] as f16 bit patterns (uint16): alpha2
    log-uniform on [1e-3, 1e-1], alpha1 = alpha2 times 3 * U(0.75, 1.25), i.e. near the
    tied ratio with a +-25% spread."""
    r = _rng(seed, _TAG_TWOPLANE, index)
    t1 = r.integers(-1, 2, (n, k), dtype=np.int8)
    t2 = r.integers(-1, 2, (n, k), dtype=np.int8)
    a2 = np.exp(r.uniform(np.log(1e-3), np.log(1e-1), (n, k // 256)))
    a1 = a2 * 3.0 * r.uniform(0.75, 1.25, (n, k // 256))
    a = np.stack([a1, a2], axis=2).astype(np.float16).view(np.uint16)
    return t1, t2, np.ascontiguousarray(a)


def mxfp4_weights(seed: int, index: int, n: int, k: int):
    """An MXFP4 matrix: e2m1 codes [n][k] (uint8, uniform on 0..15) and e8m0 exponents
    [n][k/32] (uint8, uniform on 116..124, i.e. block scales 2^-11 .. 2^-3)."""
    r = _rng(seed, _TAG_MXFP4, index)
    c4 = r.integers(0, 16, (n, k), dtype=np.uint8)
    e8 = r.integers(116, 125, (n, k // 32), dtype=np.uint8)
    return c4, e8


def token_factors(seed: int, tokens: int) -> np.ndarray:
    """Per-token factor, log-uniform on [0.1, 10] (fp32)."""
    u = _rng(seed, _TAG_FACTOR).random(tokens)
    return np.exp(np.log(0.1) + u * (np.log(10.0) - np.log(0.1))).astype(np.float32)


def zipf_probs(experts: int, s: float = 1.1) -> np.ndarray:
    p = (np.arange(1, experts + 1, dtype=np.float64)) ** (-s)
    return p / p.sum()


def routing(seed: int, layer: int, tokens: int, experts: int, topk: int, kind: str):
    """Top-k expert indices [tokens][topk] (int32, distinct per token) and softmax
    routing weights [tokens][topk] (fp32) over topk N(0,1) logits.

    ``uniform``: indices drawn without replacement, uniformly.
    ``zipf``: popularity p_e proportional to (e+1)^-1.1 over the experts; the topk
    distinct experts per token are a Gumbel-top-k draw (sequential weighted sampling
    without replacement).
    """
    rng = _rng(seed, _TAG_ROUTE, layer)
    if kind == "uniform":
        idx = np.stack([rng.choice(experts, size=topk, replace=False) for _ in range(tokens)])
    elif kind == "zipf":
        logp = np.log(zipf_probs(experts))
        g = rng.gumbel(size=(tokens, experts))
        idx = np.argsort(-(logp[None, :] + g), axis=1, kind="stable")[:, :topk]
    else:
        raise ValueError(kind)
    logits = _rng(seed, _TAG_LOGIT, layer).standard_normal((tokens, topk))
    w = np.exp(logits - logits.max(axis=1, keepdims=True))
    w = w / w.sum(axis=1, keepdims=True)
    return idx.astype(np.int32), w.astype(np.float32)


def bench_routing_schedule(seed: int, steps: int, tokens: int, experts: int, topk: int,
                           kind: str, exclude_recent: int = 3, wrap_from: int | None = None):
    """A sequence of per-step routings for timing. Each step's experts avoid those of
    the previous ``exclude_recent`` steps, so that an expert's bytes are never re-read
    while still resident in a 256 MB last-level cache (the reuse distance exceeds
    ``exclude_recent`` steps of expert bytes). With ``wrap_from``, the last
    ``exclude_recent`` steps also avoid the experts of steps ``wrap_from`` onwards (as
    many), so that steps wrap_from .. steps-1 can be replayed in a loop. Returns lists of
    (idx, w)."""
    rng = _rng(seed, _TAG_BENCH, steps)
    out = []
    recent: list[set[int]] = []
    for i in range(steps):
        banned = set().union(*recent) if recent else set()
        if wrap_from is not None and i >= steps - exclude_recent and i - wrap_from >= exclude_recent:
            for k in range(wrap_from, min(wrap_from + exclude_recent, steps)):
                if k < len(out):
                    banned |= set(int(e) for e in out[k][0].ravel())
        allowed = np.array([e for e in range(experts) if e not in banned])
        if kind == "uniform":
            idx = np.stack([rng.choice(allowed, size=topk, replace=False) for _ in range(tokens)])
        else:
            logp = np.log(zipf_probs(experts))[allowed]
            g = rng.gumbel(size=(tokens, allowed.size))
            idx = allowed[np.argsort(-(logp[None, :] + g), axis=1, kind="stable")[:, :topk]]
        logits = rng.standard_normal((tokens, topk))
        w = np.exp(logits - logits.max(axis=1, keepdims=True))
        w = w / w.sum(axis=1, keepdims=True)
        out.append((idx.astype(np.int32), w.astype(np.float32)))
        recent.append(set(int(e) for e in idx.ravel()))
        if len(recent) > exclude_recent:
            recent.pop(0)
    return out
