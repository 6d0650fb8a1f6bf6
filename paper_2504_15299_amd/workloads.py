"""Seeded synthetic MoE-layer workloads.

This module only draws inputs: activations, expert weights, gate weights, the
request map and the per-(request, expert) bit-width tables.  It holds none of
the method's arithmetic, so both the GPU path and the CPU oracle can consume
the same arrays.  There are no pretrained weights or datasets here: seeded
Gaussians of the layer shapes the paper evaluates (Mixtral-8x7B style, 8
experts, top-2) and a fine-grained MoE shape stand in for them.

Streams are independent: every tensor gets its own ``SeedSequence`` child keyed
by (seed, layer, purpose, expert).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

# purpose keys for the seed tree
_X, _WG, _W13, _W2, _BITS, _SH13, _SH2, _ROUTER = range(8)


@dataclass
class LayerSpec:
    name: str
    d: int                      # d_model
    f: int                      # d_ff of a routed expert
    E: int                      # routed experts
    k: int                      # top-k
    T: int                      # tokens in the batch
    group: int                  # MWQ group size
    x_dtype: str                # "bf16" or "f32"
    b_min: int = 2
    b_max: int = 8
    n_requests: int = 1
    shared_f: int = 0           # 0 = no shared expert
    shared_bits: int = 8
    seed: int = 0
    w_std: float = 0.02
    gate_std: float = 0.02
    zipf_s: float = 0.0         # > 0: gate bias ln p_e, p_e ~ (e+1)^-s
    bits_choices: tuple = (2, 4, 8)
    bits_probs: tuple | None = None
    bits_mode: str = "per_request_expert"   # or "per_request", "hottest_first"
    extra: dict = field(default_factory=dict)


def _rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, *key])))


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round binary32 values to the nearest bfloat16 (ties to even), returned as
    binary32 values that are exactly representable in bfloat16."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    lower = u & np.uint32(0xFFFF)
    upper = u & np.uint32(0xFFFF0000)
    up = (lower > 0x8000) | ((lower == 0x8000) & ((upper & np.uint32(0x10000)) != 0))
    upper = upper + np.where(up, np.uint32(0x10000), np.uint32(0))
    return upper.astype(np.uint32).view(np.float32)


# ---- workloads ----------------------------------------------------------------

def tiny(seed: int = 0) -> LayerSpec:
    """d_model 256, d_ff 512, 8 SwiGLU experts, top-2, 64 tokens, fp32
    activations, group 64, per-expert bit-width uniform from {2,4,8}."""
    return LayerSpec("tiny", d=256, f=512, E=8, k=2, T=64, group=64, x_dtype="f32",
                     seed=seed, bits_choices=(2, 4, 8), bits_mode="per_request_expert")


def mixtral_decode(T: int = 16, seed: int = 2) -> LayerSpec:
    """Mixtral-8x7B-shaped layer in decode: d_model 4096, d_ff 14336, 8 experts,
    top-2, one request per token, per-(request, expert) bit-width from
    {2,3,4,8} with probabilities {.2,.3,.3,.2}, group 128, bf16."""
    return LayerSpec("mixtral_decode", d=4096, f=14336, E=8, k=2, T=T, group=128,
                     x_dtype="bf16", n_requests=T, seed=seed, bits_choices=(2, 3, 4, 8),
                     bits_probs=(0.2, 0.3, 0.3, 0.2))


def mixtral_prefill(seed: int = 3) -> LayerSpec:
    """Same layer in prefill: 2048 tokens from 4 requests of 512, each request
    with its own per-expert bit-width table from {2,4,8}; gate bias so that
    expert load follows Zipf(s = 1.1)."""
    return LayerSpec("mixtral_prefill", d=4096, f=14336, E=8, k=2, T=2048, group=128,
                     x_dtype="bf16", n_requests=4, seed=seed, zipf_s=1.1,
                     bits_choices=(2, 4, 8))


def fine_grained(seed: int = 4) -> LayerSpec:
    """Fine-grained MoE: d_model 2048, 64 routed experts d_ff 1408, top-6, one
    always-on shared expert d_ff 5632 at 8 bits, 512 tokens, group 64;
    bit-widths hottest-first (16 at 8, 16 at 4, 16 at 3, rest at 2)."""
    return LayerSpec("fine_grained", d=2048, f=1408, E=64, k=6, T=512, group=64,
                     x_dtype="bf16", seed=seed, shared_f=5632, shared_bits=8,
                     bits_mode="hottest_first")


def mixtral_decode_v1(T: int = 16, seed: int = 6) -> LayerSpec:
    """The Mixtral decode layer under the paper's first configuration (Sec. 5):
    nest b_1 = 2 to b_K = 4, group 128, per-(request, expert) bit-widths
    {2,3,4} drawn with the expert capacities {.3,.4,.3}."""
    return LayerSpec("mixtral_decode_v1", d=4096, f=14336, E=8, k=2, T=T, group=128,
                     x_dtype="bf16", n_requests=T, seed=seed, b_min=2, b_max=4,
                     bits_choices=(2, 3, 4), bits_probs=(0.3, 0.4, 0.3))


def mixtral_decode_v2(T: int = 16, seed: int = 7) -> LayerSpec:
    """The Mixtral decode layer under the paper's second configuration
    (Sec. 5): nest b_1 = 5 to b_K = 8, group 128, per-(request, expert)
    bit-widths {5,6,7,8} with capacity .25 each."""
    return LayerSpec("mixtral_decode_v2", d=4096, f=14336, E=8, k=2, T=T, group=128,
                     x_dtype="bf16", n_requests=T, seed=seed, b_min=5, b_max=8,
                     bits_choices=(5, 6, 7, 8), bits_probs=(0.25, 0.25, 0.25, 0.25))


def dense_decode(T: int = 16, seed: int = 8) -> LayerSpec:
    """A dense LLM's SwiGLU FFN (LLaMA2-13B shape: d_model 5120, d_ff 13824)
    as the one-expert, top-1 case of the same layer (the paper's dense-model
    extension, Sec. 5), decoding T requests with per-request bit-widths of the
    first configuration's nest {2,3,4} ({.3,.4,.3}), group 128."""
    return LayerSpec("dense_decode", d=5120, f=13824, E=1, k=1, T=T, group=128,
                     x_dtype="bf16", n_requests=T, seed=seed, b_min=2, b_max=4,
                     bits_choices=(2, 3, 4), bits_probs=(0.3, 0.4, 0.3))


def mixtral_stack(seed: int = 5) -> LayerSpec:
    """32 Mixtral-8x7B-shaped MoE layers stacked as decoder blocks
    x <- x + MoE_l(rmsnorm(x)) (attention absent, unit normalisation weight,
    eps 1e-5), 64 sequences decoding 128 steps; every sequence is a request
    with one bit-width tier from {2,4,8} for all experts and layers; gate,
    experts and activations drawn per layer from the layer's own streams."""
    return LayerSpec("mixtral_stack", d=4096, f=14336, E=8, k=2, T=64, group=128,
                     x_dtype="bf16", n_requests=64, seed=seed, bits_choices=(2, 4, 8),
                     bits_mode="per_request",
                     extra={"layers": 32, "steps": 128, "eps": 1e-5})


def scaled(spec: LayerSpec, **kw) -> LayerSpec:
    """A copy of ``spec`` with some fields replaced (smaller test shapes)."""
    d = dict(spec.__dict__)
    d.update(kw)
    return LayerSpec(**d)


# ---- draws ------------------------------------------------------------------

def activations(spec: LayerSpec, layer: int = 0) -> np.ndarray:
    """[T][d] binary32; bf16 workloads are rounded to bf16 values."""
    x = _rng(spec.seed, layer, _X).standard_normal((spec.T, spec.d), dtype=np.float32)
    return round_to_bf16(x) if spec.x_dtype == "bf16" else x


def gate(spec: LayerSpec, layer: int = 0):
    """Gate weights [E][d] (binary32) and bias [E] or None."""
    Wg = (_rng(spec.seed, layer, _WG).standard_normal((spec.E, spec.d), dtype=np.float32)
          * np.float32(spec.gate_std))
    bias = None
    if spec.zipf_s > 0:
        p = (np.arange(spec.E, dtype=np.float64) + 1.0) ** (-spec.zipf_s)
        p /= p.sum()
        bias = np.log(p).astype(np.float32)
    return Wg, bias


def expert_w13(spec: LayerSpec, e: int, layer: int = 0) -> np.ndarray:
    """[2 d_ff][d] binary32: W1 (gate projection) rows, then W3 (up) rows."""
    return (_rng(spec.seed, layer, _W13, e).standard_normal((2 * spec.f, spec.d),
                                                             dtype=np.float32)
            * np.float32(spec.w_std))


def expert_w2(spec: LayerSpec, e: int, layer: int = 0) -> np.ndarray:
    """[d][d_ff] binary32 (down projection)."""
    return (_rng(spec.seed, layer, _W2, e).standard_normal((spec.d, spec.f), dtype=np.float32)
            * np.float32(spec.w_std))


def shared_w13(spec: LayerSpec, layer: int = 0) -> np.ndarray:
    return (_rng(spec.seed, layer, _SH13).standard_normal((2 * spec.shared_f, spec.d),
                                                           dtype=np.float32)
            * np.float32(spec.w_std))


def shared_w2(spec: LayerSpec, layer: int = 0) -> np.ndarray:
    return (_rng(spec.seed, layer, _SH2).standard_normal((spec.d, spec.shared_f),
                                                          dtype=np.float32)
            * np.float32(spec.w_std))


def bit_routers(spec: LayerSpec, layer: int = 0, std: float = 0.05):
    """Weights of the per-expert bit-width routers, one linear map from the
    token to the nest's L = b_max - b_min + 1 widths: Wr [E][L][d] and bias
    br [E][L] (binary32 Gaussians; trained router weights are not
    available)."""
    L = spec.b_max - spec.b_min + 1
    g = _rng(spec.seed, layer, _ROUTER)
    Wr = g.standard_normal((spec.E, L, spec.d), dtype=np.float32) * np.float32(std)
    br = g.standard_normal((spec.E, L), dtype=np.float32) * np.float32(std)
    return Wr, br


def token_requests(spec: LayerSpec) -> np.ndarray:
    """Request id of every token: contiguous equal blocks."""
    per = max(spec.T // spec.n_requests, 1)
    return np.minimum(np.arange(spec.T) // per, spec.n_requests - 1).astype(np.int32)


def bit_table(spec: LayerSpec, layer: int = 0, expert_counts=None) -> np.ndarray:
    """[n_requests][E] uint8 bit-widths.

    ``per_request_expert``: independent draw per (request, expert);
    ``per_request``: one tier per request for all experts;
    ``hottest_first``: needs ``expert_counts`` (tokens routed to each expert):
    experts ranked by count (descending, ties to the lower id); the first 16
    get 8 bits, the next 16 get 4, the next 16 get 3 and the rest 2."""
    R, E = spec.n_requests, spec.E
    rng = _rng(spec.seed, layer, _BITS)
    ch = np.asarray(spec.bits_choices, dtype=np.uint8)
    if spec.bits_mode == "per_request_expert":
        return rng.choice(ch, size=(R, E), p=spec.bits_probs).astype(np.uint8)
    if spec.bits_mode == "per_request":
        tiers = rng.choice(ch, size=(R, 1), p=spec.bits_probs).astype(np.uint8)
        return np.repeat(tiers, E, axis=1)
    if spec.bits_mode == "hottest_first":
        if expert_counts is None:
            raise ValueError("hottest_first bit assignment needs expert_counts")
        counts = np.asarray(expert_counts)
        order = sorted(range(E), key=lambda e: (-int(counts[e]), e))
        tiers = [8] * 16 + [4] * 16 + [3] * 16
        t = np.full(E, 2, np.uint8)
        for rank, e in enumerate(order):
            if rank < len(tiers):
                t[e] = tiers[rank]
        return np.repeat(t[None, :], R, axis=0)
    raise ValueError(spec.bits_mode)
