"""Seeded synthetic inputs for the compensated-linear workloads.

This module produces *inputs only*: weights, activations, rank tables, routing
tables and, for timing runs, stand-in compensation factors.  It holds none of
the layer's arithmetic (no quantization, no SVD, no forward), so both the fp64
oracle and the HIP path can take their inputs from it.

The paper evaluates on Llama-3.1-8B (INT3) and Qwen3-30B-A3B (INT4) with public
datasets (Section 5.1).  Neither models nor datasets are used: the workloads
below keep the layer shapes and replace the trained weights and the data by
seeded Gaussian draws.

Seeding: every array draws from
``numpy.random.default_rng(SeedSequence([workload, layer, matrix, expert, tag]))``
with tag 0 = weight, 1 = activation, 2 = sensitivity score, 3 = routing logits,
4 = per-expert rank, 5 = stand-in factors, 6 = stand-in packed codes.  Matrices of a decoder layer are
numbered q, k, v, o, gate, up, down = 0..6.
"""

from dataclasses import dataclass, field

import numpy as np

TAG_WEIGHT, TAG_ACT, TAG_SCORE, TAG_ROUTE, TAG_RANK, TAG_FACTOR, TAG_CODES = range(7)

LLAMA_MATS = ("q", "k", "v", "o", "gate", "up", "down")
# (d_out, d_in) of the Llama-3.1-8B decoder-layer linears (GQA: 8 kv heads).
LLAMA_SHAPES = {
    "q": (4096, 4096), "k": (1024, 4096), "v": (1024, 4096), "o": (4096, 4096),
    "gate": (14336, 4096), "up": (14336, 4096), "down": (4096, 14336),
}
# Qwen3-30B-A3B-shaped MoE layer: hidden 2048, 128 experts, expert FFN 768, top-8.
MOE_HIDDEN, MOE_FFN, MOE_EXPERTS, MOE_TOPK, MOE_LAYERS = 2048, 768, 128, 8, 48
MOE_SHAPES = {"gate": (MOE_FFN, MOE_HIDDEN), "up": (MOE_FFN, MOE_HIDDEN), "down": (MOE_HIDDEN, MOE_FFN)}


def rng(workload, layer=0, matrix=0, expert=0, tag=0):
    """The generator every synthetic array of a workload is drawn from."""
    return np.random.default_rng(np.random.SeedSequence([workload, layer, matrix, expert, tag]))


def weight(shape, workload, layer=0, matrix=0, expert=0, std=0.02):
    """``W ~ N(0, std^2)``: drawn in fp64, then cast to float32."""
    g = rng(workload, layer, matrix, expert, TAG_WEIGHT)
    return (std * g.standard_normal(shape)).astype(np.float32)


def fp32_to_bf16_bits(a):
    """Round float32 values to bfloat16 (nearest, ties to even); uint16 bits."""
    b = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return b.astype(np.uint16)


def bf16_bits_to_f64(bits):
    """Exact value of bfloat16 bit patterns as float64."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


@dataclass
class Activation:
    """An activation tensor in the two forms the two sides need."""
    bits: np.ndarray      # uint16 bit patterns (fp16 or bf16), what the kernels read
    values: np.ndarray    # the same numbers exactly, as float64
    dtype: str            # "fp16" or "bf16"


def activation(shape, workload, layer=0, matrix=0, expert=0, dtype="fp16", std=1.0):
    """``x ~ N(0, std^2)`` rounded to fp16 (directly from fp64) or to bf16
    (fp64 -> fp32 -> bf16, both round-to-nearest-even)."""
    g = rng(workload, layer, matrix, expert, TAG_ACT)
    v = std * g.standard_normal(shape)
    if dtype == "fp16":
        h = v.astype(np.float16)
        return Activation(h.view(np.uint16), h.astype(np.float64), "fp16")
    if dtype == "bf16":
        bits = fp32_to_bf16_bits(v.astype(np.float32))
        return Activation(bits, bf16_bits_to_f64(bits), "bf16")
    raise ValueError(dtype)


def standin_factors(d_out, d_in, r_max, workload, layer=0, matrix=0, expert=0, scale=0.05):
    """fp16 ``A`` (r_max x d_in) and ``B`` (d_out x r_max) with Gaussian entries.

    Only for timing and for parity of the forward at sizes where an SVD is too
    slow for a test: the forward's result depends on the factor values, not on
    where they came from, and both sides read the same arrays.
    """
    g = rng(workload, layer, matrix, expert, TAG_FACTOR)
    A = (scale * g.standard_normal((r_max, d_in))).astype(np.float16)
    B = (scale * g.standard_normal((d_out, r_max))).astype(np.float16)
    return A, B


def standin_codes(num_experts, d_out, d_in, bits, group_size, workload, layer=0, matrix=0):
    """Stand-in quantized experts: uniformly random packed words
    ``uint32 [E][d_out][d_in*bits/32]`` (every bit pattern is a valid set of
    codes), fp16 scales ``[E][d_out][d_in/G]`` in the range a group of
    N(0, 0.02) weights gets, and integer fp16 zero points in ``0..2^bits-1``.

    For timing and sampled parity at stacked-expert sizes where quantizing every
    expert on the host is too slow: the forward reads codes, scales and zeros,
    not the weights they came from.
    """
    g = rng(workload, layer, matrix, 0, TAG_CODES)
    words = d_in * bits // 32
    groups = d_in // group_size
    q = g.integers(0, 2 ** 32, size=(num_experts, d_out, words), dtype=np.uint64).astype(np.uint32)
    step = 0.1 / (2 ** bits - 1)
    s = (step * (0.75 + 0.5 * g.random((num_experts, d_out, groups)))).astype(np.float16)
    z = g.integers(0, 2 ** bits, size=(num_experts, d_out, groups)).astype(np.float16)
    return q, s, z


# ---------------------------------------------------------------- rank tables

def align(x, levels):
    """Nearest admissible rank level (ties to the lower level), capped at the
    largest level: the discrete alignment step of the paper's allocator."""
    levels = sorted(levels)
    best = levels[0]
    for lv in levels:
        if abs(x - lv) < abs(x - best):
            best = lv
    return best


def allocate_ranks(scores, levels, budget):
    """Turn synthetic sensitivity scores into a rank table.

    Proportional share of the budget (``score_i / sum(scores) * budget``), then
    :func:`align`, then, while the total exceeds the budget, demote the non-zero
    matrix with the lowest score (lowest index on ties) by one level.
    """
    scores = np.asarray(scores, dtype=np.float64)
    levels = sorted(levels)
    cont = scores / scores.sum() * budget
    ranks = [align(c, levels) for c in cont]
    order = sorted(range(len(ranks)), key=lambda i: (scores[i], i))
    while sum(ranks) > budget:
        for i in order:
            if ranks[i] > 0:
                ranks[i] = levels[levels.index(ranks[i]) - 1]
                break
    return ranks


def llama_layer_ranks(workload, layer=0, levels=(0, 16, 32, 64, 128), per_matrix_budget=64):
    """Per-matrix ranks for the 7 decoder-layer linears from seeded U(0,1)
    scores under a total budget of ``per_matrix_budget * 7``."""
    scores = [rng(workload, layer, m, 0, TAG_SCORE).random() for m in range(len(LLAMA_MATS))]
    ranks = allocate_ranks(scores, levels, per_matrix_budget * len(LLAMA_MATS))
    return dict(zip(LLAMA_MATS, ranks))


def moe_expert_ranks(workload, layer, matrix, num_experts=MOE_EXPERTS, levels=(0, 8, 16, 32)):
    """Per-expert ranks drawn uniformly from ``levels``."""
    g = rng(workload, layer, matrix, 0, TAG_RANK)
    return np.asarray(levels, dtype=np.int32)[g.integers(0, len(levels), num_experts)]


def dynamic_slot_ranks(ids, weights, ranks, levels, r_max):
    """Per-slot ranks from the expert-activation term (Section 4.3.3): slot
    (t, j) routed to expert e with weight g gets ``align(k g r_e)`` capped at
    ``r_max``, with ``k`` the routing width.  An even split (g = 1/k) leaves
    the expert's own rank.  Returns int32 ``[T][k]``."""
    ids = np.asarray(ids)
    k = ids.shape[1]
    out = np.zeros(ids.shape, dtype=np.int32)
    for t in range(ids.shape[0]):
        for j in range(k):
            out[t, j] = min(align(k * float(weights[t][j]) * int(ranks[int(ids[t, j])]), levels), r_max)
    return out


# ------------------------------------------------------------------- routing

def routing(T, workload, layer=0, num_experts=MOE_EXPERTS, k=MOE_TOPK):
    """Top-k routing from a softmax over N(0,1) logits.

    Returns ``(ids int32 [T][k], weights float64 [T][k])``: experts by
    descending probability (ties to the lower id), weights renormalised over the
    k chosen experts so they sum to 1 (the paper's ``sum_e g_e = 1``).
    """
    g = rng(workload, layer, 0, 0, TAG_ROUTE)
    logits = g.standard_normal((T, num_experts))
    p = np.exp(logits - logits.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    ids = np.zeros((T, k), dtype=np.int32)
    w = np.zeros((T, k), dtype=np.float64)
    for t in range(T):
        order = sorted(range(num_experts), key=lambda e: (-p[t, e], e))[:k]
        ids[t] = order
        w[t] = p[t, order] / p[t, order].sum()
    return ids, w


# ------------------------------------------------------------ workload specs

@dataclass
class LinearSpec:
    name: str
    d_out: int
    d_in: int
    bits: int
    group_size: int
    r_max: int
    rank: int


@dataclass
class Workload:
    name: str
    index: int
    linears: list = field(default_factory=list)
    tokens: tuple = (1,)


def single_linear():
    """1024 x 1024, 4-bit, group 128, rank 16, one token."""
    return Workload("single-1024x1024-w4g128-r16", 0,
                    [LinearSpec("w", 1024, 1024, 4, 128, 16, 16)], (1,))


def llama_layer(bits=4, group_size=128, levels=(0, 16, 32, 64, 128), per_matrix_budget=64,
                index=1, tokens=(1, 4, 16)):
    """The seven linears of a Llama-3.1-8B-shaped decoder layer."""
    ranks = llama_layer_ranks(index, 0, levels, per_matrix_budget)
    r_max = max(levels)
    lin = [LinearSpec(m, *LLAMA_SHAPES[m], bits, group_size, r_max, ranks[m]) for m in LLAMA_MATS]
    name = "llama8b-layer-w%dg%d" % (bits, group_size)
    return Workload(name, index, lin, tokens)


def llama_layer_2bit():
    """Aggressive variant: 2-bit, group 64, ranks up to 256 under 128 x 7."""
    return llama_layer(2, 64, (0, 16, 32, 64, 128, 256), 128, index=2, tokens=(1,))


def llama_layer_3bit():
    """The paper's dense-model setting: 3-bit codes (INT3, Section 5.1),
    group 128, ranks from {0, 16, 32, 64, 128} under 64 x 7."""
    return llama_layer(3, 128, index=7, tokens=(1, 4, 16))
