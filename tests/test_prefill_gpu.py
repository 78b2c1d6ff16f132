"""cl_linear_prefill against the fp64 oracle (Section 4.1 forward, many
tokens): relative L2 <= 1e-3 for every output dtype over ragged token and row
counts, ranks including 0 and non-multiples of 32, 2/3/4-bit codes and
fp16/bf16 activations; the Llama-8B prefill shapes (M = 2048) on sampled
outputs; agreement with the decode path; bitwise determinism.  The GEMM
multiplies dequantized weight tiles rounded to fp16 (and T = X A^T rounded
to fp16), so besides the relative L2 bar every element is held to the
rounding bound of that arithmetic (tests.helpers.fp16_tile_bound)."""

import numpy as np
import pytest
import torch

from oracle import linear, quant
from paper_2605_05819_amd import cl, workloads as wl
from tests.helpers import assert_oracle, dev_f16, dev_u16, dev_u32, fp16_tile_bound, out_to_numpy, rel_l2

pytestmark = pytest.mark.gpu


def _layer(d_out, d_in, bits, G, r_max, seed):
    W = wl.weight((d_out, d_in), 20, seed)
    Q, s, z = quant.quantize_pack(W, bits, G)
    A, B = wl.standin_factors(d_out, d_in, r_max, 20, seed)
    w = cl.QWeight(dev_u32(Q), dev_f16(s), dev_f16(z), d_out, d_in, bits, G)
    return w, (Q, s, z, A, B)


@pytest.mark.parametrize("bits,G", [(4, 128), (2, 64), (4, 64), (4, 32), (3, 128), (3, 32)])
@pytest.mark.parametrize("M,d_out,d_in", [(37, 300, 256), (256, 128, 512), (300, 1000, 1024), (70, 260, 2560)])
@pytest.mark.parametrize("rank", [0, 17, 64])
def test_prefill_ragged_vs_oracle(bits, G, M, d_out, d_in, rank):
    w, (Q, s, z, A, B) = _layer(d_out, d_in, bits, G, 64, M + d_out + rank + bits)
    c = cl.LowRank(dev_f16(A), dev_f16(B), 64, rank)
    x = wl.activation((M, d_in), 20, M, d_out)
    y = cl.linear_prefill(w, c, dev_u16(x.bits, torch.float16), out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref = linear.forward_packed(Q, s, z, bits, G, A, B, rank, x.values)
    W_hat = quant.dequant_packed(Q, s, z, bits, G, d_in)
    assert_oracle(out_to_numpy(y), ref, extra=fp16_tile_bound(W_hat, x.values, A, B, rank))


@pytest.mark.parametrize("out", [torch.float32, torch.float16, torch.bfloat16])
@pytest.mark.parametrize("act", ["fp16", "bf16"])
def test_prefill_dtypes(out, act):
    M, d_out, d_in = 129, 257, 768
    w, (Q, s, z, A, B) = _layer(d_out, d_in, 4, 128, 64, 7)
    c = cl.LowRank(dev_f16(A), dev_f16(B), 64, 48)
    x = wl.activation((M, d_in), 21, dtype=act)
    dt = torch.float16 if act == "fp16" else torch.bfloat16
    y = cl.linear_prefill(w, c, dev_u16(x.bits, dt), out_dtype=out)
    ref = linear.forward_packed(Q, s, z, 4, 128, A, B, 48, x.values)
    W_hat = quant.dequant_packed(Q, s, z, 4, 128, d_in)
    assert_oracle(out_to_numpy(y), ref, out, extra=fp16_tile_bound(W_hat, x.values, A, B, 48))


@pytest.mark.parametrize("d_out", [4096, 14336])
@pytest.mark.parametrize("act", ["fp16", "bf16"])
def test_prefill_llama_shapes_sampled(d_out, act):
    """M = 2048 tokens through a 4096-wide layer at rank 64, the prefill
    workload; outputs checked on sampled rows and tokens."""
    M, d_in, rank = 2048, 4096, 64
    W = wl.weight((d_out, d_in), 4, 0, d_out)
    w = cl.quantize_pack(torch.from_numpy(W).cuda(), 4, 128)
    A, B = wl.standin_factors(d_out, d_in, 64, 4, 0, d_out)
    c = cl.LowRank(dev_f16(A), dev_f16(B), 64, rank)
    x = wl.activation((M, d_in), 4, 0, d_out, dtype=act)
    dt = torch.float16 if act == "fp16" else torch.bfloat16
    y = cl.linear_prefill(w, c, dev_u16(x.bits, dt), out_dtype=torch.float32)
    torch.cuda.synchronize()
    g = np.random.default_rng(d_out)
    rows = np.r_[0:2, g.choice(d_out, 100, replace=False), d_out - 2:d_out]
    toks = np.r_[0:2, g.choice(M, 60, replace=False), M - 2:M]
    Q, s, z = quant.quantize_pack(W[rows], 4, 128)
    ref = linear.forward_packed(Q, s, z, 4, 128, A, B[rows], rank, x.values[toks])
    got = out_to_numpy(y)[np.ix_(toks, rows)]
    W_hat = quant.dequant_packed(Q, s, z, 4, 128, d_in)
    assert_oracle(got, ref, extra=fp16_tile_bound(W_hat, x.values[toks], A, B[rows], rank))


def test_prefill_llama_3bit_sampled():
    """The paper's INT3 setting: M = 2048 tokens through the 14336 x 4096
    gate with 3-bit codes (group 128) at rank 64, sampled rows and tokens."""
    M, d_out, d_in, rank = 2048, 14336, 4096, 64
    W = wl.weight((d_out, d_in), 4, 3, d_out)
    w = cl.quantize_pack(torch.from_numpy(W).cuda(), 3, 128)
    A, B = wl.standin_factors(d_out, d_in, 64, 4, 3, d_out)
    c = cl.LowRank(dev_f16(A), dev_f16(B), 64, rank)
    x = wl.activation((M, d_in), 4, 3, d_out)
    y = cl.linear_prefill(w, c, dev_u16(x.bits, torch.float16), out_dtype=torch.float32)
    torch.cuda.synchronize()
    g = np.random.default_rng(3)
    rows = np.r_[0:2, g.choice(d_out, 100, replace=False), d_out - 2:d_out]
    toks = np.r_[0:2, g.choice(M, 60, replace=False), M - 2:M]
    Q, s, z = quant.quantize_pack(W[rows], 3, 128)
    ref = linear.forward_packed(Q, s, z, 3, 128, A, B[rows], rank, x.values[toks])
    got = out_to_numpy(y)[np.ix_(toks, rows)]
    W_hat = quant.dequant_packed(Q, s, z, 3, 128, d_in)
    assert_oracle(got, ref, extra=fp16_tile_bound(W_hat, x.values[toks], A, B[rows], rank))


def test_prefill_bf16_activations_beyond_the_fp16_range():
    """The documented bf16 conversion in prefill's X': tokens at scale 1e5
    saturate at +-65504, tokens at scale 1e-6 round to multiples of 2^-24;
    each token against the oracle on the converted values.  The backbone
    alone: T = X A^T is fp16, whose range these scales leave."""
    M, d_out, d_in, rank = 40, 300, 1024, 0
    w, (Q, s, z, A, B) = _layer(d_out, d_in, 4, 128, 32, 41)
    c = None
    g = np.random.default_rng(41)
    scale = np.where(np.arange(M) % 2 == 0, 1e5, 1e-6)[:, None]
    xb = wl.fp32_to_bf16_bits((scale * g.standard_normal((M, d_in))).astype(np.float32))
    seen = np.clip(wl.bf16_bits_to_f64(xb), -65504.0, 65504.0).astype(np.float16).astype(np.float64)
    y = out_to_numpy(cl.linear_prefill(w, c, dev_u16(xb, torch.bfloat16), out_dtype=torch.float32))
    ref = linear.forward_packed(Q, s, z, 4, 128, A, B, rank, seen)
    W_hat = quant.dequant_packed(Q, s, z, 4, 128, d_in)
    for m in range(M):
        assert_oracle(y[m], ref[m], extra=fp16_tile_bound(W_hat, seen[m:m + 1])[0])


def _random_prefill_cases(n, seed):
    """Seeded random prefill shapes: 1..600 tokens, rows 1..3000, widths of
    64..4096 codes (odd multiples of 64 included where the group allows),
    2/3/4-bit codes, ranks 0..r_max, fp16/bf16 in, every dtype out."""
    g = np.random.default_rng(seed)
    cases = []
    while len(cases) < n:
        bits = int(g.choice([2, 3, 4]))
        G = int(g.choice([32, 64, 128, 256]))
        if G % (32 if bits == 3 else 128 // bits):
            continue
        step = max(G, 128 if bits == 3 else 64)
        d_in = int(step * g.integers(1, 4096 // step + 1))
        if d_in % G:
            continue
        M, d_out = int(g.integers(1, 601)), int(g.integers(1, 3001))
        r_max = int(g.choice([16, 64, 256]))
        rank = int(g.integers(0, r_max + 1))
        act = str(g.choice(["fp16", "bf16"]))
        out = [torch.float32, torch.float16, torch.bfloat16][int(g.integers(0, 3))]
        cases.append((bits, G, M, d_out, d_in, r_max, rank, act, out))
    return cases


@pytest.mark.parametrize("case", _random_prefill_cases(40, 2025), ids=lambda c: "b%d_g%d_M%d_%dx%d_r%d_%d_%s" % c[:8])
def test_prefill_random_shapes_against_the_oracle(case):
    """A seeded sweep of random prefill shapes against the oracle rounded to
    the output dtype, with the fp16 weight-tile rounding bound."""
    bits, G, M, d_out, d_in, r_max, rank, act, out = case
    w, (Q, s, z, A, B) = _layer(d_out, d_in, bits, G, r_max, (M * 13 + d_out * 7 + d_in + rank) % 100000)
    c = cl.LowRank(dev_f16(A), dev_f16(B), r_max, rank)
    x = wl.activation((M, d_in), 25, M, d_out, dtype=act)
    y = cl.linear_prefill(w, c, dev_u16(x.bits, torch.float16 if act == "fp16" else torch.bfloat16), out_dtype=out)
    ref = linear.forward_packed(Q, s, z, bits, G, A, B, rank, x.values)
    W_hat = quant.dequant_packed(Q, s, z, bits, G, d_in)
    assert_oracle(out_to_numpy(y), ref, out, extra=fp16_tile_bound(W_hat, x.values, A, B, rank))


def test_prefill_matches_decode():
    M, d_out, d_in = 16, 1024, 2048
    w, (Q, s, z, A, B) = _layer(d_out, d_in, 4, 128, 64, 99)
    c = cl.LowRank(dev_f16(A), dev_f16(B), 64, 64)
    xd = dev_u16(wl.activation((M, d_in), 22).bits, torch.float16)
    yp = cl.linear_prefill(w, c, xd, out_dtype=torch.float32)
    yd = cl.linear_decode(w, c, xd, out_dtype=torch.float32)
    assert rel_l2(out_to_numpy(yp), out_to_numpy(yd)) <= 5e-4


def test_prefill_deterministic():
    M, d_out, d_in = 512, 512, 1024
    w, (Q, s, z, A, B) = _layer(d_out, d_in, 4, 128, 32, 5)
    c = cl.LowRank(dev_f16(A), dev_f16(B), 32, 32)
    xd = dev_u16(wl.activation((M, d_in), 23).bits, torch.float16)
    assert torch.equal(cl.linear_prefill(w, c, xd, out_dtype=torch.float32),
                       cl.linear_prefill(w, c, xd, out_dtype=torch.float32))


@pytest.mark.parametrize("bits,G", [(4, 128), (4, 64), (4, 32), (2, 64), (3, 128), (3, 32)])
def test_prefill_small_weight_scales(bits, G):
    """Weights N(0, (5e-4)^2): group scales near 2^-12, below 2^-10 where
    s / 16 leaves the fp16 normal range.  The dequantized tile forms q - z
    exactly and rounds s (q - z) once, so the error stays at the fp16
    rounding bound whatever the scale; every output dtype."""
    M, d_out, d_in, rank = 200, 600, 1024, 40
    W = wl.weight((d_out, d_in), 24, bits, G, std=5e-4)
    Q, s, z = quant.quantize_pack(W, bits, G)
    assert float(np.median(s.astype(np.float64))) < 2.0 ** -10
    A, B = wl.standin_factors(d_out, d_in, 64, 24, bits, G, scale=5e-4)
    w = cl.QWeight(dev_u32(Q), dev_f16(s), dev_f16(z), d_out, d_in, bits, G)
    c = cl.LowRank(dev_f16(A), dev_f16(B), 64, rank)
    x = wl.activation((M, d_in), 24, bits, G)
    ref = linear.forward_packed(Q, s, z, bits, G, A, B, rank, x.values)
    bound = fp16_tile_bound(quant.dequant_packed(Q, s, z, bits, G, d_in), x.values, A, B, rank)
    for out in (torch.float32, torch.float16, torch.bfloat16):
        y = cl.linear_prefill(w, c, dev_u16(x.bits, torch.float16), out_dtype=out)
        assert_oracle(out_to_numpy(y), ref, out, extra=bound)


@pytest.mark.parametrize("rank", [96, 256])
def test_prefill_wide_ranks(rank):
    """Ranks 96 and 256 (r_max 256): three and eight 32-column tiles of the
    T = X A^T preparation and of the rank fold."""
    M, d_out, d_in = 150, 520, 1024
    w, (Q, s, z, A, B) = _layer(d_out, d_in, 4, 128, 256, 90 + rank)
    c = cl.LowRank(dev_f16(A), dev_f16(B), 256, rank)
    x = wl.activation((M, d_in), 25, rank)
    y = cl.linear_prefill(w, c, dev_u16(x.bits, torch.float16), out_dtype=torch.float32)
    ref = linear.forward_packed(Q, s, z, 4, 128, A, B, rank, x.values)
    W_hat = quant.dequant_packed(Q, s, z, 4, 128, d_in)
    assert_oracle(out_to_numpy(y), ref, extra=fp16_tile_bound(W_hat, x.values, A, B, rank))


@pytest.mark.parametrize("bits,G", [(4, 32), (4, 64), (2, 64)])
@pytest.mark.parametrize("d_in", [192, 320])
def test_prefill_half_k_step(bits, G, d_in):
    """d_in an odd multiple of 64 leaves half a 128-code K step at the end:
    its missing half reads in-bounds data met by zero scales."""
    M, d_out, rank = 70, 300, 24
    w, (Q, s, z, A, B) = _layer(d_out, d_in, bits, G, 32, 95 + d_in + bits + G)
    c = cl.LowRank(dev_f16(A), dev_f16(B), 32, rank)
    x = wl.activation((M, d_in), 26, d_in, G)
    y = cl.linear_prefill(w, c, dev_u16(x.bits, torch.float16), out_dtype=torch.float32)
    ref = linear.forward_packed(Q, s, z, bits, G, A, B, rank, x.values)
    W_hat = quant.dequant_packed(Q, s, z, bits, G, d_in)
    assert_oracle(out_to_numpy(y), ref, extra=fp16_tile_bound(W_hat, x.values, A, B, rank))
