"""cl_linear_decode against the fp64 oracle (Section 4.1 forward):
relative L2 <= 1e-3 for every output dtype, across tile-spanning and ragged
shapes, ranks, token counts, 2/4-bit codes and fp16/bf16 activations; sampled
rows at the Llama-8B decoder-layer sizes; bitwise determinism."""

import numpy as np
import pytest
import torch

from oracle import linear, quant
from paper_2605_05819_amd import cl, workloads as wl
from tests.helpers import (REL_L2_TOL, assert_oracle, dev_f16, dev_u16, dev_u32, oracle_layer, out_to_numpy,
                           rel_l2)

pytestmark = pytest.mark.gpu

OUT_DTYPES = [torch.float32, torch.float16, torch.bfloat16]


def _device_layer(Q, s, z, A, B, d_out, d_in, bits, G, r_max, rank):
    w = cl.QWeight(dev_u32(Q), dev_f16(s), dev_f16(z), d_out, d_in, bits, G)
    c = cl.LowRank(dev_f16(A), dev_f16(B), r_max, rank) if r_max else None
    return w, c


def _check(w, c, Q, s, z, A, B, rank, x, act_dtype, out_dtype, bits, G):
    xd = dev_u16(x.bits, act_dtype)
    y = cl.linear_decode(w, c, xd, out_dtype=out_dtype)
    torch.cuda.synchronize()
    ref = linear.forward_packed(Q, s, z, bits, G, A, B, rank, x.values)
    assert_oracle(out_to_numpy(y), ref, out_dtype)
    return y, ref


def _random_decode_cases(n, seed):
    """Seeded random shapes over the decode paths: rows 1..5000, widths up to
    8192 codes (at most 2^23 weights a case), 2/3/4-bit codes with every
    allowed group size up to 256, 1..40 tokens (dot2 and MFMA backbones),
    ranks 0..r_max, every dtype."""
    g = np.random.default_rng(seed)
    cases = []
    while len(cases) < n:
        bits = int(g.choice([2, 3, 4]))
        G = int(g.choice([32, 64, 128, 256]))
        if G % (32 if bits == 3 else 128 // bits):
            continue
        step = max(G, 128 if bits == 3 else G)
        d_in = int(step * g.integers(1, 8192 // step + 1))
        d_out = int(g.integers(1, 5001))
        if d_out * d_in > (8 << 20):              # keep the fp64 oracle to seconds
            continue
        T = int(g.choice([1, 2, 3, 4, 5, 9, 16, 17, 40]))
        r_max = int(g.choice([8, 32, 64, 256]))
        rank = int(g.integers(0, r_max + 1))
        act = str(g.choice(["fp16", "bf16"]))
        out = [torch.float32, torch.float16, torch.bfloat16][int(g.integers(0, 3))]
        cases.append((bits, G, d_out, d_in, T, r_max, rank, act, out))
    return cases


@pytest.mark.parametrize("case", _random_decode_cases(100, 2024), ids=lambda c: "b%d_g%d_%dx%d_T%d_r%d_%d_%s" % c[:8])
def test_random_shapes_against_the_oracle(case):
    """A seeded sweep of random shapes, token counts, ranks and dtypes; each
    output against the oracle rounded to its dtype."""
    bits, G, d_out, d_in, T, r_max, rank, act, out = case
    seed = (d_out * 7 + d_in * 3 + T * 11 + rank) % 100000
    W = wl.weight((d_out, d_in), 16, seed)
    Q, s, z = quant.quantize_pack(W, bits, G)
    A, B = wl.standin_factors(d_out, d_in, r_max, 16, seed)
    w, c = _device_layer(Q, s, z, A, B, d_out, d_in, bits, G, r_max, rank)
    x = wl.activation((T, d_in), 16, seed, dtype=act)
    _check(w, c, Q, s, z, A, B, rank, x, torch.float16 if act == "fp16" else torch.bfloat16, out, bits, G)


def _random_window_cases(n, seed):
    g = np.random.default_rng(seed)
    cases = []
    while len(cases) < n:
        bits = int(g.choice([2, 3, 4]))
        G = int(g.choice([32, 64, 128]))
        if G % (32 if bits == 3 else 128 // bits):
            continue
        step = max(G, 128 if bits == 3 else G)
        d_in = int(step * g.integers(1, 4096 // step + 1))
        nl = int(g.integers(2, 9))
        d_outs = [int(v) for v in g.integers(1, 2049, nl)]
        if sum(d_outs) * d_in > (8 << 20):
            continue
        T = int(g.choice([1, 2, 3, 5, 16, 20]))
        r_max = int(g.choice([8, 64, 256]))
        ranks = [int(v) for v in g.integers(0, r_max + 1, nl)]
        cases.append((bits, G, d_in, T, r_max, tuple(d_outs), tuple(ranks), str(g.choice(["fp16", "bf16"]))))
    return cases


@pytest.mark.parametrize("case", _random_window_cases(30, 2027),
                         ids=lambda c: "b%d_g%d_K%d_T%d_r%d_n%d" % (c[0], c[1], c[2], c[3], c[4], len(c[5])))
def test_random_windows_against_singles_and_the_oracle(case):
    """A seeded sweep of windows (2..8 linears over one input, random row
    counts and ranks): each output equals the single call bit for bit and
    the oracle within tolerance."""
    bits, G, d_in, T, r_max, d_outs, ranks, act = case
    ws_, cs, host = [], [], []
    for i, (d_out, rank) in enumerate(zip(d_outs, ranks)):
        w, c, h = _layer_dev(d_out, d_in, bits, G, r_max, rank, 200 + i + d_in % 97)
        ws_.append(w), cs.append(c), host.append(h)
    x = wl.activation((T, d_in), 17, d_in, T, dtype=act)
    xd = dev_u16(x.bits, torch.float16 if act == "fp16" else torch.bfloat16)
    ys = cl.linear_decode_window(ws_, cs, xd, out_dtype=torch.float32)
    for i, (w, c, (Q, s, z, A, B), rank) in enumerate(zip(ws_, cs, host, ranks)):
        assert torch.equal(ys[i], cl.linear_decode(w, c, xd, out_dtype=torch.float32)), i
        assert_oracle(out_to_numpy(ys[i]), linear.forward_packed(Q, s, z, bits, G, A, B, rank, x.values))


def test_single_linear_1024_rank16_all_out_dtypes():
    spec = wl.single_linear().linears[0]
    W = wl.weight((spec.d_out, spec.d_in), 0)
    Q, s, z, A, B, _ = oracle_layer(W, 4, 128, 16)
    w, c = _device_layer(Q, s, z, A, B, 1024, 1024, 4, 128, 16, 16)
    x = wl.activation((1, 1024), 0)
    for od in OUT_DTYPES:
        _check(w, c, Q, s, z, A, B, 16, x, torch.float16, od, 4, 128)


@pytest.mark.parametrize("bits,G", [(4, 128), (2, 64), (2, 128), (4, 32), (3, 128), (3, 32)])
@pytest.mark.parametrize("d_out,d_in", [(37, 256), (1000, 768), (4099, 1536)])
@pytest.mark.parametrize("T", [1, 3, 4, 5, 16])
def test_ragged_shapes_tokens_and_bits(bits, G, d_out, d_in, T):
    g = np.random.default_rng(d_out + d_in + T + bits)
    W = wl.weight((d_out, d_in), 7, d_out, d_in)
    Q, s, z = quant.quantize_pack(W, bits, G)
    r_max = 24
    rank = int(g.integers(0, r_max + 1))
    A, B = wl.standin_factors(d_out, d_in, r_max, 7, 0, d_out, d_in)
    w, c = _device_layer(Q, s, z, A, B, d_out, d_in, bits, G, r_max, rank)
    x = wl.activation((T, d_in), 7, 0, d_out, d_in)
    _check(w, c, Q, s, z, A, B, rank, x, torch.float16, torch.float32, bits, G)


@pytest.mark.parametrize("bits,G", [(4, 128), (2, 64)])
@pytest.mark.parametrize("d_in", [5120, 12416])
@pytest.mark.parametrize("T", [1, 2, 5])
def test_long_rows_split_preparation(bits, G, d_in, T):
    """Rows of A longer than 4096 are split over 2 (5120) or 4 (12416) waves
    in the preparation; the parts meet in LDS."""
    d_out, r_max, rank = 300, 48, 41
    W = wl.weight((d_out, d_in), 8, d_out, d_in)
    Q, s, z = quant.quantize_pack(W, bits, G)
    A, B = wl.standin_factors(d_out, d_in, r_max, 8, 0, d_out, d_in)
    w, c = _device_layer(Q, s, z, A, B, d_out, d_in, bits, G, r_max, rank)
    x = wl.activation((T, d_in), 8, 0, d_out, d_in)
    _check(w, c, Q, s, z, A, B, rank, x, torch.float16, torch.float32, bits, G)


@pytest.mark.parametrize("rank", [0, 1, 17, 64, 128, 256])
def test_ranks_including_zero_and_max(rank):
    d_out, d_in = 512, 1024
    W = wl.weight((d_out, d_in), 8, rank)
    Q, s, z = quant.quantize_pack(W, 4, 128)
    A, B = wl.standin_factors(d_out, d_in, 256, 8, rank)
    w, c = _device_layer(Q, s, z, A, B, d_out, d_in, 4, 128, 256, rank)
    x = wl.activation((2, d_in), 8, rank)
    _check(w, c, Q, s, z, A, B, rank, x, torch.float16, torch.float16, 4, 128)


def test_no_factors_equals_rank_zero():
    d_out, d_in = 300, 512
    W = wl.weight((d_out, d_in), 9)
    Q, s, z = quant.quantize_pack(W, 4, 128)
    A, B = wl.standin_factors(d_out, d_in, 8, 9)
    w, c = _device_layer(Q, s, z, A, B, d_out, d_in, 4, 128, 8, 0)
    x = dev_u16(wl.activation((1, d_in), 9).bits, torch.float16)
    y0 = cl.linear_decode(w, c, x, out_dtype=torch.float32)
    y1 = cl.linear_decode(w, None, x, out_dtype=torch.float32)
    assert torch.equal(y0, y1)


@pytest.mark.parametrize("bits,G", [(4, 128), (2, 64), (3, 128)])
def test_bf16_activations(bits, G):
    d_out, d_in = 777, 2048
    W = wl.weight((d_out, d_in), 10, bits)
    Q, s, z = quant.quantize_pack(W, bits, G)
    A, B = wl.standin_factors(d_out, d_in, 32, 10, bits)
    w, c = _device_layer(Q, s, z, A, B, d_out, d_in, bits, G, 32, 32)
    x = wl.activation((4, d_in), 10, bits, dtype="bf16")
    for od in OUT_DTYPES:
        _check(w, c, Q, s, z, A, B, 32, x, torch.bfloat16, od, bits, G)


def _bf16_out_of_fp16_range(T, d_in, seed):
    """bf16 activations outside fp16's normal range: even tokens at scale
    1e5 (most beyond 65504), odd tokens at scale 1e-6 (all below 2^-17 but a
    few, fp16 subnormals), and the fp16 values the kernels are documented to
    see: clamped to +-65504, then rounded to nearest even."""
    g = np.random.default_rng(seed)
    scale = np.where(np.arange(T) % 2 == 0, 1e5, 1e-6)[:, None]
    bits = wl.fp32_to_bf16_bits((scale * g.standard_normal((T, d_in))).astype(np.float32))
    seen = np.clip(wl.bf16_bits_to_f64(bits), -65504.0, 65504.0).astype(np.float16).astype(np.float64)
    return bits, seen


@pytest.mark.parametrize("bits,G", [(4, 128), (3, 128), (2, 64)])
@pytest.mark.parametrize("T", [2, 4])
def test_bf16_activations_beyond_the_fp16_range(bits, G, T):
    """The documented bf16 conversion on the dot2 (2 tokens) and MFMA (4
    tokens) backbones: saturated at +-65504, rounded to multiples of 2^-24
    below 2^-17.  Two tokens carry the rank term too (t = A x in float32, so
    it sees the same converted values); on the MFMA backbone t is an fp16
    pair whose range these scales leave (|A x| ~ 1e5 and ~ 1e-6), so that
    case runs the backbone alone.  Each token is checked on its own (the
    subnormal tokens' outputs are ~1e-6)."""
    d_out, d_in = 500, 1024
    rank = 24 if T < 3 else 0
    W = wl.weight((d_out, d_in), 14, bits, T)
    Q, s, z = quant.quantize_pack(W, bits, G)
    A, B = wl.standin_factors(d_out, d_in, 32, 14, bits, T)
    w, c = _device_layer(Q, s, z, A, B, d_out, d_in, bits, G, 32, rank)
    xb, seen = _bf16_out_of_fp16_range(T, d_in, 40 + T + bits)
    assert np.abs(seen[0]).max() == 65504.0 and np.abs(seen[1]).max() < 2.0 ** -14
    y = out_to_numpy(cl.linear_decode(w, c, dev_u16(xb, torch.bfloat16), out_dtype=torch.float32))
    ref = linear.forward_packed(Q, s, z, bits, G, A, B, rank, seen)
    for tk in range(T):
        assert_oracle(y[tk], ref[tk])


@pytest.mark.parametrize("mat", wl.LLAMA_MATS)
@pytest.mark.parametrize("T", [1, 4, 16])
def test_llama_layer_full_size_sampled_rows(mat, T):
    """Every Llama-8B layer linear at full size with its allocated rank; the
    backbone is quantized on the GPU and rows sampled over the whole output
    are checked against the oracle, which quantizes those rows itself."""
    layer = wl.llama_layer()
    spec = [l for l in layer.linears if l.name == mat][0]
    m = wl.LLAMA_MATS.index(mat)
    W = wl.weight((spec.d_out, spec.d_in), layer.index, 0, m)
    w = cl.quantize_pack(torch.from_numpy(W).cuda(), 4, 128)
    A, B = wl.standin_factors(spec.d_out, spec.d_in, spec.r_max, layer.index, 0, m)
    c = cl.LowRank(dev_f16(A), dev_f16(B), spec.r_max, spec.rank)
    x = wl.activation((T, spec.d_in), layer.index, 0, m)
    y = cl.linear_decode(w, c, dev_u16(x.bits, torch.float16), out_dtype=torch.float32)
    torch.cuda.synchronize()
    rows = np.r_[0:4, np.random.default_rng(m).choice(spec.d_out, 120, replace=False), spec.d_out - 4:spec.d_out]
    Q, s, z = quant.quantize_pack(W[rows], 4, 128)
    ref = linear.forward_packed(Q, s, z, 4, 128, A, B[rows], spec.rank, x.values)
    assert_oracle(out_to_numpy(y)[:, rows], ref)


@pytest.mark.parametrize("mat", wl.LLAMA_MATS)
@pytest.mark.parametrize("T", [1, 4, 16])
def test_llama_layer_3bit_full_size_sampled_rows(mat, T):
    """The paper's INT3 setting: every Llama-8B layer linear with 3-bit codes
    (group 128) at full size, quantized on the GPU, with its allocated rank;
    sampled rows against the oracle, which quantizes those rows itself."""
    layer = wl.llama_layer_3bit()
    spec = [l for l in layer.linears if l.name == mat][0]
    m = wl.LLAMA_MATS.index(mat)
    W = wl.weight((spec.d_out, spec.d_in), layer.index, 0, m)
    w = cl.quantize_pack(torch.from_numpy(W).cuda(), 3, 128)
    A, B = wl.standin_factors(spec.d_out, spec.d_in, spec.r_max, layer.index, 0, m)
    c = cl.LowRank(dev_f16(A), dev_f16(B), spec.r_max, spec.rank)
    x = wl.activation((T, spec.d_in), layer.index, 0, m)
    for od in (torch.float32, torch.float16):
        y = cl.linear_decode(w, c, dev_u16(x.bits, torch.float16), out_dtype=od)
        torch.cuda.synchronize()
        rows = np.r_[0:4, np.random.default_rng(m).choice(spec.d_out, 120, replace=False), spec.d_out - 4:spec.d_out]
        Q, s, z = quant.quantize_pack(W[rows], 3, 128)
        ref = linear.forward_packed(Q, s, z, 3, 128, A, B[rows], spec.rank, x.values)
        assert_oracle(out_to_numpy(y)[:, rows], ref, od)


@pytest.mark.parametrize("mat", wl.LLAMA_MATS)
@pytest.mark.parametrize("T", [4, 16])
def test_llama_layer_2bit_many_tokens_full_size_sampled_rows(mat, T):
    """Every Llama-8B layer linear with 2-bit codes (group 64) at full size,
    quantized on the GPU, with its allocated rank, at 4 and 16 tokens (the
    MFMA backbone with two quantization groups per 128-code block); sampled
    rows against the oracle, which quantizes those rows itself."""
    layer = wl.llama_layer_2bit()
    spec = [l for l in layer.linears if l.name == mat][0]
    m = wl.LLAMA_MATS.index(mat)
    W = wl.weight((spec.d_out, spec.d_in), layer.index, 0, m)
    w = cl.quantize_pack(torch.from_numpy(W).cuda(), 2, 64)
    A, B = wl.standin_factors(spec.d_out, spec.d_in, spec.r_max, layer.index, 0, m)
    c = cl.LowRank(dev_f16(A), dev_f16(B), spec.r_max, spec.rank)
    x = wl.activation((T, spec.d_in), layer.index, 0, m)
    y = cl.linear_decode(w, c, dev_u16(x.bits, torch.float16), out_dtype=torch.float32)
    torch.cuda.synchronize()
    rows = np.r_[0:4, np.random.default_rng(m).choice(spec.d_out, 120, replace=False), spec.d_out - 4:spec.d_out]
    Q, s, z = quant.quantize_pack(W[rows], 2, 64)
    ref = linear.forward_packed(Q, s, z, 2, 64, A, B[rows], spec.rank, x.values)
    assert_oracle(out_to_numpy(y)[:, rows], ref)


@pytest.mark.parametrize("T", [9, 16, 40])
def test_gate_up_window_many_tokens_sampled_rows(T):
    """The gate and up projections as one window (1792 row tiles: the MFMA
    backbone's four-tiles-per-wave form) for 9, 16 and 40 tokens (one to
    three passes of 16): equal to the single calls (one tile per wave) bit
    for bit, and to the oracle on sampled rows."""
    layer = wl.llama_layer()
    ws_, cs, host = [], [], []
    for m in (4, 5):
        spec = layer.linears[m]
        W = wl.weight((spec.d_out, spec.d_in), layer.index, 0, m)
        ws_.append(cl.quantize_pack(torch.from_numpy(W).cuda(), 4, 128))
        A, B = wl.standin_factors(spec.d_out, spec.d_in, spec.r_max, layer.index, 0, m)
        cs.append(cl.LowRank(dev_f16(A), dev_f16(B), spec.r_max, spec.rank))
        host.append((W, A, B, spec.rank))
    x = wl.activation((T, 4096), layer.index, 0, 4)
    xd = dev_u16(x.bits, torch.float16)
    ys = cl.linear_decode_window(ws_, cs, xd, out_dtype=torch.float32)
    for i, (W, A, B, rank) in enumerate(host):
        y1 = cl.linear_decode(ws_[i], cs[i], xd, out_dtype=torch.float32)
        assert torch.equal(ys[i], y1), i
        rows = np.r_[0:4, np.random.default_rng(70 + i).choice(14336, 60, replace=False), 14332:14336]
        Q, s, z = quant.quantize_pack(W[rows], 4, 128)
        ref = linear.forward_packed(Q, s, z, 4, 128, A, B[rows], rank, x.values)
        assert_oracle(out_to_numpy(ys[i])[:, rows], ref)


def test_2bit_gate_rank_sweep_sampled_rows():
    layer = wl.llama_layer_2bit()
    W = wl.weight((14336, 4096), layer.index, 0, 4)
    w = cl.quantize_pack(torch.from_numpy(W).cuda(), 2, 64)
    A, B = wl.standin_factors(14336, 4096, 256, layer.index, 0, 4)
    x = wl.activation((1, 4096), layer.index, 0, 4)
    rows = np.random.default_rng(5).choice(14336, 100, replace=False)
    Q, s, z = quant.quantize_pack(W[rows], 2, 64)
    for rank in (0, 32, 128, 256):
        c = cl.LowRank(dev_f16(A), dev_f16(B), 256, rank)
        y = cl.linear_decode(w, c, dev_u16(x.bits, torch.float16), out_dtype=torch.float32)
        torch.cuda.synchronize()
        ref = linear.forward_packed(Q, s, z, 2, 64, A, B[rows], rank, x.values)
        assert_oracle(out_to_numpy(y)[:, rows], ref)


@pytest.mark.parametrize("bits,G,T", [(4, 128, 4), (4, 128, 1), (2, 64, 16), (3, 128, 16), (3, 32, 2)])
def test_deterministic_bitwise(bits, G, T):
    """Two calls on the same inputs give the same bits (every backbone: the
    K slices and waves' partial sums meet in a fixed order)."""
    d_out, d_in = 4096, 4096
    W = wl.weight((d_out, d_in), 11)
    w = cl.quantize_pack(torch.from_numpy(W).cuda(), bits, G)
    A, B = wl.standin_factors(d_out, d_in, 64, 11)
    c = cl.LowRank(dev_f16(A), dev_f16(B), 64, 64)
    x = dev_u16(wl.activation((T, d_in), 11).bits, torch.float16)
    y1 = cl.linear_decode(w, c, x, out_dtype=torch.float32)
    y2 = cl.linear_decode(w, c, x, out_dtype=torch.float32)
    assert torch.equal(y1, y2)


def _layer_dev(d_out, d_in, bits, G, r_max, rank, seed):
    W = wl.weight((d_out, d_in), 12, seed)
    Q, s, z = quant.quantize_pack(W, bits, G)
    A, B = wl.standin_factors(d_out, d_in, r_max, 12, seed)
    w, c = _device_layer(Q, s, z, A, B, d_out, d_in, bits, G, r_max, rank)
    return w, c, (Q, s, z, A, B)


@pytest.mark.parametrize("bits,G,d_in", [(4, 32, 192), (4, 64, 320), (2, 64, 192), (2, 64, 320), (4, 32, 384),
                                          (3, 32, 384), (3, 64, 384)])
@pytest.mark.parametrize("T", [3, 16])
def test_mfma_rows_ending_in_a_partial_block(bits, G, d_in, T):
    """Rows whose width is not a multiple of the 128-code block (2- and
    4-bit: an odd multiple of 64 codes) on the MFMA backbone: the last
    block's missing groups have clamped loads and a zero scale; 3-bit rows
    (multiples of 128 codes) with two and four groups per block; every
    output dtype."""
    w, c, (Q, s, z, A, B) = _layer_dev(300, d_in, bits, G, 64, 37, d_in + bits + T)
    x = wl.activation((T, d_in), 12, d_in, T)
    for od in OUT_DTYPES:
        _check(w, c, Q, s, z, A, B, 37, x, torch.float16, od, bits, G)


def test_one_workspace_reused_across_shapes_ranks_and_token_counts():
    """One workspace serves consecutive calls of different shapes, ranks and
    token counts."""
    cases = [(4096, 4096, 64, 1), (37, 512, 8, 3), (14336, 4096, 128, 4), (5, 256, 256, 2),
             (4096, 14336, 32, 1), (4096, 4096, 64, 5)]
    ws = cl.workspace(1 << 20, "cuda")
    for i, (d_out, d_in, rank, T) in enumerate(cases):
        w, c, (Q, s, z, A, B) = _layer_dev(d_out, d_in, 4, 128, 256, rank, i)
        x = wl.activation((T, d_in), 12, i)
        y = cl.linear_decode(w, c, dev_u16(x.bits, torch.float16), out_dtype=torch.float32, ws=ws)
        rows = np.arange(d_out) if d_out < 512 else np.random.default_rng(i).choice(d_out, 256, replace=False)
        ref = linear.forward_rows(Q, s, z, 4, 128, A, B, rank, x.values, rows)
        assert_oracle(out_to_numpy(y)[:, rows], ref)


def test_few_rows_many_factor_rows():
    """Three output rows against 256 factor rows."""
    w, c, (Q, s, z, A, B) = _layer_dev(3, 4096, 4, 128, 256, 256, 40)
    x = wl.activation((2, 4096), 12, 40)
    y = cl.linear_decode(w, c, dev_u16(x.bits, torch.float16), out_dtype=torch.float32)
    ref = linear.forward_packed(Q, s, z, 4, 128, A, B, 256, x.values)
    assert_oracle(out_to_numpy(y), ref)


@pytest.mark.parametrize("bits,G", [(4, 128), (2, 64), (3, 128)])
def test_wide_input_uses_eight_k_slices(bits, G):
    """d_in = 20480 (4-bit: 640 chunks of 32 codes) splits K over 8 waves."""
    d_out, d_in = 300, 20480
    w, c, (Q, s, z, A, B) = _layer_dev(d_out, d_in, bits, G, 32, 32, 41 + bits)
    x = wl.activation((1, d_in), 12, 41 + bits)
    y = cl.linear_decode(w, c, dev_u16(x.bits, torch.float16), out_dtype=torch.float32)
    ref = linear.forward_packed(Q, s, z, bits, G, A, B, 32, x.values)
    assert_oracle(out_to_numpy(y), ref)


@pytest.mark.parametrize("T,act", [(1, "fp16"), (4, "bf16"), (16, "fp16")])
def test_window_matches_single_calls_bitwise_and_oracle(T, act):
    """A Q/K/V-shaped window (4096/1024/1024 x 2048, ranks 64/0/17) equals the
    three single calls bit for bit, and the oracle within tolerance."""
    dt = torch.float16 if act == "fp16" else torch.bfloat16
    shapes, ranks = [(4096, 2048), (1024, 2048), (1024, 2048)], [64, 0, 17]
    ws_, cs, host = [], [], []
    for i, ((d_out, d_in), rank) in enumerate(zip(shapes, ranks)):
        w, c, h = _layer_dev(d_out, d_in, 4, 128, 64, rank, 60 + i)
        ws_.append(w); cs.append(c); host.append(h)
    x = wl.activation((T, 2048), 12, 60, dtype=act)
    xd = dev_u16(x.bits, dt)
    ys = cl.linear_decode_window(ws_, cs, xd, out_dtype=torch.float32)
    for i, (w, c, (Q, s, z, A, B), rank) in enumerate(zip(ws_, cs, host, ranks)):
        y1 = cl.linear_decode(w, c, xd, out_dtype=torch.float32)
        assert torch.equal(ys[i], y1), i
        rows = np.random.default_rng(i).choice(w.d_out, 200, replace=False)
        ref = linear.forward_rows(Q, s, z, 4, 128, A, B, rank, x.values, rows)
        assert_oracle(out_to_numpy(ys[i])[:, rows], ref)


def test_window_without_factors_and_two_bit():
    ws_, host = [], []
    for i in range(2):
        W = wl.weight((700 + 100 * i, 1024), 13, i)
        Q, s, z = quant.quantize_pack(W, 2, 64)
        ws_.append(cl.QWeight(dev_u32(Q), dev_f16(s), dev_f16(z), W.shape[0], 1024, 2, 64))
        host.append((Q, s, z))
    x = wl.activation((3, 1024), 13, 9)
    ys = cl.linear_decode_window(ws_, None, dev_u16(x.bits, torch.float16), out_dtype=torch.float32)
    for y, (Q, s, z) in zip(ys, host):
        ref = linear.forward_packed(Q, s, z, 2, 64, None, None, 0, x.values)
        assert_oracle(out_to_numpy(y), ref)


def _glu_pair(d_out, d_in, bits, G, ranks, seed):
    pair = [_layer_dev(d_out, d_in, bits, G, 64, r, seed + i) for i, r in enumerate(ranks)]
    return [p[0] for p in pair], [p[1] for p in pair], [p[2] for p in pair]


def _glu_ref_rows(host, ranks, bits, G, d_in, X, rows):
    """Oracle SiLU(gate x) * (up x) on a row sample (each output element
    depends only on its own rows of the backbone and of B)."""
    mats = []
    for (Q, s, z, A, B), r in zip(host, ranks):
        W_hat = quant.dequant_packed(Q[rows], s[rows], z[rows], bits, G, d_in)
        mats.append((W_hat, A, B[rows], r))
    return linear.forward_glu(mats[0], mats[1], X)


@pytest.mark.parametrize("T,act,out,bits,G,d_out,d_in", [
    (1, torch.float16, torch.float16, 4, 128, 1000, 2048),      # one token per pass, one K slice
    (2, torch.bfloat16, torch.float32, 4, 128, 1000, 4096),     # two tokens per pass (prefetch), 2 K slices
    (3, torch.float16, torch.bfloat16, 4, 128, 1000, 2048),     # MFMA backbone, ragged last tile
    (5, torch.float16, torch.float16, 2, 64, 700, 1024),        # 2-bit, MFMA, two groups per block
    (1, torch.float16, torch.float32, 4, 128, 14336, 4096),     # Llama-8B gate/up, one token
    (16, torch.float16, torch.float32, 4, 128, 14336, 4096),    # Llama-8B gate/up, MFMA with 4 tiles per wave
    (64, torch.bfloat16, torch.float16, 4, 128, 1000, 2048),    # the most tokens: four MFMA passes
    (4, torch.float16, torch.bfloat16, 2, 64, 1000, 4096),      # 2-bit, MFMA, one tile per wave
    (2, torch.float16, torch.float16, 2, 64, 1000, 4096),       # 2-bit, two tokens per pass (dot2)
    (16, torch.float16, torch.float32, 2, 64, 14336, 4096),     # 2-bit Llama-8B gate/up, MFMA, 4 tiles per wave
    (1, torch.float16, torch.bfloat16, 3, 128, 1000, 2048),     # 3-bit, one token
    (6, torch.bfloat16, torch.float16, 3, 32, 700, 1024),       # 3-bit, MFMA, four groups per block
    (2, torch.bfloat16, torch.float16, 3, 64, 700, 1024),       # 3-bit, two tokens per pass (dot2)
    (16, torch.float16, torch.float32, 3, 128, 14336, 4096),    # 3-bit Llama-8B gate/up, MFMA, 4 tiles per wave
])
def test_glu_matches_oracle(T, act, out, bits, G, d_out, d_in):
    """cl_linear_decode_glu = SiLU(gate x) * (up x) of the fp64 oracle (gate
    rank 64, up rank 17), every output dtype against the oracle rounded to
    it; the fp16/bf16 result is also the round-to-nearest-even of the fp32
    result, bit for bit."""
    ranks = (64, 17)
    ws_, cs, host = _glu_pair(d_out, d_in, bits, G, ranks, 70 + T)
    x = wl.activation((T, d_in), 12, 70, dtype="fp16" if act == torch.float16 else "bf16")
    xd = dev_u16(x.bits, act)
    h32 = cl.linear_decode_glu(ws_, cs, xd, out_dtype=torch.float32)
    rows = np.arange(d_out) if d_out <= 1000 else np.random.default_rng(T).choice(d_out, 300, replace=False)
    ref = _glu_ref_rows(host, ranks, bits, G, d_in, x.values, rows)
    assert_oracle(out_to_numpy(h32)[:, rows], ref)
    if out != torch.float32:
        h = cl.linear_decode_glu(ws_, cs, xd, out_dtype=out)
        assert_oracle(out_to_numpy(h)[:, rows], ref, out)
        assert torch.equal(h, h32.to(out))


@pytest.mark.parametrize("T", [1, 2, 16])
def test_glu_is_the_window_with_its_epilogue(T):
    """The fused epilogue sees the same fp32 gate and up values as the window
    call writes: SiLU(y_gate) * y_up from the window's fp32 outputs matches to
    fp32 rounding; two calls agree bit for bit."""
    ws_, cs, _ = _glu_pair(1536, 2048, 4, 128, (32, 0), 80)
    x = wl.activation((T, 2048), 12, 80)
    xd = dev_u16(x.bits, torch.float16)
    yg, yu = cl.linear_decode_window(ws_, cs, xd, out_dtype=torch.float32)
    want = torch.nn.functional.silu(yg) * yu
    h = cl.linear_decode_glu(ws_, cs, xd, out_dtype=torch.float32)
    torch.testing.assert_close(h, want, rtol=1e-5, atol=1e-6)
    assert torch.equal(cl.linear_decode_glu(ws_, cs, xd, out_dtype=torch.float32), h)


def test_glu_without_factors():
    ws_, _, host = _glu_pair(512, 1024, 4, 128, (0, 0), 90)
    x = wl.activation((1, 1024), 12, 90)
    h = cl.linear_decode_glu(ws_, None, dev_u16(x.bits, torch.float16), out_dtype=torch.float32)
    ref = _glu_ref_rows(host, (0, 0), 4, 128, 1024, x.values, np.arange(512))
    assert_oracle(out_to_numpy(h), ref)


# ------------------------------------------- small quantization scales


@pytest.mark.parametrize("T", [1, 3, 16])
@pytest.mark.parametrize("bits,G", [(4, 128), (4, 64), (4, 32), (2, 64), (3, 128)])
@pytest.mark.parametrize("std", [5e-4, 1e-4])
def test_small_weight_scales(T, bits, G, std):
    """Weights N(0, std^2) with std 5e-4 and 1e-4 put the group scales at
    about 2^-12 and 2^-15, below 2^-10 where s / 16 leaves the fp16 normal
    range: the backbone must not depend on the scale's magnitude.  One token
    runs the dot2 backbone, 3 and 16 tokens the MFMA backbone (one, two or
    four quantization groups per 128-code block); every output dtype against
    the oracle rounded to it, plus the elementwise bound."""
    d_out, d_in, r_max, rank = 1000, 2048, 32, 24
    W = wl.weight((d_out, d_in), 14, T, bits + G, std=std)
    Q, s, z = quant.quantize_pack(W, bits, G)
    assert float(np.median(s.astype(np.float64))) < 2.0 ** -10
    A, B = wl.standin_factors(d_out, d_in, r_max, 14, T, bits + G, scale=std)
    w, c = _device_layer(Q, s, z, A, B, d_out, d_in, bits, G, r_max, rank)
    x = wl.activation((T, d_in), 14, T, bits + G)
    for od in OUT_DTYPES:
        _check(w, c, Q, s, z, A, B, rank, x, torch.float16, od, bits, G)


@pytest.mark.parametrize("T", [3, 16])
def test_small_weight_scales_glu(T):
    """The gated call on the MFMA backbone with std 5e-4 weights: h in bf16
    against the rounded oracle."""
    d_out, d_in, bits, G = 1000, 2048, 4, 128
    ranks = (16, 8)
    ws_, cs, host = [], [], []
    for i, rank in enumerate(ranks):
        W = wl.weight((d_out, d_in), 15, T, i, std=5e-4)
        Q, s, z = quant.quantize_pack(W, bits, G)
        A, B = wl.standin_factors(d_out, d_in, 16, 15, T, i, scale=5e-4)
        w, c = _device_layer(Q, s, z, A, B, d_out, d_in, bits, G, 16, rank)
        ws_.append(w), cs.append(c), host.append((Q, s, z, A, B))
    x = wl.activation((T, d_in), 15, T)
    ref = _glu_ref_rows(host, ranks, bits, G, d_in, x.values, np.arange(d_out))
    for od in OUT_DTYPES:
        h = cl.linear_decode_glu(ws_, cs, dev_u16(x.bits, torch.float16), out_dtype=od)
        assert_oracle(out_to_numpy(h), ref, od)


def test_single_element_error_is_caught():
    """The elementwise bound rejects one wrong element that the relative L2
    bar alone lets through (a 10 % error on one of 65536 outputs)."""
    from tests.helpers import elem_ratio
    g = np.random.default_rng(0)
    ref = g.standard_normal((4, 16384))
    got = ref.copy()
    got[2, 777] *= 1.1
    assert rel_l2(got, ref) <= REL_L2_TOL
    assert elem_ratio(got, ref) > 1.0
