"""cl_moe_linear_decode against the fp64 oracle (Section 4.2.2 and
Appendix A.1: every routed expert's same projection in one step, only routed
experts read).  Full outputs at sizes the oracle finishes in seconds (oracle
quantizer, SVD factors, ragged rows, duplicate and invalid ids, rank 0 and
clamped ranks, 2/4-bit, fp16/bf16 activations, every output dtype); sampled
rows at the 128-expert, hidden-2048 / FFN-768 layer with top-8 routing for
1, 8 and 64 tokens; bitwise determinism and workspace reuse."""

import numpy as np
import pytest
import torch

from oracle import linear, moe, quant
from paper_2605_05819_amd import cl, workloads as wl
from tests.helpers import REL_L2_TOL, assert_oracle, dev_f16, dev_u16, dev_u32, oracle_layer, out_to_numpy, rel_l2

pytestmark = pytest.mark.gpu

OUT_DTYPES = [torch.float32, torch.float16, torch.bfloat16]


def _stack(arrs):
    return np.ascontiguousarray(np.stack(arrs))


def _device_experts(Q, s, z, A, B, ranks, d_out, d_in, bits, G, r_max):
    """Stacked host arrays [E][...] -> cl.MoeExperts on the device."""
    return cl.MoeExperts(dev_u32(Q), dev_f16(s), dev_f16(z),
                         dev_f16(A) if r_max else None, dev_f16(B) if r_max else None,
                         torch.from_numpy(np.asarray(ranks, dtype=np.int32)).cuda() if r_max else None,
                         len(Q), d_out, d_in, bits, G, r_max)


def _oracle_experts(E, d_out, d_in, bits, G, r_max, seed, svd=True, std=0.02):
    """E experts quantized by the oracle; factors from the SVD of the error
    (or seeded stand-ins of the weights' scale)."""
    Qs, ss, zs, As, Bs = [], [], [], [], []
    for e in range(E):
        W = wl.weight((d_out, d_in), seed, 0, 0, e, std=std)
        if svd:
            Q, s, z, A, B, _ = oracle_layer(W, bits, G, r_max)
        else:
            Q, s, z = quant.quantize_pack(W, bits, G)
            A, B = wl.standin_factors(d_out, d_in, r_max, seed, 0, 0, e, scale=2.5 * std)
        Qs.append(Q), ss.append(s), zs.append(z), As.append(A), Bs.append(B)
    return _stack(Qs), _stack(ss), _stack(zs), _stack(As), _stack(Bs)


def _full_ref(Q, s, z, A, B, ranks, X, ids, x_per_slot, bits, G, d_in):
    """The oracle over all rows; out-of-range ids give zero rows."""
    E = len(Q)
    ids = np.asarray(ids)
    experts = [(quant.dequant_packed(Q[e], s[e], z[e], bits, G, d_in), A[e], B[e]) for e in range(E)]
    valid = (ids >= 0) & (ids < E)
    safe = np.where(valid, ids, 0)
    Y = moe.forward(experts, ranks, X, safe, x_per_slot)
    Y[~valid] = 0.0
    return Y


def _run(ex, X_bits, act, ids, out_dtype, x_per_slot):
    x = dev_u16(X_bits, act)
    idd = torch.from_numpy(np.ascontiguousarray(ids, dtype=np.int32)).cuda()
    y = cl.moe_linear_decode(ex, x, idd, out_dtype=out_dtype)
    torch.cuda.synchronize()
    assert tuple(y.shape) == (ids.shape[0], ids.shape[1], ex.d_out)
    return out_to_numpy(y)


@pytest.mark.parametrize("x_per_slot", [False, True])
@pytest.mark.parametrize("T,k", [(1, 4), (5, 3), (16, 8)])
def test_small_experts_svd_factors_full_outputs(T, k, x_per_slot):
    E, d_out, d_in, bits, G, r_max = 12, 100, 512, 4, 128, 16
    Q, s, z, A, B = _oracle_experts(E, d_out, d_in, bits, G, r_max, 40)
    ranks = wl.moe_expert_ranks(40, 0, 0, E, levels=(0, 4, 8, 16))
    ids, _ = wl.routing(T, 40, 0, E, k)
    shape = (T, k, d_in) if x_per_slot else (T, d_in)
    x = wl.activation(shape, 40, 0, 1)
    ex = _device_experts(Q, s, z, A, B, ranks, d_out, d_in, bits, G, r_max)
    ref = _full_ref(Q, s, z, A, B, ranks, x.values, ids, x_per_slot, bits, G, d_in)
    for od in OUT_DTYPES:
        got = _run(ex, x.bits, torch.float16, ids, od, x_per_slot)
        assert_oracle(got, ref, od)


@pytest.mark.parametrize("bits,G", [(2, 64), (4, 32)])
@pytest.mark.parametrize("act", [torch.float16, torch.bfloat16])
def test_bits_groups_and_bf16_activations(bits, G, act):
    E, d_out, d_in, r_max, T, k = 9, 37, 1536, 24, 6, 4
    Q, s, z, A, B = _oracle_experts(E, d_out, d_in, bits, G, r_max, 41, svd=False)
    ranks = np.array([0, 24, 8, 17, 24, 1, 0, 12, 5], dtype=np.int32)
    ids, _ = wl.routing(T, 41, 0, E, k)
    x = wl.activation((T, d_in), 41, 0, 1, dtype="bf16" if act == torch.bfloat16 else "fp16")
    ex = _device_experts(Q, s, z, A, B, ranks, d_out, d_in, bits, G, r_max)
    ref = _full_ref(Q, s, z, A, B, ranks, x.values, ids, False, bits, G, d_in)
    got = _run(ex, x.bits, act, ids, torch.float32, False)
    assert_oracle(got, ref)


def _random_moe_cases(n, seed):
    """Seeded random MoE calls: 1..160 experts, top-1..8 (ids drawn
    independently, so a token may repeat an expert), 1..64 tokens (the
    one-launch, VALU and MFMA paths by slots per expert), 2/4-bit codes with
    every group size to 256, widths to 4096, factor widths 0..64, ranks
    0..r_max per expert, shared or per-slot inputs, every dtype; at most
    2^24 expert weights a case."""
    g = np.random.default_rng(seed)
    cases = []
    while len(cases) < n:
        bits = int(g.choice([2, 4]))
        G = int(g.choice([32, 64, 128, 256]))
        if G % (128 // bits):
            continue
        d_in = int(G * g.integers(1, 4096 // G + 1))
        E = int(g.integers(1, 161))
        d_out = int(g.integers(1, 801))
        if E * d_out * d_in > (1 << 24):
            continue
        k = int(g.integers(1, min(8, E) + 1))
        T = int(g.choice([1, 2, 5, 8, 16, 33, 64]))
        r_max = int(g.choice([0, 8, 32, 64]))
        cases.append((bits, G, E, k, T, d_out, d_in, r_max, bool(g.integers(0, 2)),
                      str(g.choice(["fp16", "bf16"])), int(g.integers(0, 3)), int(g.integers(0, 1 << 30))))
    return cases


@pytest.mark.parametrize("case", _random_moe_cases(80, 2026),
                         ids=lambda c: "b%d_g%d_E%d_k%d_T%d_%dx%d_r%d_%s" % c[:9])
def test_random_moe_calls_against_the_oracle(case):
    """A seeded sweep of random MoE calls, each against the oracle rounded to
    its output dtype."""
    bits, G, E, k, T, d_out, d_in, r_max, per_slot, act, od, seed = case
    Q, s, z, A, B = _oracle_experts(E, d_out, d_in, bits, G, max(r_max, 1), seed % 1000, svd=False)
    g = np.random.default_rng(seed)
    ranks = g.integers(0, r_max + 1, E).astype(np.int32)
    ids = g.integers(0, E, (T, k)).astype(np.int32)
    shape = (T, k, d_in) if per_slot else (T, d_in)
    x = wl.activation(shape, seed % 1000, 1, 1, dtype=act)
    if r_max == 0:
        A, B = A[:, :0], B[:, :, :0]
    ex = _device_experts(Q, s, z, A, B, ranks, d_out, d_in, bits, G, r_max)
    ref = _full_ref(Q, s, z, A, B, ranks, x.values, ids, per_slot, bits, G, d_in)
    out = OUT_DTYPES[od]
    got = _run(ex, x.bits, torch.float16 if act == "fp16" else torch.bfloat16, ids, out, per_slot)
    assert_oracle(got, ref, out)


def test_duplicate_invalid_ids_and_clamped_ranks():
    E, d_out, d_in, bits, G, r_max, T, k = 6, 64, 256, 4, 128, 8, 4, 5
    Q, s, z, A, B = _oracle_experts(E, d_out, d_in, bits, G, r_max, 42, svd=False)
    ranks = np.array([-3, 8, 100, 0, 5, 2], dtype=np.int32)       # clamped to 0..r_max
    ids = np.array([[2, 2, 2, -1, 0],
                    [6, 1, 99, 5, 5],
                    [3, 3, 3, 3, 3],
                    [-7, 4, 1, 0, 2]], dtype=np.int32)
    x = wl.activation((T, d_in), 42, 0, 1)
    ex = _device_experts(Q, s, z, A, B, ranks, d_out, d_in, bits, G, r_max)
    got = _run(ex, x.bits, torch.float16, ids, torch.float32, False)
    ref = _full_ref(Q, s, z, A, B, np.clip(ranks, 0, r_max), x.values, ids, False, bits, G, d_in)
    invalid = (ids < 0) | (ids >= E)
    assert (got[invalid] == 0).all()
    assert_oracle(got, ref)
    # all slots invalid: zeros only
    bad = np.full((2, 3), E, dtype=np.int32)
    assert (_run(ex, x.bits[:2], torch.float16, bad, torch.float16, False) == 0).all()


@pytest.mark.parametrize("x_per_slot", [False, True])
def test_expert_with_more_than_64_slots_without_hoist(x_per_slot):
    """200 slots over 128 experts keep the per-slot unpack (slots < 2 x active
    experts); one expert takes 70 of them, so its slot ids are re-read into the
    lanes after the first 64."""
    E, d_out, d_in, bits, G, r_max, T, k = 128, 64, 256, 4, 128, 8, 25, 8
    Q, s, z, A, B = _oracle_experts(E, d_out, d_in, bits, G, r_max, 44, svd=False)
    ranks = wl.moe_expert_ranks(44, 0, 0, E, levels=(0, 4, 8))
    g = np.random.default_rng(44)
    flat = g.integers(0, E, T * k).astype(np.int32)
    flat[g.permutation(T * k)[:70]] = 7
    ids = flat.reshape(T, k)
    x = wl.activation((T, k, d_in) if x_per_slot else (T, d_in), 44, 0, 1)
    ex = _device_experts(Q, s, z, A, B, ranks, d_out, d_in, bits, G, r_max)
    got = _run(ex, x.bits, torch.float16, ids, torch.float32, x_per_slot)
    ref = _full_ref(Q, s, z, A, B, ranks, x.values, ids, x_per_slot, bits, G, d_in)
    assert_oracle(got, ref)
    assert_oracle(got[ids == 7], ref[ids == 7])


def test_rank_zero_without_factors():
    E, d_out, d_in, bits, G, T, k = 5, 70, 384, 4, 128, 3, 2
    Q, s, z, A, B = _oracle_experts(E, d_out, d_in, bits, G, 4, 43, svd=False)
    ex = _device_experts(Q, s, z, None, None, None, d_out, d_in, bits, G, 0)
    ids, _ = wl.routing(T, 43, 0, E, k)
    x = wl.activation((T, k, d_in), 43, 0, 1)
    got = _run(ex, x.bits, torch.float16, ids, torch.float32, True)
    ref = _full_ref(Q, s, z, A, B, np.zeros(E, dtype=np.int32), x.values, ids, True, bits, G, d_in)
    assert_oracle(got, ref)


# ---------------------------------------------- the 128-expert MoE layer


@pytest.fixture(scope="module")
def moe_layer():
    """gate and down of one layer: 128 stacked experts of stand-in codes and
    factors, per-expert ranks from {0, 8, 16, 32}."""
    out = {}
    for m, name in ((0, "gate"), (2, "down")):
        d_out, d_in = wl.MOE_SHAPES[name]
        Q, s, z = wl.standin_codes(wl.MOE_EXPERTS, d_out, d_in, 4, 128, 44, 0, m)
        A = np.empty((wl.MOE_EXPERTS, 32, d_in), np.float16)
        B = np.empty((wl.MOE_EXPERTS, d_out, 32), np.float16)
        for e in range(wl.MOE_EXPERTS):
            A[e], B[e] = wl.standin_factors(d_out, d_in, 32, 44, 0, m, e)
        ranks = wl.moe_expert_ranks(44, 0, m)
        ex = _device_experts(Q, s, z, A, B, ranks, d_out, d_in, 4, 128, 32)
        out[name] = (ex, Q, s, z, A, B, ranks)
    return out


@pytest.mark.parametrize("name", ["gate", "down"])
@pytest.mark.parametrize("T", [1, 8, 64])
def test_layer_sampled_rows(moe_layer, name, T):
    ex, Q, s, z, A, B, ranks = moe_layer[name]
    x_per_slot = name == "down"
    ids, _ = wl.routing(T, 44, 0)
    shape = (T, wl.MOE_TOPK, ex.d_in) if x_per_slot else (T, ex.d_in)
    x = wl.activation(shape, 44, 0, 7)
    got = _run(ex, x.bits, torch.float16, ids, torch.float32, x_per_slot)
    g = np.random.default_rng(T)
    rows = np.unique(np.concatenate([[0, ex.d_out - 1], g.integers(0, ex.d_out, 40)]))
    packed = [(Q[e], s[e], z[e], A[e], B[e]) for e in range(wl.MOE_EXPERTS)]
    ref = moe.forward_rows(packed, ranks, x.values, ids, x_per_slot, rows, 4, 128)
    assert_oracle(got[:, :, rows], ref)
    # bitwise deterministic, and the workspace carries nothing between calls
    again = _run(ex, x.bits, torch.float16, ids, torch.float32, x_per_slot)
    assert np.array_equal(got, again)


def test_layer_workspace_reuse_across_routings(moe_layer):
    ex, Q, s, z, A, B, ranks = moe_layer["gate"]
    ws = cl.workspace(cl.moe_workspace(ex, 64, 8, False), torch.device("cuda"))
    packed = [(Q[e], s[e], z[e], A[e], B[e]) for e in range(wl.MOE_EXPERTS)]
    rows = np.arange(0, ex.d_out, 97)
    for T, seed in ((64, 45), (3, 46), (17, 47)):
        ids, _ = wl.routing(T, seed, 0)
        x = wl.activation((T, ex.d_in), seed, 0, 7)
        y = cl.moe_linear_decode(ex, dev_u16(x.bits, torch.float16),
                                 torch.from_numpy(ids).cuda(), out_dtype=torch.float32, ws=ws)
        torch.cuda.synchronize()
        ref = moe.forward_rows(packed, ranks, x.values, ids, False, rows, 4, 128)
        assert_oracle(out_to_numpy(y)[:, :, rows], ref)


def _random_experts(E, d_out, d_in, r_max, seed):
    """Seeded device experts (packed codes, scales, zeros, factors, ranks)."""
    g = torch.Generator(device="cuda").manual_seed(seed)
    q = torch.randint(-2 ** 31, 2 ** 31 - 1, (E, d_out, d_in // 8), dtype=torch.int32, device="cuda", generator=g)
    s = (torch.rand((E, d_out, d_in // 128), device="cuda", generator=g) * 0.004 + 0.005).half()
    z = torch.randint(0, 16, (E, d_out, d_in // 128), device="cuda", generator=g).half()
    A = (torch.randn((E, r_max, d_in), device="cuda", generator=g) * 0.05).half()
    B = (torch.randn((E, d_out, r_max), device="cuda", generator=g) * 0.05).half()
    ranks = torch.randint(0, r_max + 1, (E,), dtype=torch.int32, device="cuda", generator=g)
    return cl.MoeExperts(q, s, z, A, B, ranks, E, d_out, d_in, 4, 128, r_max)


@pytest.mark.parametrize("x_per_slot", [False, True])
@pytest.mark.parametrize("T", [1, 8, 64])
def test_window_equals_singles_bitwise(T, x_per_slot):
    """A gate/up-style window (two linears of different d_out and r_max) over
    one routing gives each linear exactly its single-call result."""
    E, d_in, k = 128, 512, 8
    exs = [_random_experts(E, 96, d_in, 16, 50), _random_experts(E, 160, d_in, 8, 51)]
    ids = torch.from_numpy(wl.routing(T, 52, 0)[0]).cuda()
    x = torch.from_numpy(wl.activation((T, k, d_in) if x_per_slot else (T, d_in), 52, 0, 1).bits.view(np.int16))
    x = x.view(torch.float16).cuda()
    ys = cl.moe_linear_decode_window(exs, x, ids)
    singles = [cl.moe_linear_decode(ex, x, ids) for ex in exs]
    torch.cuda.synchronize()
    for y, ys1 in zip(ys, singles):
        assert torch.equal(y, ys1)
    # the window again, on a workspace reused from a different routing
    ws = cl.workspace(cl.moe_window_workspace(exs, T, k, x_per_slot), x.device)
    ids2 = torch.from_numpy(wl.routing(T, 53, 0)[0]).cuda()
    cl.moe_linear_decode_window(exs, x, ids2, ws=ws)
    again = cl.moe_linear_decode_window(exs, x, ids, ws=ws)
    torch.cuda.synchronize()
    for y, y2 in zip(ys, again):
        assert torch.equal(y, y2)


def test_window_matches_oracle():
    E, d_in, bits, G, k, T = 12, 512, 4, 128, 3, 5
    exs, host = [], []
    for i, (d_out, r_max) in enumerate(((100, 16), (60, 8))):
        Q, s, z, A, B = _oracle_experts(E, d_out, d_in, bits, G, r_max, 60 + i)
        ranks = wl.moe_expert_ranks(60 + i, 0, 0, E, levels=(0, 4, 8, r_max))
        exs.append(_device_experts(Q, s, z, A, B, ranks, d_out, d_in, bits, G, r_max))
        host.append((Q, s, z, A, B, ranks))
    ids = np.random.default_rng(62).integers(0, E, (T, k)).astype(np.int32)
    x = wl.activation((T, d_in), 62, 0, 1)
    ys = cl.moe_linear_decode_window(exs, dev_u16(x.bits, torch.float16),
                                     torch.from_numpy(ids).cuda(), out_dtype=torch.float32)
    torch.cuda.synchronize()
    for y, (Q, s, z, A, B, ranks) in zip(ys, host):
        ref = _full_ref(Q, s, z, A, B, ranks, x.values, ids, False, bits, G, d_in)
        assert_oracle(out_to_numpy(y), ref)


@pytest.mark.parametrize("x_per_slot", [False, True])
@pytest.mark.parametrize("T,k", [(3, 4), (16, 8)])
def test_slot_ranks_match_oracle(T, k, x_per_slot):
    """Per-slot ranks from the routing weights (Section 4.3.3) on the VALU
    path (3 x 4 slots) and the MFMA path (16 x 8 slots over 12 experts), against
    the oracle with the same per-slot ranks."""
    E, d_out, d_in, bits, G, r_max = 12, 100, 512, 4, 128, 16
    Q, s, z, A, B = _oracle_experts(E, d_out, d_in, bits, G, r_max, 70)
    ranks = wl.moe_expert_ranks(70, 0, 0, E, levels=(0, 4, 8, 16))
    ids, w = wl.routing(T, 70, 0, E, k)
    slot = wl.dynamic_slot_ranks(ids, w, ranks, (0, 4, 8, 16), r_max)
    x = wl.activation((T, k, d_in) if x_per_slot else (T, d_in), 70, 0, 1)
    ex = _device_experts(Q, s, z, A, B, ranks, d_out, d_in, bits, G, r_max)
    ys = cl.moe_linear_decode_window([ex], dev_u16(x.bits, torch.float16), torch.from_numpy(ids).cuda(),
                                     out_dtype=torch.float32, slot_ranks=[torch.from_numpy(slot).cuda()])
    torch.cuda.synchronize()
    experts = [(quant.dequant_packed(Q[e], s[e], z[e], bits, G, d_in), A[e], B[e]) for e in range(E)]
    ref = moe.forward(experts, ranks, x.values, ids, x_per_slot, slot_ranks=slot)
    assert_oracle(out_to_numpy(ys[0]), ref)
    # the per-slot ranks matter here: the static ranks miss the reference
    assert rel_l2(moe.forward(experts, ranks, x.values, ids, x_per_slot), ref) > 2 * REL_L2_TOL


@pytest.mark.parametrize("T", [1, 64])
def test_static_ranks_as_slot_ranks_are_bitwise_static(T):
    E, d_in, k = 128, 512, 8
    ex = _random_experts(E, 96, d_in, 16, 71)
    ids = torch.from_numpy(wl.routing(T, 72, 0)[0]).cuda()
    x = torch.from_numpy(wl.activation((T, d_in), 72, 0, 1).bits.view(np.int16)).view(torch.float16).cuda()
    slot = ex.ranks[ids.long()].to(torch.int32).contiguous()
    a = cl.moe_linear_decode_window([ex], x, ids)[0]
    b = cl.moe_linear_decode_window([ex], x, ids, slot_ranks=[slot])[0]
    torch.cuda.synchronize()
    assert torch.equal(a, b)


@pytest.mark.parametrize("G", [128, 64, 32])
@pytest.mark.parametrize("T", [1, 64])
def test_small_weight_scales(G, T):
    """Weights N(0, (5e-4)^2), group scales below 2^-10: 64 tokens over 12
    experts (several slots per expert: the MFMA backbone, one, two or four
    groups per 128-code block) and one token (the VALU backbone); every
    output dtype against the rounded oracle, elementwise bound included."""
    E, d_out, d_in, bits, r_max, k = 12, 100, 1024, 4, 16, 4
    Q, s, z, A, B = _oracle_experts(E, d_out, d_in, bits, G, r_max, 48 + G, svd=False, std=5e-4)
    assert float(np.median(s.astype(np.float64))) < 2.0 ** -10
    ranks = wl.moe_expert_ranks(48, 0, 0, E, levels=(0, 4, 8, 16))
    ids, _ = wl.routing(T, 48, 0, E, k)
    x = wl.activation((T, d_in), 48, 0, 1)
    ex = _device_experts(Q, s, z, A, B, ranks, d_out, d_in, bits, G, r_max)
    ref = _full_ref(Q, s, z, A, B, ranks, x.values, ids, False, bits, G, d_in)
    for od in OUT_DTYPES:
        assert_oracle(_run(ex, x.bits, torch.float16, ids, od, False), ref, od)


def test_out_of_range_ids_are_recorded_and_reported():
    """Routing ids -1 and E: zero output rows, and the device's routing-error
    record makes cl_moe_status report CL_EINVAL (naming the id) once; valid
    routing leaves it clear."""
    E, d_out, d_in, bits, G, r_max, T, k = 6, 64, 256, 4, 128, 8, 3, 2
    Q, s, z, A, B = _oracle_experts(E, d_out, d_in, bits, G, r_max, 49, svd=False)
    ranks = np.array([0, 8, 4, 0, 5, 2], dtype=np.int32)
    ex = _device_experts(Q, s, z, A, B, ranks, d_out, d_in, bits, G, r_max)
    x = wl.activation((T, d_in), 49, 0, 1)
    try:                                              # an earlier test's invalid ids may be on record
        cl.moe_status()
    except cl.ClError:
        pass
    cl.moe_status()                                   # reading the record cleared it
    good = np.array([[0, 1], [2, 3], [4, 5]], dtype=np.int32)
    _run(ex, x.bits, torch.float16, good, torch.float32, False)
    cl.moe_status()                                   # valid routing: nothing recorded
    for bad_id in (-1, E):
        ids = good.copy()
        ids[1, 1] = bad_id
        got = _run(ex, x.bits, torch.float16, ids, torch.float32, False)
        assert (got[1, 1] == 0).all()
        with pytest.raises(cl.ClError) as e:
            cl.moe_status()
        assert e.value.status == cl.CL_EINVAL
        assert "routing id %d in slot 3" % bad_id in str(e.value), str(e.value)
        cl.moe_status()                               # the record was cleared


@pytest.mark.parametrize("d_in,G,r_max,d_out", [(512, 128, 16, 100), (768, 64, 48, 333), (2048, 32, 128, 130),
                                                (4096, 128, 64, 77), (1536, 64, 0, 50)])
@pytest.mark.parametrize("x_per_slot", [False, True])
def test_direct_path_few_slots(d_in, G, r_max, d_out, x_per_slot):
    """At most 8 slots with 4-bit codes take the one-launch path (each
    workgroup forms its slot's activations and A_e x itself): rows of 16 to
    128 chunks (32- and 64-lane row sets, one or two chunks per lane), factor
    columns up to 128 (two per lane), rank 0, ragged row counts; one token
    of top-8 and two tokens of top-3 with an out-of-range id; static and
    per-slot ranks; fp16 and bf16 activations."""
    E = 10
    Q, s, z, A, B = _oracle_experts(E, d_out, d_in, 4, G, max(r_max, 1), 80 + d_in, svd=False)
    levels = (0, r_max // 4, r_max // 2, r_max) if r_max else (0,)
    ranks = wl.moe_expert_ranks(80, 0, d_in, E, levels=levels)
    ex = _device_experts(Q, s, z, A, B, ranks, d_out, d_in, 4, G, r_max)
    experts = [(quant.dequant_packed(Q[e], s[e], z[e], 4, G, d_in), A[e], B[e]) for e in range(E)]
    for (T, k), act in (((1, 8), "fp16"), ((2, 3), "bf16")):
        ids, w = wl.routing(T, 80, d_in, E, k)
        if T == 2:
            ids = ids.copy()
            ids[1, 2] = E                             # out of range: a zero row
        x = wl.activation((T, k, d_in) if x_per_slot else (T, d_in), 80, d_in, T, dtype=act)
        dt = torch.float16 if act == "fp16" else torch.bfloat16
        got = _run(ex, x.bits, dt, ids, torch.float32, x_per_slot)
        ref = _full_ref(Q, s, z, A, B, ranks, x.values, ids, x_per_slot, 4, G, d_in)
        assert_oracle(got, ref)
        if T == 2:
            assert (got[1, 2] == 0).all()
            with pytest.raises(cl.ClError):
                cl.moe_status()
        if r_max:
            valid = np.where((ids >= 0) & (ids < E), ids, 0)
            slot = wl.dynamic_slot_ranks(valid, w, ranks, levels, r_max)
            ys = cl.moe_linear_decode_window([ex], dev_u16(x.bits, dt), torch.from_numpy(ids).cuda(),
                                             out_dtype=torch.float32, slot_ranks=[torch.from_numpy(slot).cuda()])
            torch.cuda.synchronize()
            sref = moe.forward(experts, ranks, x.values, valid, x_per_slot, slot_ranks=slot)
            sref[(ids < 0) | (ids >= E)] = 0.0
            assert_oracle(out_to_numpy(ys[0]), sref)
            if T == 2:
                with pytest.raises(cl.ClError):
                    cl.moe_status()


# ------------------------- the down projection of the gated activations

def _abs_experts(Q, s, z, A, B, bits, G, d_in):
    """|W_e|, |A_e|, |B_e|: a forward over these and |h| bounds sum |W_eff h|."""
    return [(np.abs(quant.dequant_packed(Q[e], s[e], z[e], bits, G, d_in)), np.abs(A[e].astype(np.float64)),
             np.abs(B[e].astype(np.float64))) for e in range(len(Q))]


def _h_rounding_bound(absx, ranks, h, ids):
    """Elementwise bound of the output error that rounding each h to fp16
    (relative error <= 2^-11) can cause: 2^-11 sum_j |W_eff[i, j]| |h_j|."""
    return 2.0 ** -11 * moe.forward(absx, ranks, np.abs(h), ids, True)


@pytest.mark.parametrize("act", [torch.float16, torch.bfloat16])
@pytest.mark.parametrize("T,k", [(1, 4), (5, 3), (16, 8)])
def test_gated_down_full_outputs(T, k, act):
    """cl_moe_linear_decode_gated against the oracle down projection of
    h = SiLU(g) u (the expert nonlinearity between the gate/up and down
    windows, Section 4.2.2): the one-launch path (4 slots), the VALU path (15
    slots over 12 experts) and the MFMA path (128 slots), every output dtype,
    fp16 and bf16 gate/up values.  The kernel rounds each h to fp16; the
    elementwise bound adds what that rounding can move an output."""
    E, d_out, d_in, bits, G, r_max = 12, 100, 512, 4, 128, 16
    Q, s, z, A, B = _oracle_experts(E, d_out, d_in, bits, G, r_max, 80)
    ranks = wl.moe_expert_ranks(80, 0, 0, E, levels=(0, 4, 8, 16))
    ids, _ = wl.routing(T, 80, 0, E, k)
    dt = "bf16" if act == torch.bfloat16 else "fp16"
    g = wl.activation((T, k, d_in), 80, 0, 1, dtype=dt)
    u = wl.activation((T, k, d_in), 80, 0, 2, dtype=dt)
    h = linear.silu(g.values) * u.values
    ref = _full_ref(Q, s, z, A, B, ranks, h, ids, True, bits, G, d_in)
    extra = _h_rounding_bound(_abs_experts(Q, s, z, A, B, bits, G, d_in), ranks, h, ids)
    ex = _device_experts(Q, s, z, A, B, ranks, d_out, d_in, bits, G, r_max)
    gd, ud, idd = dev_u16(g.bits, act), dev_u16(u.bits, act), torch.from_numpy(ids).cuda()
    for od in OUT_DTYPES:
        y = cl.moe_linear_decode_gated(ex, gd, ud, idd, out_dtype=od)
        torch.cuda.synchronize()
        assert_oracle(out_to_numpy(y), ref, od, extra=extra)
    # the gating is applied: the plain down projection of g misses the reference
    assert rel_l2(_full_ref(Q, s, z, A, B, ranks, g.values, ids, True, bits, G, d_in), ref) > 0.5


@pytest.mark.parametrize("T", [1, 8, 64])
def test_gated_down_layer_sampled_rows(moe_layer, T):
    """The 128-expert down projection (2048 x 768) of gated activations at
    1, 8 and 64 tokens with top-8 routing, sampled rows; per-slot ranks."""
    ex, Q, s, z, A, B, ranks = moe_layer["down"]
    ids, w = wl.routing(T, 81, 0)
    g = wl.activation((T, wl.MOE_TOPK, ex.d_in), 81, 0, 1)
    u = wl.activation((T, wl.MOE_TOPK, ex.d_in), 81, 0, 2)
    slot = wl.dynamic_slot_ranks(ids, w, ranks, (0, 8, 16, 32), 32)
    idd = torch.from_numpy(ids).cuda()
    y = cl.moe_linear_decode_gated(ex, dev_u16(g.bits, torch.float16), dev_u16(u.bits, torch.float16), idd,
                                   out_dtype=torch.float32, slot_ranks=torch.from_numpy(slot).cuda())
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, ex.d_out - 1], np.random.default_rng(T).integers(0, ex.d_out, 40)]))
    h = linear.silu(g.values) * u.values
    experts = [(quant.dequant_packed(Q[e], s[e], z[e], 4, 128, ex.d_in)[rows], A[e], B[e][rows])
               for e in range(wl.MOE_EXPERTS)]
    ref = moe.forward(experts, ranks, h, ids, True, slot_ranks=slot)
    absx = [(np.abs(W), np.abs(a.astype(np.float64)), np.abs(b.astype(np.float64))) for W, a, b in experts]
    extra = 2.0 ** -11 * moe.forward(absx, ranks, np.abs(h), ids, True, slot_ranks=slot)
    assert_oracle(out_to_numpy(y)[:, :, rows], ref, extra=extra)


@pytest.mark.parametrize("T,k", [(1, 8), (16, 8)])
def test_gate_up_window_into_gated_down(T, k):
    """The MoE FFN chain: the gate/up window (fp16 outputs) feeds the gated
    down call directly.  Each stage against the oracle on the values it was
    handed: the window's outputs against the oracle gate and up projections,
    the down output against the oracle down projection of SiLU(g) u formed
    from the window's fp16 outputs; and the chain end to end against the
    oracle's own chain (intermediates in fp64)."""
    E, hid, ffn, bits, G = 16, 512, 256, 4, 128
    host, exs = [], []
    for m, (d_out, d_in, r_max) in enumerate(((ffn, hid, 16), (ffn, hid, 8), (hid, ffn, 16))):
        Q, s, z, A, B = _oracle_experts(E, d_out, d_in, bits, G, r_max, 82 + m)
        ranks = wl.moe_expert_ranks(82 + m, 0, m, E, levels=(0, 4, 8, r_max))
        host.append((Q, s, z, A, B, ranks, d_in))
        exs.append(_device_experts(Q, s, z, A, B, ranks, d_out, d_in, bits, G, r_max))
    ids, _ = wl.routing(T, 85, 0, E, k)
    x = wl.activation((T, hid), 85, 0, 1)
    idd = torch.from_numpy(ids).cuda()
    gy, uy = cl.moe_linear_decode_window(exs[:2], dev_u16(x.bits, torch.float16), idd, out_dtype=torch.float16)
    y = cl.moe_linear_decode_gated(exs[2], gy, uy, idd, out_dtype=torch.float32)
    torch.cuda.synchronize()
    refs = []
    for (Q, s, z, A, B, ranks, d_in), got in zip(host[:2], (gy, uy)):
        ref = _full_ref(Q, s, z, A, B, ranks, x.values, ids, False, bits, G, d_in)
        assert_oracle(out_to_numpy(got), ref, torch.float16)
        refs.append(ref)
    Q, s, z, A, B, ranks, d_in = host[2]
    h = linear.silu(out_to_numpy(gy)) * out_to_numpy(uy)
    ref = _full_ref(Q, s, z, A, B, ranks, h, ids, True, bits, G, d_in)
    extra = _h_rounding_bound(_abs_experts(Q, s, z, A, B, bits, G, d_in), ranks, h, ids)
    assert_oracle(out_to_numpy(y), ref, extra=extra)
    chain = _full_ref(Q, s, z, A, B, ranks, linear.silu(refs[0]) * refs[1], ids, True, bits, G, d_in)
    assert rel_l2(out_to_numpy(y), chain) <= REL_L2_TOL
