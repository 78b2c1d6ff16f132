"""Input generators: reproducible, in the documented value sets, and the rank
tables follow the discrete alignment of the paper's allocator (Appendix B.1)."""

import os

import numpy as np

from paper_2605_05819_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_seeds_reproduce_identical_arrays():
    a = wl.weight((64, 128), 1, 0, 4)
    b = wl.weight((64, 128), 1, 0, 4)
    c = wl.weight((64, 128), 1, 0, 5)
    assert a.dtype == np.float32 and np.array_equal(a, b) and not np.array_equal(a, c)
    x1 = wl.activation((4, 128), 1, dtype="fp16")
    x2 = wl.activation((4, 128), 1, dtype="fp16")
    assert np.array_equal(x1.bits, x2.bits)


def test_activation_bits_and_values_agree():
    x = wl.activation((3, 256), 9, dtype="fp16")
    assert np.array_equal(x.bits.view(np.float16).astype(np.float64), x.values)
    y = wl.activation((3, 256), 9, dtype="bf16")
    # bf16 values are float32 values with the low 16 bits clear
    f = y.values.astype(np.float32).view(np.uint32)
    assert np.all(f & 0xFFFF == 0) and np.array_equal((f >> 16).astype(np.uint16), y.bits)
    # same draws, two roundings: close to each other
    assert np.max(np.abs(x.values - y.values)) < 0.05


def test_bf16_rounding_ties_to_even():
    # 1 + 2^-8 is halfway between bf16 neighbours 1 and 1 + 2^-7 -> 1 (even)
    v = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8)], dtype=np.float32)
    got = wl.bf16_bits_to_f64(wl.fp32_to_bf16_bits(v))
    assert got.tolist() == [1.0, 1 + 2 ** -6, -1.0]


def test_align_is_nearest_level_ties_low():
    L = (0, 16, 32, 64, 128)
    assert [wl.align(x, L) for x in (0, 7.9, 8, 8.1, 24, 47, 49, 96, 97, 500)] == \
        [0, 0, 0, 16, 16, 32, 64, 64, 128, 128]


def test_rank_tables_respect_levels_budget_and_order():
    for wk in range(20):
        scores = [wl.rng(wk, 0, m, 0, wl.TAG_SCORE).random() for m in range(7)]
        L = (0, 16, 32, 64, 128)
        ranks = wl.allocate_ranks(scores, L, 448)
        assert all(r in L for r in ranks) and sum(ranks) <= 448
        for i in range(7):
            for j in range(7):
                if scores[i] > scores[j]:
                    assert ranks[i] >= ranks[j]
    layer = wl.llama_layer()
    assert sum(l.rank for l in layer.linears) <= 448
    layer2 = wl.llama_layer_2bit()
    assert sum(l.rank for l in layer2.linears) <= 896
    assert all(l.rank in (0, 16, 32, 64, 128, 256) for l in layer2.linears)


def test_paper_rank_tuples_lie_on_the_power_of_two_level_set():
    """Table 2's allocations use ranks in {0} U {2^k, k >= 3}; the level sets
    the workloads draw from are subsets of that set."""
    rows = [list(map(int, l.split(","))) for l in open(os.path.join(GOLDEN, "table2_rank_tuples.txt"))
            if l.strip() and not l.startswith("#")]
    assert len(rows) == 24 and all(len(r) == 7 for r in rows)
    admissible = {0} | {2 ** k for k in range(3, 12)}
    assert all(v in admissible for r in rows for v in r)
    for L in ((0, 16, 32, 64, 128), (0, 16, 32, 64, 128, 256), (0, 8, 16, 32)):
        assert set(L) <= admissible


def test_routing_is_topk_of_softmax_and_normalised():
    ids, w = wl.routing(64, 5, 0)
    assert ids.shape == (64, 8) and ids.dtype == np.int32
    g = wl.rng(5, 0, 0, 0, wl.TAG_ROUTE)
    logits = g.standard_normal((64, 128))
    for t in range(64):
        assert len(set(ids[t].tolist())) == 8
        # chosen experts are the 8 largest logits, in descending order
        assert ids[t].tolist() == list(np.argsort(-logits[t], kind="stable")[:8])
        assert abs(w[t].sum() - 1) < 1e-12 and np.all(np.diff(w[t]) <= 0)
        # expert activation score k * g_e averages to 1 over the slots
        assert abs((8 * w[t]).mean() - 1) < 1e-12


def test_standin_codes_shapes_ranges_and_seeding():
    q, s, z = wl.standin_codes(3, 5, 256, 4, 128, 9, 1, 2)
    assert q.shape == (3, 5, 32) and q.dtype == np.uint32
    assert s.shape == z.shape == (3, 5, 2) and s.dtype == z.dtype == np.float16
    assert (s > 0).all() and np.isfinite(s).all()
    assert (z == np.round(z)).all() and z.min() >= 0 and z.max() <= 15
    q2, s2, z2 = wl.standin_codes(3, 5, 256, 4, 128, 9, 1, 2)
    assert (q == q2).all() and (s == s2).all() and (z == z2).all()
    # every nibble value occurs (uniform words)
    nib = (q[..., None] >> (4 * np.arange(8, dtype=np.uint32))) & 15
    assert set(np.unique(nib)) == set(range(16))
    q3, _, z3 = wl.standin_codes(2, 4, 128, 2, 64, 9)
    assert q3.shape == (2, 4, 8) and z3.max() <= 3


def test_dynamic_slot_ranks_scale_with_routing_weight():
    levels, r_max = (0, 8, 16, 32), 32
    ranks = np.array([0, 8, 16, 32, 16], dtype=np.int32)
    ids = np.array([[1, 2, 3, 4], [4, 3, 2, 1], [2, 2, 0, 3]])
    k = ids.shape[1]
    # an even split (g = 1/k) keeps every expert's own rank
    even = np.full(ids.shape, 1.0 / k)
    np.testing.assert_array_equal(wl.dynamic_slot_ranks(ids, even, ranks, levels, r_max), ranks[ids])
    # real routing weights: every rank is a level, capped at r_max, and for one
    # expert the rank does not fall as its weight grows
    T = 32
    ids, w = wl.routing(T, 9, 0, num_experts=5, k=4)
    r = wl.dynamic_slot_ranks(ids, w, ranks, levels, r_max)
    assert set(np.unique(r)) <= set(levels) and r.max() <= r_max
    for e in range(5):
        sel = ids == e
        order = np.argsort(w[sel], kind="stable")
        assert np.all(np.diff(r[sel][order]) >= 0)
    # a heavy slot gets more than its expert's rank, a light one less
    assert wl.dynamic_slot_ranks(np.array([[1, 4]]), np.array([[0.9, 0.1]]), ranks, levels, r_max).tolist() == [[16, 0]]


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU: --gpus above 1 exits with a message before
    touching a device."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr
