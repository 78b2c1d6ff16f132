"""Pins for the fp64 oracle: each test fixes part of it against something other
than itself -- a hand-worked example, a closed form, a theorem, brute force on
tiny inputs, or an independent numerical route.

Section 4.1 (compensated forward), Section 5.1 (GPTQ backbone; RTN without
calibration data), Appendix B.2 (Eckart-Young-Mirsky), Appendix B.1 (discrete
rank levels), Appendix C.1 Table 2 (rank tuples).
"""

import os

import numpy as np
import pytest

from oracle import comp, linear, moe, quant

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _finite_fp16_table():
    """All finite non-negative fp16 values, ascending, with their bit patterns."""
    bits = np.arange(0, 0x7C00, dtype=np.uint16)  # +0 .. largest finite
    vals = bits.view(np.float16).astype(np.float64)
    return vals, bits


def _nearest_fp16_brute(v):
    """Nearest fp16 by search over the whole finite grid, ties to even bits."""
    vals, bits = _finite_fp16_table()
    out = np.empty_like(v)
    for i, x in enumerate(v):
        a = abs(x)
        if a > 65504.0 + 16.0:  # beyond half an ulp past the max: overflow
            out[i] = np.inf if x > 0 else -np.inf
            continue
        j = np.searchsorted(vals, a)
        cands = [k for k in (j - 1, j) if 0 <= k < len(vals)]
        d = [abs(vals[k] - a) for k in cands]
        best = min(d)
        tied = [k for k, dk in zip(cands, d) if dk == best]
        k = tied[0] if len(tied) == 1 else [k for k in tied if bits[k] % 2 == 0][0]
        out[i] = np.copysign(vals[k], x)
    return out


# ----------------------------------------------------------- fp16 rounding

def test_fp16_rne_matches_brute_force_nearest():
    g = np.random.default_rng(11)
    vals, _ = _finite_fp16_table()
    mids = (vals[:-1] + vals[1:]) / 2  # exact in fp64: every tie case
    pick = g.choice(len(mids), 3000, replace=False)
    v = np.concatenate([
        mids[pick], -mids[pick[:500]],
        g.standard_normal(2000) * 0.03,             # the range scales live in
        g.standard_normal(500) * 1e-6,              # subnormal range
        g.uniform(1000, 65504, 500),
        vals[pick] * (1 + 1e-12),                   # just off a grid point
    ])
    got = quant.fp16_rne(v).astype(np.float64)
    np.testing.assert_array_equal(got, _nearest_fp16_brute(v))


# ---------------------------------------------------------- quantization

def _worked_examples():
    blocks, cur = [], {}
    for line in open(os.path.join(GOLDEN, "quant_worked_example.txt")):
        if line.startswith("#"):
            continue
        if not line.strip():
            if cur:
                blocks.append(cur)
            cur = {}
            continue
        k, v = line.split(":", 1)
        cur[k] = v
    if cur:
        blocks.append(cur)
    return blocks


def test_hand_worked_groups():
    examples = _worked_examples()
    assert len(examples) == 2
    for ex in examples:
        w = np.array([float(t) for t in ex["w"].split()], dtype=np.float32)[None, :]
        codes, s, z = quant.quantize(w, 4, 8)
        assert float(s[0, 0]) == int(ex["scale_units_of_2^-16"]) * 2.0 ** -16
        assert float(z[0, 0]) == int(ex["zero"])
        assert codes[0].tolist() == [int(t) for t in ex["codes"].split()]
        Q = quant.pack(codes, 4)
        assert int(Q[0, 0]) == int(ex["packed_word_hex"], 16)


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_one_sided_groups_keep_zero_on_the_grid(bits):
    """All-positive and all-negative groups: the grid still contains 0, so a
    group of exact multiples of a power-of-two step is recovered exactly."""
    qmax = (1 << bits) - 1
    step = 2.0 ** -5
    k = np.arange(1, qmax + 1, dtype=np.float64)
    G = 2 * len(k) if bits == 2 else len(k) + 1
    pos = np.resize(k, G); pos[-1] = qmax
    W = np.stack([pos * step, -pos * step]).astype(np.float32)
    if W.shape[1] % (32 // bits):
        pad = (32 // bits) - W.shape[1] % (32 // bits)
        W = np.concatenate([W, np.repeat(W[:, -1:], pad, axis=1)], axis=1)
    G = W.shape[1]
    codes, s, z = quant.quantize(W, bits, G)
    assert np.all(s.astype(np.float64) == step)
    assert float(z[0, 0]) == 0 and float(z[1, 0]) == qmax
    np.testing.assert_array_equal(quant.dequant(codes, s, z, G), W.astype(np.float64))


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_on_grid_weights_are_recovered_exactly(bits):
    """Weights built on a grid with a power-of-two step are fixed points of
    quantize -> dequantize: same codes, same zero point, zero residual."""
    g = np.random.default_rng(bits)
    qmax = (1 << bits) - 1
    G, n_groups, rows = 32, 6, 5
    step = 2.0 ** -7
    codes = g.integers(0, qmax + 1, (rows, n_groups, G))
    codes[:, :, 0] = 0
    codes[:, :, 1] = qmax          # group spans the whole grid -> s == step
    z = g.integers(0, qmax + 1, (rows, n_groups))
    W = (step * (codes - z[:, :, None])).astype(np.float32).reshape(rows, n_groups * G)
    c2, s2, z2 = quant.quantize(W, bits, G)
    np.testing.assert_array_equal(c2, codes.reshape(rows, -1))
    np.testing.assert_array_equal(z2.astype(np.int64), z)
    assert np.all(s2.astype(np.float64) == step)
    np.testing.assert_array_equal(quant.dequant(c2, s2, z2, G), W.astype(np.float64))


def test_round_half_to_even_on_exact_ties():
    step = 2.0 ** -6
    # lo = -3 step, hi = 12 step fix s = step, z = 3; the middle values sit on
    # exact half steps: 2.5 -> 2 and 3.5 -> 4 (even), -0.5 -> 0, -1.5 -> -2.
    w = np.array([-3, 12, 2.5, 3.5, -0.5, -1.5, 0.5, 5.5], dtype=np.float64) * step
    codes, s, z = quant.quantize(w.astype(np.float32)[None, :], 4, 8)
    assert float(s[0, 0]) == step and float(z[0, 0]) == 3
    assert (codes[0] - 3).tolist() == [-3, 12, 2, 4, 0, -2, 0, 6]


@pytest.mark.parametrize("bits,G", [(4, 8), (2, 8), (3, 8), (4, 128), (2, 64), (3, 128)])
def test_codes_are_brute_force_nearest_grid_points(bits, G):
    g = np.random.default_rng(100 + bits + G)
    qmax = (1 << bits) - 1
    W = (0.02 * g.standard_normal((8, 2 * G))).astype(np.float32)
    W[0, :G] = 0.0                                   # degenerate all-zero group
    W[1, :G] = np.abs(W[1, :G])                      # one-sided group (lo = 0)
    codes, s, z = quant.quantize(W, bits, G)
    s64 = np.repeat(s.astype(np.float64), G, axis=1)
    z64 = np.repeat(z.astype(np.float64), G, axis=1)
    cand = np.arange(qmax + 1, dtype=np.float64)
    for o in range(W.shape[0]):
        for c in range(W.shape[1]):
            err = np.abs(float(W[o, c]) - s64[o, c] * (cand - z64[o, c]))
            best = np.flatnonzero(err == err.min())
            if len(best) > 1:
                best = [b for b in best if (b - z64[o, c]) % 2 == 0]
            assert codes[o, c] == best[0], (o, c)
    # all-zero group: the grid falls back to [-1, 1]
    qs = quant.fp16_rne(2.0 / qmax).astype(np.float64)
    assert np.all(s[0, 0] == qs) and np.all(quant.dequant(codes, s, z, G)[0, :G] == 0)


def test_quantizer_invariants():
    g = np.random.default_rng(7)
    for bits, G in [(4, 128), (2, 64), (3, 128)]:
        qmax = (1 << bits) - 1
        W = (0.02 * g.standard_normal((64, 512))).astype(np.float32)
        codes, s, z = quant.quantize(W, bits, G)
        assert codes.min() >= 0 and codes.max() <= qmax
        zf = z.astype(np.float64)
        assert np.all(zf == np.round(zf)) and zf.min() >= 0 and zf.max() <= qmax
        Wh = quant.dequant(codes, s, z, G)
        assert np.all(Wh.astype(np.float32).astype(np.float64) == Wh)   # exact in fp32
        s64 = np.repeat(s.astype(np.float64), G, axis=1)
        z64 = np.repeat(zf, G, axis=1)
        raw = np.rint(W.astype(np.float64) / s64) + z64
        unclamped = (raw >= 0) & (raw <= qmax)
        assert np.all(np.abs(W - Wh)[unclamped] <= s64[unclamped] / 2)


# ------------------------------------------------------------------ packing

@pytest.mark.parametrize("bits", [2, 4])
def test_pack_exhaustive_slots_and_values(bits):
    per = 32 // bits
    rows = []
    for slot in range(per):
        for v in range(1 << bits):
            r = np.zeros(per, dtype=np.int64)
            r[slot] = v
            rows.append(r)
    codes = np.array(rows)
    Q = quant.pack(codes, bits)
    for i, r in enumerate(rows):
        expect = sum(int(c) << (bits * j) for j, c in enumerate(r))
        assert int(Q[i, 0]) == expect
    np.testing.assert_array_equal(quant.unpack(Q, bits, per), codes)


@pytest.mark.parametrize("bits", [2, 4])
def test_pack_random_rows_against_integer_arithmetic(bits):
    g = np.random.default_rng(bits)
    per = 32 // bits
    codes = g.integers(0, 1 << bits, (7, 5 * per))
    Q = quant.pack(codes, bits)
    for o in range(codes.shape[0]):
        for wi in range(5):
            expect = sum(int(codes[o, wi * per + j]) << (bits * j) for j in range(per))
            assert int(Q[o, wi]) == expect
    np.testing.assert_array_equal(quant.unpack(Q, bits, codes.shape[1]), codes)


def _pack3_examples():
    blocks = []
    cur = {}
    for line in open(os.path.join(GOLDEN, "pack3_straddling_codes.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        key, val = line.split(":", 1)
        cur[key] = val.split()
        if key == "words_hex":
            blocks.append(cur)
            cur = {}
    return blocks


def test_pack3_hand_worked_straddling_codes():
    """3-bit codes: the hand-worked units of the golden file, including the
    two codes of every 32 that straddle a word boundary."""
    ex = _pack3_examples()
    assert len(ex) == 4
    for e in ex:
        codes = np.array([int(t) for t in e["codes"]], dtype=np.int64)[None, :]
        Q = quant.pack(codes, 3)
        assert [int(v) for v in Q[0]] == [int(h, 16) for h in e["words_hex"]]
        np.testing.assert_array_equal(quant.unpack(Q, 3, 32), codes)


def _row_as_integer_words(codes_row, bits):
    """Words of a row read off one big integer sum(code_c << (bits c))."""
    v = 0
    for c, q in enumerate(codes_row):
        v += int(q) << (bits * c)
    n = len(codes_row) * bits // 32
    return [(v >> (32 * i)) & 0xFFFFFFFF for i in range(n)]


def test_pack3_exhaustive_slots_and_values():
    """Every value 0..7 at every one of the 32 positions of a 3-word unit
    (codes 10 and 21 straddle words) against the row read as one integer."""
    rows = []
    for slot in range(32):
        for v in range(8):
            r = np.zeros(32, dtype=np.int64)
            r[slot] = v
            rows.append(r)
    codes = np.array(rows)
    Q = quant.pack(codes, 3)
    for i, r in enumerate(rows):
        assert [int(w) for w in Q[i]] == _row_as_integer_words(r, 3), i
    np.testing.assert_array_equal(quant.unpack(Q, 3, 32), codes)


@pytest.mark.parametrize("bits", [2, 3, 4])
def test_pack_random_rows_against_one_integer_per_row(bits):
    g = np.random.default_rng(10 + bits)
    codes = g.integers(0, 1 << bits, (6, 160))
    Q = quant.pack(codes, bits)
    for o in range(codes.shape[0]):
        assert [int(w) for w in Q[o]] == _row_as_integer_words(codes[o], bits)
    np.testing.assert_array_equal(quant.unpack(Q, bits, codes.shape[1]), codes)


# ------------------------------------------------------------- compensation

def test_eckart_young_mirsky_tail_energy_and_spectral_norm():
    g = np.random.default_rng(3)
    E = g.standard_normal((12, 9))
    W_hat = np.zeros_like(E)
    A, B, sigma = comp.build_compensation(E, W_hat, 9)
    fro2 = np.sum(E * E)
    for r in range(0, 10):
        R = E - B[:, :r] @ A[:r]
        tail = np.sum(sigma[r:] ** 2)
        assert abs(np.sum(R * R) - tail) <= 1e-12 * fro2
        spec = np.linalg.norm(R, 2)
        assert abs(spec - (sigma[r] if r < 9 else 0.0)) <= 1e-12 * sigma[0]


def test_singular_values_and_subspaces_match_gram_eigendecomposition():
    """Independent route: eigen-decomposition of E^T E gives sigma^2 and the
    right singular subspaces."""
    g = np.random.default_rng(4)
    E = g.standard_normal((10, 7)) @ np.diag([9, 7, 5, 3, 2, 1, 0.5])
    A, B, sigma = comp.build_compensation(E, np.zeros_like(E), 7)
    lam, V = np.linalg.eigh(E.T @ E)
    lam, V = lam[::-1], V[:, ::-1]
    np.testing.assert_allclose(sigma ** 2, lam, rtol=1e-10)
    for r in range(1, 7):
        P_oracle = A[:r].T @ np.linalg.pinv(A[:r].T)     # projector onto span(A_r^T)
        P_eig = V[:, :r] @ V[:, :r].T
        np.testing.assert_allclose(P_oracle, P_eig, atol=1e-10)


def test_sign_convention_and_factor_shapes():
    g = np.random.default_rng(5)
    E = g.standard_normal((6, 11))
    A, B, sigma = comp.build_compensation(E, np.zeros_like(E), 4)
    assert A.shape == (4, 11) and B.shape == (6, 4)
    for j in range(4):
        col = B[:, j]
        assert col[np.argmax(np.abs(col))] > 0


def test_full_rank_factors_reproduce_the_full_precision_layer():
    """With every singular pair kept in fp64 the compensated layer equals the
    unquantized layer ``W x`` (spec property, 1e-10)."""
    g = np.random.default_rng(6)
    W = (0.02 * g.standard_normal((64, 96))).astype(np.float32)
    Q, s, z = quant.quantize_pack(W, 4, 32)
    W_hat = quant.dequant_packed(Q, s, z, 4, 32, 96)
    A, B, _ = comp.build_compensation(W, W_hat, 64)
    X = g.standard_normal((3, 96))
    Y = linear.forward(W_hat, A, B, 64, X)
    ref = X @ W.astype(np.float64).T
    assert np.linalg.norm(Y - ref) / np.linalg.norm(ref) < 1e-10
    # ...and rank 0 is the quantized layer alone, which is measurably different
    Y0 = linear.forward(W_hat, A, B, 0, X)
    assert np.linalg.norm(Y0 - ref) / np.linalg.norm(ref) > 1e-3


# ------------------------------------------------------------------ forward

def _forward_scalar_loops(W_hat, A, B, r, X):
    T, d_in = X.shape
    d_out = W_hat.shape[0]
    Y = [[0.0] * d_out for _ in range(T)]
    for t in range(T):
        tt = [sum(float(A[i][c]) * float(X[t][c]) for c in range(d_in)) for i in range(r)]
        for o in range(d_out):
            acc = sum(float(W_hat[o][c]) * float(X[t][c]) for c in range(d_in))
            acc += sum(float(B[o][i]) * tt[i] for i in range(r))
            Y[t][o] = acc
    return np.array(Y)


@pytest.mark.parametrize("rank", [0, 1, 3, 5])
def test_forward_matches_scalar_triple_loops(rank):
    g = np.random.default_rng(20 + rank)
    d_out, d_in, r_max, T = 6, 16, 5, 3            # non-square: catches transposes
    W = (0.02 * g.standard_normal((d_out, d_in))).astype(np.float32)
    Q, s, z = quant.quantize_pack(W, 4, 8)
    A = g.standard_normal((r_max, d_in))
    B = g.standard_normal((d_out, r_max))
    X = g.standard_normal((T, d_in))
    W_hat = quant.dequant_packed(Q, s, z, 4, 8, d_in)
    got = linear.forward_packed(Q, s, z, 4, 8, A, B, rank, X)
    np.testing.assert_allclose(got, _forward_scalar_loops(W_hat, A, B, rank, X), rtol=1e-12, atol=1e-14)


def test_silu_against_logistic_function_and_lambert_w_minimum():
    """SiLU(v) = v * sigma(v) with scipy's logistic function; its odd part is
    v / 2 (SiLU(v) - SiLU(-v) = v); its minimum, where 1 + v (1 - sigma(v)) = 0,
    is at v* = -1 - W(1/e) with value v* + 1 = -W(1/e) (Lambert W)."""
    from scipy import special
    v = np.concatenate([np.linspace(-60.0, 60.0, 2001), [-1000.0, -745.0, 0.0, 745.0, 1000.0]])
    got = linear.silu(v)
    np.testing.assert_allclose(got, v * special.expit(v), rtol=1e-14, atol=1e-300)
    np.testing.assert_allclose(linear.silu(v) - linear.silu(-v), v, rtol=1e-14, atol=1e-14)
    w = float(np.real(special.lambertw(np.exp(-1.0))))
    vmin = -1.0 - w
    assert abs(float(linear.silu(vmin)) - (-w)) < 1e-15
    grid = np.linspace(vmin - 0.5, vmin + 0.5, 100001)
    assert float(linear.silu(grid).min()) >= -w - 1e-15
    assert linear.silu(np.array([-1000.0]))[0] == 0.0 and linear.silu(np.array([1000.0]))[0] == 1000.0


def test_forward_glu_matches_scalar_loops():
    """SiLU(gate x) * (up x) on a 5 x 16 pair of compensated linears, every
    output by scalar loops and math.exp."""
    import math
    g = np.random.default_rng(24)
    d_out, d_in, T = 5, 16, 3
    mats = []
    for rank in (3, 0):
        W = (0.05 * g.standard_normal((d_out, d_in))).astype(np.float32)
        Q, s, z = quant.quantize_pack(W, 4, 8)
        mats.append((quant.dequant_packed(Q, s, z, 4, 8, d_in), g.standard_normal((4, d_in)),
                     g.standard_normal((d_out, 4)), rank))
    X = g.standard_normal((T, d_in))
    yg = _forward_scalar_loops(*mats[0], X)
    yu = _forward_scalar_loops(*mats[1], X)
    want = [[yg[t][o] / (1.0 + math.exp(-yg[t][o])) * yu[t][o] for o in range(d_out)] for t in range(T)]
    np.testing.assert_allclose(linear.forward_glu(mats[0], mats[1], X), want, rtol=1e-12, atol=1e-14)


def test_forward_rows_is_a_row_sample_of_forward():
    g = np.random.default_rng(21)
    W = (0.02 * g.standard_normal((40, 64))).astype(np.float32)
    Q, s, z = quant.quantize_pack(W, 4, 32)
    A = g.standard_normal((8, 64)); B = g.standard_normal((40, 8))
    X = g.standard_normal((2, 64))
    full = linear.forward_packed(Q, s, z, 4, 32, A, B, 6, X)
    rows = np.array([0, 7, 39, 12])
    # same arithmetic on a row subset; BLAS may order the sums differently
    np.testing.assert_allclose(linear.forward_rows(Q, s, z, 4, 32, A, B, 6, X, rows), full[:, rows],
                               rtol=1e-13, atol=1e-13)


def test_8x8_end_to_end_brute_force():
    """Quantize, build factors, run the forward: every step on an 8x8 case
    checked by brute force (scalar loops, exhaustive grid search)."""
    g = np.random.default_rng(8)
    W = (0.02 * g.standard_normal((8, 8))).astype(np.float32)
    for bits in (2, 3, 4):
        codes, s, z = quant.quantize(W, bits, 8)
        W_hat = quant.dequant(codes, s, z, 8)
        A, B, sigma = comp.build_compensation(W, W_hat, 8)
        X = g.standard_normal((2, 8))
        for r in range(9):
            got = linear.forward(W_hat, A, B, r, X)
            np.testing.assert_allclose(got, _forward_scalar_loops(W_hat, A, B, r, X), rtol=1e-12, atol=1e-15)
        E = W.astype(np.float64) - W_hat
        lam = np.sort(np.linalg.eigvalsh(E @ E.T))[::-1]
        np.testing.assert_allclose(sigma ** 2, np.clip(lam, 0, None), rtol=1e-9, atol=1e-20)


# ---------------------------------------------------------------------- MoE

def _tiny_experts(g, E, d_out, d_in, r_max):
    experts = []
    for _ in range(E):
        W = (0.02 * g.standard_normal((d_out, d_in))).astype(np.float32)
        codes, s, z = quant.quantize(W, 4, 8)
        experts.append((quant.dequant(codes, s, z, 8), g.standard_normal((r_max, d_in)),
                        g.standard_normal((d_out, r_max))))
    return experts


def test_moe_matches_scalar_loops_and_reduces_to_dense():
    g = np.random.default_rng(30)
    E, d_out, d_in, r_max, T, k = 5, 4, 8, 3, 3, 2
    experts = _tiny_experts(g, E, d_out, d_in, r_max)
    ranks = [0, 1, 3, 2, 3]
    ids = np.array([[1, 4], [0, 2], [4, 3]])
    X = g.standard_normal((T, d_in))
    Y = moe.forward(experts, ranks, X, ids, x_per_slot=False)
    for t in range(T):
        for j in range(k):
            W_hat, A, B = experts[ids[t, j]]
            ref = _forward_scalar_loops(W_hat, A, B, ranks[ids[t, j]], X[t:t + 1])[0]
            np.testing.assert_allclose(Y[t, j], ref, rtol=1e-12, atol=1e-15)
    Xs = g.standard_normal((T, k, d_in))
    Ys = moe.forward(experts, ranks, Xs, ids, x_per_slot=True)
    W_hat, A, B = experts[ids[2, 1]]
    np.testing.assert_allclose(Ys[2, 1], _forward_scalar_loops(W_hat, A, B, ranks[ids[2, 1]], Xs[2, 1][None])[0],
                               rtol=1e-12, atol=1e-15)
    # one token, one slot: the dense layer of that expert
    d = moe.forward(experts, ranks, X[:1], ids[:1, :1], False)[0, 0]
    np.testing.assert_array_equal(d, linear.forward(*experts[1], ranks[1], X[:1])[0])
    # permuting tokens permutes outputs
    perm = np.array([2, 0, 1])
    np.testing.assert_array_equal(moe.forward(experts, ranks, X[perm], ids[perm], False), Y[perm])


def test_moe_slot_ranks_follow_each_slot():
    """Per-slot ranks (Section 4.3.3): each slot is its expert's dense layer at
    that slot's own rank (scalar loops); the experts' ranks as slot ranks give
    the static result exactly."""
    g = np.random.default_rng(32)
    E, d_out, d_in, r_max, T, k = 4, 3, 8, 3, 3, 2
    experts = _tiny_experts(g, E, d_out, d_in, r_max)
    ranks = [3, 1, 2, 0]
    ids = np.array([[1, 0], [0, 0], [3, 2]])
    slot = np.array([[0, 3], [1, 2], [3, 1]])
    X = g.standard_normal((T, d_in))
    Y = moe.forward(experts, ranks, X, ids, False, slot_ranks=slot)
    for t in range(T):
        for j in range(k):
            W_hat, A, B = experts[ids[t, j]]
            ref = _forward_scalar_loops(W_hat, A, B, slot[t, j], X[t:t + 1])[0]
            np.testing.assert_allclose(Y[t, j], ref, rtol=1e-12, atol=1e-15)
    static = np.array([[ranks[e] for e in row] for row in ids])
    np.testing.assert_array_equal(moe.forward(experts, ranks, X, ids, False, slot_ranks=static),
                                  moe.forward(experts, ranks, X, ids, False))


def test_moe_forward_rows_is_forward_restricted_to_rows():
    g = np.random.default_rng(31)
    E, d_out, d_in, r_max, T, k = 4, 6, 16, 3, 2, 3
    packed, experts = [], []
    for _ in range(E):
        W = (0.02 * g.standard_normal((d_out, d_in))).astype(np.float32)
        Q, s, z = quant.quantize_pack(W, 4, 8)
        A, B = g.standard_normal((r_max, d_in)), g.standard_normal((d_out, r_max))
        packed.append((Q, s, z, A, B))
        experts.append((quant.dequant_packed(Q, s, z, 4, 8, d_in), A, B))
    ranks = [3, 0, 2, 1]
    ids = np.array([[0, 3, 1], [2, 2, 0]])
    rows = np.array([5, 0, 3])
    for x_per_slot, X in ((False, g.standard_normal((T, d_in))), (True, g.standard_normal((T, k, d_in)))):
        full = moe.forward(experts, ranks, X, ids, x_per_slot)
        np.testing.assert_allclose(moe.forward_rows(packed, ranks, X, ids, x_per_slot, rows, 4, 8),
                                   full[:, :, rows], rtol=1e-12, atol=1e-15)
