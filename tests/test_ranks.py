"""Rank allocation from residual spectra (Section 4.3; Appendix B.1): the
oracle pinned by hand-worked spectra, closed forms and an independent
characterisation of proportional sharing; the host library's
cl_allocate_ranks / cl_layer_sensitivity equal to the oracle exactly (host
code: no GPU needed)."""

import ctypes
import math

import numpy as np
import pytest

from oracle import ranks
from paper_2605_05819_amd import cl

LEVELS = (0, 8, 16, 32, 64, 128, 256)


def test_hand_worked_knee():
    """sigma = (4, 3, 1, 1, 1): sigma / 4 = (1, .75, .25, .25, .25); second
    differences at j = 2, 3, 4 are -.25, .5, 0; the knee is j = 3, so the
    salient set is {1, 2, 3} and phi = (8 / 3) / 1."""
    size, phi = ranks.salience([4.0, 3.0, 1.0, 1.0, 1.0], 0.01)
    assert size == 3 and phi == pytest.approx(8.0 / 3.0, rel=1e-15)


def test_equal_second_differences_take_the_first():
    """sigma = (4, 2, 2, 2, 0, 0): sigma / 4 = (1, .5, .5, .5, 0, 0) with second
    differences .5, 0, -.5, .5 at j = 2..5 (exact in binary); the first
    maximum, j = 2, gives the salient set {1, 2} and phi = .75 / .25 = 3."""
    assert ranks.salience([4.0, 2.0, 2.0, 2.0, 0.0, 0.0], 0.01) == (2, 3.0)


@pytest.mark.parametrize("q,n", [(0.5, 10), (0.8, 40), (0.95, 64)])
def test_geometric_spectrum_closed_form(q, n):
    """sigma_j = q^(j-1): the second difference q^(j-2) (1 - q)^2 falls with j,
    so the knee is j = 2 when (1 - q)^2 > tau (else no salient set), and
    phi = ((1 + q) / 2) / (sum_{j>=3} q^(j-1) / (n - 2))."""
    sigma = [q ** j for j in range(n)]
    size, phi = ranks.salience(sigma, 0.01)
    if (1 - q) ** 2 > 0.01:
        tail = (q * q) * (1 - q ** (n - 2)) / (1 - q) / (n - 2)
        assert size == 2 and phi == pytest.approx((1 + q) / 2 / tail, rel=1e-12)
    else:
        assert (size, phi) == (0, 1.0)


def test_flat_and_linear_spectra_have_no_knee_and_scale_does_not_matter():
    assert ranks.salience([2.0] * 50, 0.01) == (0, 1.0)
    assert ranks.salience(list(np.linspace(5.0, 1.0, 50)), 0.01) == (0, 1.0)
    assert ranks.salience([1.0, 0.5], 0.01) == (0, 1.0)          # no interior index
    assert ranks.salience([0.0, 0.0, 0.0], 0.01) == (0, 1.0)     # zero residual
    g = np.random.default_rng(3)
    for _ in range(20):
        s = np.sort(np.abs(g.standard_normal(30)) ** 3)[::-1]
        for c in (1e-3, 7.0, 2.0 ** 20):
            a, b = ranks.salience(s, 0.01), ranks.salience(s * c, 0.01)
            assert a[0] == b[0] and a[1] == pytest.approx(b[1], rel=1e-12)


def test_zero_residual_set_takes_the_recoverability():
    """A residual set of zeros: phi = inf, and that linear takes the whole
    recoverability share of its window."""
    size, phi = ranks.salience([3.0, 1.0, 0.0, 0.0], 0.01)
    assert size == 2 and math.isinf(phi)
    got = ranks.window_ranks([[3.0, 1.0, 0.0, 0.0], [1.0] * 8], [1.0, 1.0], 1.0, 4.0, (0, 1, 2, 4), 8,
                             continuous=True)
    assert got == [4.0, 0.0]     # r~ = (4, 0): its 2 salient components, then its 2 residual ones


def _lambda_share(weights, caps, budget):
    """Independent route to proportional sharing with caps: a_i = min(cap_i,
    lam w_i) with sum a = budget, lam found by bisection."""
    lo, hi = 0.0, 1.0
    f = lambda lam: sum(min(c, lam * w) for w, c in zip(weights, caps))
    while f(hi) < budget:
        hi *= 2.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        lo, hi = (mid, hi) if f(mid) < budget else (lo, mid)
    return [min(c, hi * w) for w, c in zip(weights, caps)]


def test_proportional_sharing_matches_the_capped_proportional_solution():
    g = np.random.default_rng(5)
    for _ in range(200):
        n = int(g.integers(1, 9))
        w = list(g.random(n) * (g.random(n) > 0.2))
        caps = list(np.floor(g.random(n) * 50))
        budget = float(g.random() * sum(caps)) if sum(caps) > 0 else 0.0
        if sum(x for x, c in zip(w, caps) if c > 0) == 0:
            continue
        reachable = sum(c for x, c in zip(w, caps) if x > 0)
        budget = min(budget, reachable)
        got = ranks._proportional(w, caps, budget)
        want = _lambda_share([x if c > 0 else 0.0 for x, c in zip(w, caps)], caps, budget)
        np.testing.assert_allclose(got, want, rtol=1e-9, atol=1e-9)


def _window(g, n):
    sig, sens = [], []
    for _ in range(n):
        L = int(g.integers(3, 300))
        base = np.sort(g.random(L))[::-1] * 0.1
        knee = int(g.integers(0, min(L, 40)))
        base[:knee] += g.random() * 2.0 * np.linspace(1.0, 0.5, knee)   # planted salient head
        sig.append(np.sort(base)[::-1].astype(np.float32))
        sens.append(float(g.random()) if g.random() > 0.1 else 0.0)
    return sig, sens


def test_two_stage_allocation_invariants():
    g = np.random.default_rng(7)
    for _ in range(200):
        n = int(g.integers(1, 9))
        sig, sens = _window(g, n)
        r_std, ls = float(g.random() * 200), float(g.random())
        cont = ranks.window_ranks(sig, sens, ls, r_std, LEVELS, 256, continuous=True)
        sal, phi = zip(*[ranks.salience(s, 0.01) for s in sig])
        assert not any(math.isinf(p) for p in phi)
        total = ls * r_std
        # linears with a positive continuous rank: positive sensitivity (or all zero)
        pos = [i for i in range(n) if sens[i] > 0] if any(sens) else list(range(n))
        assert sum(cont) == pytest.approx(min(total, sum(len(sig[i]) for i in pos)), rel=1e-9, abs=1e-9)
        for i in range(n):
            assert -1e-12 <= cont[i] <= len(sig[i]) + 1e-9
            assert i in pos or cont[i] == 0.0
        if total <= sum(sal[i] for i in pos):     # the budget fits their salient sets: nothing residual
            for i in range(n):
                assert cont[i] <= sal[i] + 1e-9
        out = ranks.window_ranks(sig, sens, ls, r_std, LEVELS, 256)
        assert all(r in LEVELS and r <= len(sig[i]) for i, r in enumerate(out))


def test_align_nearest_level_ties_down_and_caps():
    lv = [0, 8, 16, 32]
    assert ranks.align(3.99, lv, 32) == 0 and ranks.align(4.0, lv, 32) == 0 and ranks.align(4.01, lv, 32) == 8
    assert ranks.align(24.0, lv, 32) == 16 and ranks.align(100.0, lv, 32) == 32 and ranks.align(100.0, lv, 20) == 16


def test_layer_scores_closed_form():
    D = [0.5, 2.0, 1.0, 2.0, 0.25]
    # top 2: layers 1 and 3 (D = 2); the others D / 2
    assert ranks.layer_scores(D, 2) == [0.25, 1.0, 0.5, 1.0, 0.125]
    # top 3 reaches the tie-free layer 2 (D = 1): others D / 1
    assert ranks.layer_scores(D, 3) == [0.5, 1.0, 1.0, 1.0, 0.25]
    assert ranks.layer_scores([0.0, 0.0, 3.0], 2) == [1.0, 1.0, 1.0]


def test_library_allocator_equals_oracle():
    """cl_allocate_ranks (host code in the library) against the oracle on
    random windows with planted knees: the same ranks, exactly."""
    g = np.random.default_rng(11)
    for t in range(400):
        n = int(g.integers(1, 9))
        sig, sens = _window(g, n)
        r_std, ls = float(g.random() * 300), float(g.random() * 1.5)
        r_max = int(g.choice([32, 128, 256]))
        tau = float(g.choice([0.0, 0.01, 0.05]))
        want = ranks.window_ranks(sig, sens, ls, r_std, LEVELS, r_max, tau)
        got = cl.allocate_ranks(sig, sens, ls, r_std, LEVELS, r_max, tau)
        assert got == want, (t, got, want)


def test_library_layer_scores_equal_oracle():
    g = np.random.default_rng(13)
    for _ in range(100):
        L = int(g.integers(1, 60))
        D = list(np.round(g.random(L) * 4, 1))           # rounded: ties happen
        K = int(g.integers(1, L + 1))
        assert cl.layer_sensitivity(D, K) == ranks.layer_scores(D, K)


def test_allocator_validation():
    lib = cl.lib()
    s = np.array([3.0, 2.0, 1.0], dtype=np.float32)
    sp = (ctypes.c_void_p * 1)(s.ctypes.data)

    def call(n=1, ln=3, sens=1.0, ls=1.0, r_std=16.0, levels=(0, 8, 16), r_max=16, tau=0.01, sarr=None):
        if sarr is not None:
            sp[0] = sarr.ctypes.data
        lv = (ctypes.c_int32 * len(levels))(*levels)
        return lib.cl_allocate_ranks(n, sp, (ctypes.c_int32 * 1)(ln), (ctypes.c_double * 1)(sens), ls, r_std, lv,
                                     len(levels), r_max, tau, (ctypes.c_int32 * 1)())

    assert call() == cl.CL_OK
    assert call(n=0) == cl.CL_EINVAL and call(n=65) == cl.CL_EINVAL
    assert call(ln=0) == cl.CL_EINVAL
    assert call(sens=-1.0) == cl.CL_EINVAL and call(sens=float("nan")) == cl.CL_EINVAL
    assert call(ls=-0.5) == cl.CL_EINVAL and call(r_std=float("inf")) == cl.CL_EINVAL
    assert call(levels=(8, 16)) == cl.CL_EINVAL and b"levels" in lib.cl_last_error()
    assert call(levels=(0, 16, 16)) == cl.CL_EINVAL
    assert call(r_max=-1) == cl.CL_EINVAL and call(tau=-0.1) == cl.CL_EINVAL
    bad = np.array([1.0, 2.0, 0.5], dtype=np.float32)
    assert call(sarr=bad) == cl.CL_EINVAL and b"descending" in lib.cl_last_error()
    out = (ctypes.c_double * 2)()
    assert lib.cl_layer_sensitivity(2, (ctypes.c_double * 2)(1.0, 2.0), 3, out) == cl.CL_EINVAL
    assert lib.cl_layer_sensitivity(0, (ctypes.c_double * 2)(1.0, 2.0), 1, out) == cl.CL_EINVAL
    assert lib.cl_layer_sensitivity(2, (ctypes.c_double * 2)(1.0, -2.0), 1, out) == cl.CL_EINVAL
