"""Oracle: sensitivity-aware rank allocation from the residual spectra.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Section 4.3 and Appendix B.1.  For each linear ``i`` of a compensation window
with singular values ``sigma_i`` (descending) of its residual:

1. ``hat_sigma = sigma / sigma_1``; second differences
   ``k_j = hat_sigma_{j-1} - 2 hat_sigma_j + hat_sigma_{j+1}`` at the interior
   indices; ``r_i = argmax_j k_j``.  If ``max k > tau`` the salient set is
   ``{1..r_i}`` and ``phi_i`` the ratio of the salient to the residual mean,
   else the salient set is empty and ``phi_i = 1``.
2. ``V_i = phi_i / sum_W phi``; ``S_i = D_i / sum_W D``;
   ``P_i = Norm_W(V_i S_i) * S_l``; ``r~_i = P_i * r_std``.
3. Two stages: the window's total ``sum r~`` goes to the salient sets in
   proportion to ``r~`` (none past its size); if it exceeds their total, the
   rest goes to the residual sets the same way.
4. ``Align``: nearest admissible level.

Where the paper leaves a choice open this follows the readings listed with
the design notes: index 1 is the first singular value, ``argmax`` takes the
first of equal maxima, "in proportion" means water-filling (a part that
would overflow a set fills it and the rest is shared again among the
others), ``Align`` breaks ties towards the lower level and never exceeds
``min(r_max, len(sigma))``, a residual set of zeros makes ``phi`` infinite
(the window's recoverability then goes, evenly, to such linears only), and
all-zero sensitivities count as equal.  Sums run left to right in float
arithmetic (fp64), one value at a time.
"""

import math


def salience(sigma, tau):
    """(size of the salient set, phi) of one descending spectrum."""
    sigma = [float(v) for v in sigma]
    n = len(sigma)
    if n < 3 or not sigma[0] > 0.0:
        return 0, 1.0
    hat = [v / sigma[0] for v in sigma]
    best, r = -math.inf, 0
    for j in range(2, n):                       # 1-based interior index j = 2 .. n-1
        k = hat[j - 2] - 2.0 * hat[j - 1] + hat[j]
        if k > best:
            best, r = k, j
    if not best > tau:
        return 0, 1.0
    s_sum = 0.0
    for v in sigma[:r]:
        s_sum += v
    r_sum = 0.0
    for v in sigma[r:]:
        r_sum += v
    s_mean, r_mean = s_sum / r, r_sum / (n - r)
    return r, (s_mean / r_mean if r_mean > 0.0 else math.inf)


def _proportional(weights, caps, budget):
    """Share ``budget`` in proportion to ``weights`` with per-part caps."""
    n = len(weights)
    got = [0.0] * n
    open_ = [weights[i] > 0.0 and caps[i] > 0.0 for i in range(n)]
    left = budget
    while left > 0.0:
        wsum = 0.0
        for i in range(n):
            if open_[i]:
                wsum += weights[i]
        if not wsum > 0.0:
            break
        full = [i for i in range(n) if open_[i] and left * weights[i] / wsum >= caps[i] - got[i]]
        if not full:
            for i in range(n):
                if open_[i]:
                    got[i] += left * weights[i] / wsum
            break
        for i in full:
            got[i] = caps[i]
            open_[i] = False
        used = 0.0
        for v in got:
            used += v
        left = budget - used
    return got


def align(x, levels, top):
    """Nearest level not above ``top`` (ties to the lower)."""
    best = levels[0]
    for lv in levels[1:]:
        if lv > top:
            break
        if abs(x - lv) < abs(x - best):
            best = lv
    return best


def window_ranks(sigmas, sens, layer_score, r_std, levels, r_max, tau=0.01, continuous=False):
    """Ranks of one compensation window (or, with ``continuous``, the
    two-stage allocation before alignment)."""
    n = len(sigmas)
    sal, phi = zip(*[salience(s, tau) for s in sigmas])
    lens = [len(s) for s in sigmas]
    n_inf = sum(1 for p in phi if math.isinf(p))
    if n_inf:
        V = [(1.0 / n_inf if math.isinf(p) else 0.0) for p in phi]
    else:
        psum = 0.0
        for p in phi:
            psum += p
        V = [p / psum for p in phi]
    dsum = 0.0
    for d in sens:
        dsum += float(d)
    S = [(float(d) / dsum if dsum > 0.0 else 1.0 / n) for d in sens]
    prod = [V[i] * S[i] for i in range(n)]
    xsum = 0.0
    for v in prod:
        xsum += v
    P = [(prod[i] / xsum * layer_score if xsum > 0.0 else 0.0) for i in range(n)]
    r_cont = [P[i] * r_std for i in range(n)]
    total = 0.0
    for v in r_cont:
        total += v
    stage1 = _proportional(r_cont, [float(c) for c in sal], total)
    used = 0.0
    for v in stage1:
        used += v
    stage2 = _proportional(r_cont, [float(lens[i] - sal[i]) for i in range(n)], total - used)
    cont = [stage1[i] + stage2[i] for i in range(n)]
    if continuous:
        return cont
    return [align(cont[i], list(levels), min(r_max, lens[i])) for i in range(n)]


def layer_scores(D, K):
    """``S_l``: 1 for the K layers of largest ``D`` (ties to the lower index),
    ``D_l / min_{m in top K} D_m`` for the others (1 when that minimum is 0)."""
    order = sorted(range(len(D)), key=lambda l: (-float(D[l]), l))
    top = set(order[:K])
    dmin = min(float(D[l]) for l in top)
    return [1.0 if l in top else (float(D[l]) / dmin if dmin > 0.0 else 1.0) for l in range(len(D))]
