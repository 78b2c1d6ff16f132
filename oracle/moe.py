"""Oracle: expert-gathered compensated forward for a MoE layer.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Section 4.2.2 (cross-expert pipeline reorganisation) and Appendix A.1 (MoE
windows) group the same projection of every activated expert into one step; for
a token only its routed experts' weights and compensation factors enter.  With a
routing table ``ids[T][k]`` the result is, slot by slot,

  y[t][j] = W_hat_e x + B_e[:, :r_e] (A_e[:r_e] x),   e = ids[t][j]

where ``x`` is the token's input (shared by its slots, e.g. gate/up) or the
slot's own input (e.g. down, whose input is that expert's hidden state), and
``r_e`` is the expert's compensation rank.  Written as the literal loop.
"""

import numpy as np

from . import linear


def forward(experts, ranks, X, ids, x_per_slot, slot_ranks=None):
    """``experts[e] = (W_hat_e, A_e, B_e)`` (fp64-convertible arrays);
    ``ranks[e]`` ints; ``X`` is ``[T][d_in]`` (shared) or ``[T][k][d_in]``
    (per slot); ``ids`` is ``[T][k]``; ``slot_ranks`` (optional ``[T][k]``)
    replaces ``ranks[e]`` slot by slot (Section 4.3.3: each routed expert's
    compensation follows its routing weight).  Returns fp64
    ``[T][k][d_out]``."""
    ids = np.asarray(ids)
    T, k = ids.shape
    d_out = np.asarray(experts[int(ids[0, 0])][0]).shape[0]
    Y = np.zeros((T, k, d_out), dtype=np.float64)
    for t in range(T):
        for j in range(k):
            e = int(ids[t, j])
            W_hat, A, B = experts[e]
            x = X[t, j] if x_per_slot else X[t]
            r = int(ranks[e]) if slot_ranks is None else int(slot_ranks[t][j])
            Y[t, j] = linear.forward(W_hat, A, B, r, np.asarray(x)[None, :])[0]
    return Y


def forward_rows(packed, ranks, X, ids, x_per_slot, rows, bits, group_size):
    """:func:`forward` on output rows ``rows`` only, from packed experts
    ``packed[e] = (Q_e, scales_e, zeros_e, A_e, B_e)``: each slot's rows come
    from :func:`linear.forward_rows` of its expert.  Returns fp64
    ``[T][k][len(rows)]``."""
    ids = np.asarray(ids)
    T, k = ids.shape
    rows = np.asarray(rows)
    Y = np.zeros((T, k, len(rows)), dtype=np.float64)
    for t in range(T):
        for j in range(k):
            Q, s, z, A, B = packed[int(ids[t, j])]
            x = X[t, j] if x_per_slot else X[t]
            Y[t, j] = linear.forward_rows(Q, s, z, bits, group_size, A, B, int(ranks[int(ids[t, j])]),
                                          np.asarray(x)[None, :], rows)[0]
    return Y
