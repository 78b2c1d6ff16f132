"""Oracle: the error-compensated linear forward.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Section 4.1 writes the compensated layer as ``Y = X W_hat + (X A_r) B_r``.  With
column vectors and the weight stored ``d_out x d_in`` every token ``x_t`` gives

  y_t = W_hat x_t + B[:, :r] (A[:r, :] x_t)

The GPU merge step of the paper's pipeline (Algorithm 1: backbone result plus
the returned compensation) is the ``+``; the compensation worker's inner product
(Algorithm 2) is the bracketed term.  Decode (few tokens) and prefill (many
tokens) compute the same function; only the kernels differ.  Everything is fp64
and unrounded; the caller rounds to the output dtype when it compares.

The gate and up projections of a gated MLP (the Llama and Qwen models the
paper evaluates) read the same input and form one compensation window
(Section 4.2.2, Communication Fusion); their outputs meet elementwise as
``SiLU(g) * u``.  :func:`forward_glu` is that product of two compensated
forwards, unrounded.
"""

import numpy as np

from . import quant


def forward(W_hat, A, B, rank, X):
    """``Y[t] = W_hat @ X[t] + B[:, :rank] @ (A[:rank] @ X[t])`` for ``X`` of
    shape ``[T][d_in]``; returns fp64 ``[T][d_out]``."""
    W_hat = np.asarray(W_hat, dtype=np.float64)
    X = np.asarray(X, dtype=np.float64)
    Y = X @ W_hat.T
    r = int(rank)
    if r > 0:
        A = np.asarray(A, dtype=np.float64)[:r]
        B = np.asarray(B, dtype=np.float64)[:, :r]
        T = X @ A.T
        Y = Y + T @ B.T
    return Y


def forward_packed(Q, scales, zeros, bits, group_size, A, B, rank, X):
    """Unpack + dequantize the packed backbone, then :func:`forward`."""
    X = np.asarray(X)
    W_hat = quant.dequant_packed(Q, scales, zeros, bits, group_size, X.shape[1])
    return forward(W_hat, A, B, rank, X)


def forward_rows(Q, scales, zeros, bits, group_size, A, B, rank, X, rows):
    """:func:`forward_packed` restricted to output rows ``rows`` (for sampled
    checks of full-size layers: each output element depends only on its own
    weight row, its own row of ``B`` and the shared ``A``)."""
    rows = np.asarray(rows)
    Qr = np.asarray(Q)[rows]
    sr = np.asarray(scales)[rows]
    zr = np.asarray(zeros)[rows]
    Br = np.asarray(B)[rows] if int(rank) > 0 else B
    return forward_packed(Qr, sr, zr, bits, group_size, A, Br, rank, X)


def silu(v):
    """``SiLU(v) = v / (1 + e^-v)`` in fp64 (for ``v`` far below zero ``e^-v``
    overflows to inf and the quotient is a signed zero)."""
    v = np.asarray(v, dtype=np.float64)
    with np.errstate(over="ignore"):
        return v / (1.0 + np.exp(-v))


def forward_glu(gate, up, X):
    """``SiLU(g) * u`` with ``g`` and ``u`` the compensated forwards of the
    gate and up linears, each given as ``(W_hat, A, B, rank)``; fp64
    ``[T][d_out]``."""
    return silu(forward(*gate, X)) * forward(*up, X)
