"""Oracle: low-rank compensation factors from the SVD of the quantization error.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Section 4.1 takes the compensation factors from the singular value decomposition
of the residual ``Delta W = W - W_hat``; Appendix B.2 (Eckart-Young-Mirsky) says
the truncated SVD is the best rank-r approximation and that its squared
Frobenius error is the sum of the squared tail singular values.

In the column-vector convention used here (weight stored ``d_out x d_in``):

  E = W - W_hat = U diag(sigma) V^T            (LAPACK, fp64, sigma descending)
  B = U[:, :r_max] diag(sqrt(sigma[:r_max]))   (d_out x r_max)
  A = diag(sqrt(sigma[:r_max])) V^T[:r_max]    (r_max x d_in)

so ``B[:, :r] @ A[:r]`` is the rank-r truncation for every ``r <= r_max`` (the
factors are sorted by descending sigma, so one stored pool serves any prefix
rank, which is how the paper's worker selects a per-matrix rank at run time).

Readings the paper leaves open: the split of sigma between the factors is not
stated -- the symmetric ``sqrt(sigma)`` split keeps both factors in the same
range, which matters once they are stored in fp16; the sign of each singular
pair is fixed so that the largest-magnitude entry of each ``U`` column is
positive (first index on ties), making the factors a function of ``E``.
"""

import numpy as np


def residual(W, W_hat):
    """``E = W - W_hat`` in fp64."""
    return np.asarray(W, dtype=np.float64) - np.asarray(W_hat, dtype=np.float64)


def svd_sorted(E):
    """Thin SVD with the deterministic sign convention described above."""
    U, sigma, Vt = np.linalg.svd(np.asarray(E, dtype=np.float64), full_matrices=False)
    idx = np.argmax(np.abs(U), axis=0)
    sign = np.sign(U[idx, np.arange(U.shape[1])])
    sign[sign == 0] = 1.0
    return U * sign, sigma, Vt * sign[:, None]


def build_compensation(W, W_hat, r_max):
    """Return ``(A, B, sigma)`` in fp64: ``A`` is ``r_max x d_in``, ``B`` is
    ``d_out x r_max`` and ``sigma`` holds every singular value of ``W - W_hat``."""
    E = residual(W, W_hat)
    U, sigma, Vt = svd_sorted(E)
    r_max = int(r_max)
    if r_max > sigma.shape[0]:
        raise ValueError("r_max exceeds min(d_out, d_in)")
    root = np.sqrt(sigma[:r_max])
    A = root[:, None] * Vt[:r_max]
    B = U[:, :r_max] * root[None, :]
    return A, B, sigma


def to_fp16(a):
    """Store a factor as fp16 (round to nearest even, from fp64)."""
    return np.asarray(a, dtype=np.float64).astype(np.float16)
