"""Oracle: group-wise asymmetric low-bit quantization, packing and dequantization.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The paper quantizes its backbones with GPTQ (Section 5.1, Experimental Setup;
INT4 for the MoE model, INT3 for the dense one).  GPTQ walks the columns of a
group, rounds each to the nearest point of an asymmetric min/max grid and feeds
the rounding error back into the not-yet-quantized columns through the inverse
calibration Hessian.  The synthetic workloads here have no calibration data; with
an identity Hessian the feedback term vanishes and GPTQ is plain
round-to-nearest on the same grid.  That special case is what this module writes
out, in fp64:

  for each row ``o`` and each group ``g`` of ``G`` consecutive input columns
    lo  = min(min_c w, 0),   hi = max(max_c w, 0)         (grid contains 0)
    if hi == lo:  lo, hi = -1, +1                         (all-zero group)
    s   = (hi - lo) / (2**b - 1)                          (fp64)
    s16 = fp16 round-to-nearest-even of s, kept within [2**-24, 65504]
    z   = clamp(rint(-lo / s16), 0, 2**b - 1)             (integer zero point)
    q_c = clamp(rint(w_c / s16) + z, 0, 2**b - 1)         (rint: half to even)
  dequant:  w_hat_c = s16 * (q_c - z)

Codes are computed against the *stored* fp16 scale, so the kernel that
dequantizes sees exactly the grid the codes were chosen on.  Packing is
LSB-first over the row's bit string: the code of column ``c`` occupies bits
``b c .. b c + b - 1`` of the row, and bit ``i`` of the row is bit ``i % 32`` of
its 32-bit word ``i // 32``.  For b = 2 and 4 the code of column ``c`` is then
in word ``c // (32 // b)`` at bit offset ``b * (c % (32 // b))``; for b = 3 (the
paper's INT3 backbone) 32 codes fill 3 words and the codes of columns
``32 k + 10`` and ``32 k + 21`` straddle two words.

Readings the paper leaves open (fixed here, listed in the design notes): RTN for
GPTQ without calibration data; 0 inside the grid; the degenerate all-equal
group; fp16 scale rounded once, directly from fp64; the integer zero point
stored exactly in fp16; the clamp after ``rint`` (needed because
``s16 < s`` can push the group maximum one step past ``2**b - 1``); a scale
that rounds to 0 or overflows fp16 is held at the nearest finite positive fp16.
"""

import numpy as np

FP16_MIN_SUBNORMAL = 2.0 ** -24
FP16_MAX = 65504.0


def fp16_rne(a):
    """Round fp64 values to the nearest fp16, ties to even, in one step.

    numpy converts float64 -> float16 directly (no intermediate float32), so a
    single correctly-rounded step is what ``astype`` gives; the tests pin this
    against a brute-force nearest-neighbour search over the fp16 grid.
    """
    return np.asarray(a, dtype=np.float64).astype(np.float16)


def quantize(W, bits, group_size):
    """Quantize ``W`` (``d_out x d_in``, float32 values) group-wise along d_in.

    Returns ``(codes, scales, zeros)``: codes as int64 ``[d_out][d_in]``,
    scales and zeros as float16 ``[d_out][d_in // group_size]``.
    """
    W = np.asarray(W)
    d_out, d_in = W.shape
    G = int(group_size)
    if d_in % G:
        raise ValueError("d_in must be a multiple of the group size")
    qmax = (1 << bits) - 1
    Wg = W.astype(np.float64).reshape(d_out, d_in // G, G)

    lo = np.minimum(Wg.min(axis=2), 0.0)
    hi = np.maximum(Wg.max(axis=2), 0.0)
    flat = hi == lo
    lo = np.where(flat, -1.0, lo)
    hi = np.where(flat, 1.0, hi)

    s = (hi - lo) / qmax
    s16 = fp16_rne(s).astype(np.float64)
    s16 = np.clip(s16, FP16_MIN_SUBNORMAL, FP16_MAX)

    z = np.clip(np.rint(-lo / s16), 0, qmax)
    q = np.clip(np.rint(Wg / s16[:, :, None]) + z[:, :, None], 0, qmax)

    codes = q.reshape(d_out, d_in).astype(np.int64)
    return codes, s16.astype(np.float16), z.astype(np.float16)


ROW_BLOCK = 256   # rows per step of pack/unpack (bounds the bit-string temporaries)


def pack(codes, bits):
    """Pack integer codes ``[d_out][d_in]`` LSB-first into uint32 words: the
    row's codes are written out as a bit string (code ``c`` at bits
    ``bits * c ..``, least significant bit first) that is cut into 32-bit
    words, least significant bit first.  ``d_in * bits`` must be a multiple
    of 32."""
    codes = np.asarray(codes, dtype=np.int64)
    d_out, d_in = codes.shape
    if (d_in * bits) % 32:
        raise ValueError("d_in * bits must be a multiple of 32")
    if codes.min(initial=0) < 0 or codes.max(initial=0) >= (1 << bits):
        raise ValueError("codes out of range")
    out = np.empty((d_out, d_in * bits // 32), dtype=np.uint32)
    for r0 in range(0, d_out, ROW_BLOCK):
        c = codes[r0:r0 + ROW_BLOCK]
        n = c.shape[0]
        # bit j of code c is bit bits * c + j of the row
        bitstr = ((c[:, :, None] >> np.arange(bits)) & 1).reshape(n, d_in * bits)
        # bit i of the row is bit i % 32 of word i // 32
        w = bitstr.reshape(n, d_in * bits // 32, 32).astype(np.uint64)
        out[r0:r0 + n] = (w << np.arange(32, dtype=np.uint64)).sum(axis=2, dtype=np.uint64).astype(np.uint32)
    return out


def unpack(Q, bits, d_in):
    """Inverse of :func:`pack`: uint32 ``[d_out][d_in*bits/32]`` -> int64
    codes.  Code ``c`` starts at bit ``p = bits * c`` of the row: read the
    64-bit value of words ``p // 32`` (low) and ``p // 32 + 1`` (high),
    shift it right by ``p % 32`` and keep ``bits`` bits (a code of at most
    32 bits never spans more than those two words)."""
    Q = np.asarray(Q, dtype=np.uint32)
    d_out, nw = Q.shape
    p = bits * np.arange(d_in)
    w0 = p // 32
    w1 = np.minimum(w0 + 1, nw - 1)
    has_hi = (w0 + 1 < nw).astype(np.uint64)
    shift = (p % 32).astype(np.uint64)
    mask = np.uint64((1 << bits) - 1)
    out = np.empty((d_out, d_in), dtype=np.int64)
    for r0 in range(0, d_out, ROW_BLOCK):
        q = Q[r0:r0 + ROW_BLOCK].astype(np.uint64)
        v = (q[:, w0] | ((q[:, w1] * has_hi) << np.uint64(32))) >> shift
        out[r0:r0 + ROW_BLOCK] = (v & mask).astype(np.int64)
    return out


def dequant(codes, scales, zeros, group_size):
    """``w_hat = s16 * (q - z)`` in fp64 (exact: every value fits in fp32 too)."""
    codes = np.asarray(codes, dtype=np.float64)
    g = np.arange(codes.shape[1]) // int(group_size)
    s = np.asarray(scales, dtype=np.float64)[:, g]
    z = np.asarray(zeros, dtype=np.float64)[:, g]
    return s * (codes - z)


def quantize_pack(W, bits, group_size):
    """Quantize then pack: returns ``(Q uint32, scales fp16, zeros fp16)``."""
    codes, s, z = quantize(W, bits, group_size)
    return pack(codes, bits), s, z


def dequant_packed(Q, scales, zeros, bits, group_size, d_in):
    """Unpack then dequantize a packed weight to fp64 ``[d_out][d_in]``."""
    return dequant(unpack(Q, bits, d_in), scales, zeros, group_size)
