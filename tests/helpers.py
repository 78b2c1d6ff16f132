"""Shared test helpers: moving seeded numpy inputs to the device, error
metrics and rounding of oracle results to the output dtype."""

import numpy as np
import torch

from oracle import comp, quant

# Relative L2 bound on outputs (fp16/bf16 inputs, fp32 accumulation).
REL_L2_TOL = 1e-3
# Elementwise bound: |got - ref| <= u |ref| + ELEM_TOL * rms(row of ref), with
# ref the unrounded fp64 oracle and u the output dtype's unit roundoff (the
# rounding of a correct result).  A whole-tensor relative L2 lets one wrong
# element among many pass; this does not.  (fp32 accumulation over a few
# thousand terms leaves ~1e-6 of the row scale; dequantized fp16 weight tiles
# of the prefill GEMM ~2e-4.)
ELEM_TOL = 1e-3
UNIT_ROUNDOFF = {torch.float32: 0.0, torch.float16: 2.0 ** -11, torch.bfloat16: 2.0 ** -8}


def rel_l2(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))


def elem_ratio(got, ref, out_dtype=torch.float32, extra=None):
    """Largest |got - ref| / (u |ref| + ELEM_TOL rms(row) + extra) over all
    elements, rows along the last axis (<= 1 passes); a zero reference row
    must be matched exactly.  extra: a further allowed error per element (the
    rounding bound of an arithmetic that rounds intermediate values)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    g2 = got.reshape(-1, ref.shape[-1])
    r2 = ref.reshape(-1, ref.shape[-1])
    rms = np.sqrt(np.mean(r2 * r2, axis=1, keepdims=True))
    allow = UNIT_ROUNDOFF[out_dtype] * (1 + 2.0 ** -10) * np.abs(r2) + ELEM_TOL * rms
    if extra is not None:
        allow = allow + np.asarray(extra, dtype=np.float64).reshape(allow.shape)
    err = np.abs(g2 - r2)
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(allow > 0, err / np.where(allow > 0, allow, 1.0), np.where(err > 0, np.inf, 0.0))
    return float(ratio.max())


def assert_oracle(got, ref, out_dtype=torch.float32, extra=None):
    """got (the kernel's output as float64) against the fp64 oracle: relative
    L2 against the oracle rounded to out_dtype within REL_L2_TOL, and every
    element within the elementwise bound (see elem_ratio)."""
    err = rel_l2(got, round_to(ref, out_dtype))
    worst = elem_ratio(got, ref, out_dtype, extra)
    assert err <= REL_L2_TOL and worst <= 1.0, "rel L2 %.3e (bar %.0e), worst element %.3f of its bound" % (
        err, REL_L2_TOL, worst)
    return err, worst


def round_to(y, dtype):
    """Round fp64 oracle values to the kernel's output dtype (RNE)."""
    y = np.asarray(y, dtype=np.float64)
    if dtype == torch.float32:
        return y
    if dtype == torch.float16:
        return y.astype(np.float16).astype(np.float64)
    t = torch.from_numpy(y.astype(np.float32)).to(torch.bfloat16)  # fp32 -> bf16 RNE
    return t.to(torch.float64).numpy()


def out_to_numpy(y):
    return y.detach().to("cpu").to(torch.float64).numpy()


def dev_u16(bits_u16, dtype, device="cuda"):
    """uint16 bit patterns -> a device tensor of dtype (fp16/bf16)."""
    t = torch.from_numpy(np.ascontiguousarray(bits_u16).view(np.int16))
    return t.view(dtype).to(device)


def dev_f16(a, device="cuda"):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float16)).to(device)


def dev_u32(a, device="cuda"):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.uint32).view(np.int32)).to(device)


def host_u32(t):
    return t.detach().to("cpu").numpy().view(np.uint32)


def host_u16(t):
    return t.detach().to("cpu").view(torch.int16).numpy().view(np.uint16)


def oracle_layer(W, bits, G, r_max):
    """Oracle-quantized backbone plus fp16 compensation factors from the SVD."""
    Q, s, z = quant.quantize_pack(W, bits, G)
    W_hat = quant.dequant_packed(Q, s, z, bits, G, W.shape[1])
    A, B, sigma = comp.build_compensation(W, W_hat, r_max)
    return Q, s, z, comp.to_fp16(A), comp.to_fp16(B), sigma


def fp16_tile_bound(W_hat, X, A=None, B=None, rank=0):
    """Rounding bound of a product whose weights s (q - z) and low-rank
    activations T = X A^T are rounded to fp16 before an exactly accumulated
    contraction (the prefill GEMM's dequantized tiles): per output element
    2^-11 (sum_k |W_hat[n, k] x[m, k]| + sum_i |T[m, i] B[n, i]|), with a
    1 % margin for the fp32 accumulation."""
    u = 2.0 ** -11
    b = np.abs(np.asarray(X, np.float64)) @ np.abs(np.asarray(W_hat, np.float64)).T
    if rank:
        T = np.asarray(X, np.float64) @ np.asarray(A[:rank], np.float64).T
        b = b + np.abs(T) @ np.abs(np.asarray(B[:, :rank], np.float64)).T
    return 1.01 * u * b
