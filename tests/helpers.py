"""Shared test helpers: moving seeded numpy inputs to the device, error
metrics and rounding of oracle results to the output dtype."""

import numpy as np
import torch

from oracle import comp, quant

# Relative L2 bound on outputs (fp16/bf16 inputs, fp32 accumulation).
REL_L2_TOL = 1e-3


def rel_l2(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))


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
