"""cl_quantize_pack and cl_dequantize against the oracle: bit-exact codes,
scales, zeros and dequantized values (Section 5.1 backbone quantizer, RTN
reading of GPTQ without calibration data)."""

import numpy as np
import pytest
import torch

from oracle import quant
from paper_2605_05819_amd import cl, workloads as wl
from tests.helpers import dev_u32, dev_f16, host_u16, host_u32

pytestmark = pytest.mark.gpu


def _adversarial(bits, G, rows):
    """Rows that stress the rounding rules: exact ties, constant and zero
    groups, one-sided groups, clamped maxima, tiny and huge magnitudes."""
    g = np.random.default_rng(1234 + bits)
    qmax = (1 << bits) - 1
    d_in = 4 * G
    W = (0.02 * g.standard_normal((rows, d_in))).astype(np.float64)
    step = 2.0 ** -8
    # exact half-steps on a power-of-two grid -> ties to even
    W[0, :G] = step * (np.resize(np.arange(-3, qmax - 2) + 0.5, G))
    W[0, 0], W[0, 1] = -3 * step, (qmax - 3) * step
    W[1, :G] = 0.0                                  # all-zero group
    W[1, G:2 * G] = 0.37                            # constant positive group
    W[1, 2 * G:3 * G] = -0.01                       # constant negative group
    W[2, :G] = np.abs(W[2, :G])                     # one-sided
    W[2, G:2 * G] = -np.abs(W[2, G:2 * G])
    W[3, :G] *= 1e-6                                # subnormal-range scale
    W[3, G:2 * G] *= 1e-9                           # scale rounds to 0 -> held at 2^-24
    W[4, :G] *= 1e5                                 # huge values: scale beyond fp16 -> 65504
    return W.astype(np.float32)


@pytest.mark.parametrize("bits,G", [(4, 128), (2, 64), (4, 32), (2, 128), (3, 128), (3, 32)])
def test_quantize_pack_bit_exact(bits, G):
    rows = 37                                       # ragged: not a multiple of anything
    W = np.concatenate([_adversarial(bits, G, 8),
                        wl.weight((rows - 8, 4 * G), 0, 0, bits, G)], axis=0)
    w = cl.quantize_pack(torch.from_numpy(W).cuda(), bits, G)
    torch.cuda.synchronize()
    Q, s, z = quant.quantize_pack(W, bits, G)
    np.testing.assert_array_equal(host_u32(w.q), Q)
    np.testing.assert_array_equal(host_u16(w.scales), s.view(np.uint16))
    np.testing.assert_array_equal(host_u16(w.zeros), z.view(np.uint16))


def test_quantize_pack_llama_gate_rows_bit_exact():
    """Full 14336 x 4096 gate matrix quantized on the GPU; rows sampled across
    the whole matrix (quantization is row-independent) checked bit-exactly."""
    W = wl.weight((14336, 4096), 1, 0, 4)
    w = cl.quantize_pack(torch.from_numpy(W).cuda(), 4, 128)
    torch.cuda.synchronize()
    rows = np.r_[0:3, np.random.default_rng(0).choice(14336, 60, replace=False), 14333:14336]
    Q, s, z = quant.quantize_pack(W[rows], 4, 128)
    np.testing.assert_array_equal(host_u32(w.q)[rows], Q)
    np.testing.assert_array_equal(host_u16(w.scales)[rows], s.view(np.uint16))
    np.testing.assert_array_equal(host_u16(w.zeros)[rows], z.view(np.uint16))


@pytest.mark.parametrize("bits,G", [(4, 128), (2, 64), (3, 128), (3, 32)])
def test_dequantize_exact(bits, G):
    W = wl.weight((50, 512), 0, 3, bits)
    Q, s, z = quant.quantize_pack(W, bits, G)
    w = cl.QWeight(dev_u32(Q), dev_f16(s), dev_f16(z), 50, 512, bits, G)
    got = cl.dequantize(w).cpu().numpy().astype(np.float64)
    np.testing.assert_array_equal(got, quant.dequant_packed(Q, s, z, bits, G, 512))


def test_quantize_pack_3bit_llama_rows_bit_exact():
    """3-bit codes (32 in 3 words, two of them straddling words) of a full
    14336 x 4096 matrix quantized on the GPU, sampled rows bit-exact."""
    W = wl.weight((14336, 4096), 7, 0, 4)
    w = cl.quantize_pack(torch.from_numpy(W).cuda(), 3, 128)
    torch.cuda.synchronize()
    assert tuple(w.q.shape) == (14336, 384)
    rows = np.r_[0:2, np.random.default_rng(3).choice(14336, 40, replace=False), 14334:14336]
    Q, s, z = quant.quantize_pack(W[rows], 3, 128)
    np.testing.assert_array_equal(host_u32(w.q)[rows], Q)
    np.testing.assert_array_equal(host_u16(w.scales)[rows], s.view(np.uint16))
    np.testing.assert_array_equal(host_u16(w.zeros)[rows], z.view(np.uint16))
