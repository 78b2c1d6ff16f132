"""cl_linear_decode_noalloc (the decode entry point that allocates nothing:
its workspace is the library's per-device scratch array) against
cl_linear_decode on the same inputs, through the C ABI: two calls in a row,
the second with a smaller input, bit for bit equal to the workspace call and
within the oracle bar; the scratch keeps the first call's contents when the
second runs, and nothing in it needs to start at zero."""

import numpy as np
import pytest
import torch

from oracle import linear, quant
from paper_2605_05819_amd import cl, workloads as wl
from tests.helpers import assert_oracle, dev_f16, dev_u16, dev_u32, out_to_numpy

pytestmark = pytest.mark.gpu


def _case(d_out, d_in, bits, G, r_max, rank, T, seed):
    W = wl.weight((d_out, d_in), 16, seed)
    Q, s, z = quant.quantize_pack(W, bits, G)
    A, B = wl.standin_factors(d_out, d_in, r_max, 16, seed)
    w = cl.QWeight(dev_u32(Q), dev_f16(s), dev_f16(z), d_out, d_in, bits, G)
    c = cl.LowRank(dev_f16(A), dev_f16(B), r_max, rank)
    x = wl.activation((T, d_in), 16, seed)
    return w, c, x, (Q, s, z, A, B)


def test_noalloc_equals_decode_on_two_calls_second_smaller():
    # first: 16 tokens through a 4096 x 14336 matrix at rank 128 (MFMA
    # backbone, the down projection's shape); second: one token through
    # 1000 x 2048 at rank 17 (dot2 backbone), a much smaller input
    cases = [(4096, 14336, 4, 128, 128, 128, 16, 1), (1000, 2048, 4, 128, 32, 17, 1, 2)]
    for d_out, d_in, bits, G, r_max, rank, T, seed in cases:
        w, c, x, (Q, s, z, A, B) = _case(d_out, d_in, bits, G, r_max, rank, T, seed)
        xd = dev_u16(x.bits, torch.float16)
        y_ws = cl.linear_decode(w, c, xd, out_dtype=torch.float32)
        y_na = cl.linear_decode_noalloc(w, c, xd, out_dtype=torch.float32)
        torch.cuda.synchronize()
        assert torch.equal(y_na, y_ws), (d_out, d_in, T)
        rows = np.arange(d_out) if d_out <= 1000 else np.random.default_rng(seed).choice(d_out, 200, replace=False)
        ref = linear.forward_rows(Q, s, z, bits, G, A, B, rank, x.values, rows)
        assert_oracle(out_to_numpy(y_na)[:, rows], ref)


def test_noalloc_repeated_calls_and_output_dtypes():
    """The same small call three times in a row (the scratch holding the
    previous call's values each time) and in every output dtype."""
    w, c, x, (Q, s, z, A, B) = _case(700, 1024, 2, 64, 16, 16, 5, 3)
    xd = dev_u16(x.bits, torch.float16)
    for out in (torch.float32, torch.float16, torch.bfloat16, torch.float32):
        y_ws = cl.linear_decode(w, c, xd, out_dtype=out)
        y_na = cl.linear_decode_noalloc(w, c, xd, out_dtype=out)
        torch.cuda.synchronize()
        assert torch.equal(y_na, y_ws), out
