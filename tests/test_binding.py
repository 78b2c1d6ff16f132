"""The Python binding checks every tensor before a pointer crosses the C ABI
(CPU): wrong dtypes (int64 routing ids from torch.topk), shapes (a 1-D
activation, a last dimension that is not d_in, per-slot inputs that do not
match the routing), non-contiguous views and host tensors raise ValueError
instead of reaching the kernels."""

import pytest
import torch

from paper_2605_05819_amd import cl


def _qweight(d_out=64, d_in=256, bits=4, G=128):
    return cl.QWeight(torch.zeros((d_out, d_in * bits // 32), dtype=torch.int32),
                      torch.zeros((d_out, d_in // G), dtype=torch.float16),
                      torch.zeros((d_out, d_in // G), dtype=torch.float16), d_out, d_in, bits, G)


def _experts(E=4, d_out=32, d_in=256, r_max=8):
    return cl.MoeExperts(torch.zeros((E, d_out, d_in // 8), dtype=torch.int32),
                         torch.zeros((E, d_out, d_in // 128), dtype=torch.float16),
                         torch.zeros((E, d_out, d_in // 128), dtype=torch.float16),
                         torch.zeros((E, r_max, d_in), dtype=torch.float16),
                         torch.zeros((E, d_out, r_max), dtype=torch.float16),
                         torch.zeros((E,), dtype=torch.int32), E, d_out, d_in, 4, 128, r_max)


def _raises(fn, needle):
    with pytest.raises(ValueError) as e:
        fn()
    assert needle in str(e.value), str(e.value)


def test_decode_rejects_bad_activations():
    w = _qweight()
    x = torch.zeros((2, 256), dtype=torch.float16)
    _raises(lambda: cl.linear_decode(w, None, x.float()), "x must have dtype")
    _raises(lambda: cl.linear_decode(w, None, torch.zeros(256, dtype=torch.float16)), "x must be")
    _raises(lambda: cl.linear_decode(w, None, torch.zeros((2, 255), dtype=torch.float16)), "x must be")
    _raises(lambda: cl.linear_decode(w, None, torch.zeros((256, 4), dtype=torch.float16).t()), "contiguous")
    _raises(lambda: cl.linear_decode(w, None, x), "on the GPU")


def test_decode_rejects_bad_weights_factors_and_outputs():
    w = _qweight()
    x = torch.zeros((2, 256), dtype=torch.float16)
    bad = cl.QWeight(w.q.long(), w.scales, w.zeros, 64, 256, 4, 128)
    _raises(lambda: cl.linear_decode(bad, None, x), "w.q must have dtype")
    short = cl.QWeight(w.q[:10], w.scales, w.zeros, 64, 256, 4, 128)
    _raises(lambda: cl.linear_decode(short, None, x), "w.q must have shape")
    c = cl.LowRank(torch.zeros((8, 255), dtype=torch.float16), torch.zeros((64, 8), dtype=torch.float16), 8, 4)
    _raises(lambda: cl.linear_decode(w, c, x), "c.A must have shape")
    y = torch.zeros((2, 63), dtype=torch.float16)
    _raises(lambda: cl.linear_decode(w, None, x, y=y), "y must have shape")
    _raises(lambda: cl.linear_prefill(w, None, x, Y=torch.zeros((2, 64), dtype=torch.int16)), "Y must have dtype")


def test_window_and_glu_check_every_linear():
    w = _qweight()
    x = torch.zeros((1, 256), dtype=torch.float16)
    _raises(lambda: cl.linear_decode_window([w, _qweight(d_in=512)], None, x), "share d_in")
    _raises(lambda: cl.linear_decode_glu([w], None, x), "pairs")


def test_moe_rejects_int64_ids_and_mismatched_inputs():
    ex = _experts()
    x = torch.zeros((3, 256), dtype=torch.float16)
    ids64 = torch.zeros((3, 2), dtype=torch.int64)                      # what torch.topk returns
    _raises(lambda: cl.moe_linear_decode(ex, x, ids64), "topk_ids must have dtype torch.int32")
    ids = torch.zeros((3, 2), dtype=torch.int32)
    _raises(lambda: cl.moe_linear_decode(ex, torch.zeros((3, 3, 256), dtype=torch.float16), ids), "x must be")
    _raises(lambda: cl.moe_linear_decode(ex, torch.zeros((3, 128), dtype=torch.float16), ids), "x must be")
    _raises(lambda: cl.moe_linear_decode(ex, x, ids.t()), "contiguous")
    _raises(lambda: cl.moe_linear_decode_window([ex], x, ids, slot_ranks=[torch.zeros((2, 3), dtype=torch.int32)]),
            "slot_ranks[0] must have shape")
    bad = _experts()
    bad.ranks = torch.zeros((5,), dtype=torch.int32)
    _raises(lambda: cl.moe_linear_decode(bad, x, ids), "ranks must have shape")
    _raises(lambda: cl.moe_linear_decode(ex, x, ids), "on the GPU")
