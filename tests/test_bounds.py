"""The test harness's parity bounds (CPU): the elementwise bound catches one
wrong element that the whole-tensor relative L2 bar lets through, and the
fp16-tile rounding bound covers a simulated fp16-tile product."""

import numpy as np
import torch

from tests.helpers import REL_L2_TOL, elem_ratio, fp16_tile_bound, rel_l2, round_to


def test_single_element_error_is_caught():
    g = np.random.default_rng(0)
    ref = g.standard_normal((4, 16384))
    got = ref.copy()
    got[2, 777] *= 1.1
    assert rel_l2(got, ref) <= REL_L2_TOL
    assert elem_ratio(got, ref) > 1.0
    assert elem_ratio(ref, ref) == 0.0


def test_rounded_outputs_sit_inside_the_bound():
    g = np.random.default_rng(1)
    ref = g.standard_normal((8, 1000)) * np.exp(g.standard_normal((8, 1000)))
    for dt in (torch.float16, torch.bfloat16):
        assert elem_ratio(round_to(ref, dt), ref, dt) <= 1.0
    zero = np.zeros((2, 5))
    assert elem_ratio(zero, zero) == 0.0
    assert elem_ratio(zero + 1e-30, zero) == float("inf")


def test_fp16_tile_bound_covers_fp16_weights():
    g = np.random.default_rng(2)
    W = g.standard_normal((64, 512)) * 0.01
    X = g.standard_normal((16, 512))
    W16 = W.astype(np.float16).astype(np.float64)
    err = np.abs(X @ W16.T - X @ W.T)
    assert (err <= fp16_tile_bound(W, X)).all()
