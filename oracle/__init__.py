"""Plain fp64 CPU oracle for the error-compensated quantized linear layer.

TEST INFRASTRUCTURE ONLY.  This package is the slow, obviously-correct
definition that the HIP kernels are checked against.  Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it.  It shares no code with ``paper_2605_05819_amd`` (the product path),
and the product path never calls it.

What it computes (HCInfer, arXiv 2605.05819):

* Section 4.1 (Theoretical Framework): a linear layer ``Y = X W`` is replaced by
  the quantized backbone plus a low-rank correction of the quantization error,
  ``Y ~= X W_hat + (X A_r) B_r`` with ``A_r, B_r`` taken from the SVD of
  ``Delta W = W - W_hat``.  This package uses column vectors and stores the
  weight as ``d_out x d_in``, so the same operation reads
  ``y = W_hat x + B[:, :r] (A[:r, :] x)``.
* Section 5.1 (Experimental Setup): the backbone is a GPTQ low-bit weight.  With
  no calibration data the GPTQ update reduces to round-to-nearest on an
  asymmetric group-wise grid, which is what :mod:`oracle.quant` implements.
* Appendix B.2: the Eckart-Young-Mirsky theorem fixes the error of the rank-r
  truncation, which the tests use as a pin.
* Section 4.2.2 / Appendix A.1 (cross-expert reorganisation): for a MoE layer
  only the routed experts' backbone and compensation factors enter the result;
  :mod:`oracle.moe` is the literal per-(token, slot) loop.

Modules
-------
quant   -- fp16 rounding, quantize, pack/unpack, dequantize
comp    -- compensation factors from the SVD of the residual
linear  -- the compensated forward (decode and prefill compute the same thing)
moe     -- expert-gathered compensated forward
ranks   -- rank allocation from the residual spectra (Section 4.3, Appendix B.1)
"""

from . import quant, comp, linear, moe, ranks  # noqa: F401
