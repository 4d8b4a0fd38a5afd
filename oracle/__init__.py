"""CPU oracle for the LUQ 4-bit backward hot path (test infrastructure only).

This package is a plain, slow, deliberately unoptimised restatement of what the
method computes, written from the paper "Accurate Neural Training with 4-bit
Matrix Multiplications at Standard Formats" (Chmiel et al., arXiv 2112.10769):

* ``philox``  -- Philox4x32-10 counter-based generator (Salmon et al., SC'11),
                 the source of the stochastic-rounding uniforms.  The paper
                 only says its quantizer was a CUDA kernel; the generator is
                 this implementation's choice.
* ``luq``     -- logarithmic unbiased quantization of neural gradients
                 (Section 4: stochastic underflow, Eq. StochasticPruning;
                 underflow threshold, Eq. alpha; logarithmic SR,
                 Eq. unbiasedFpQ; their composition X_q = Q_alpha(T_alpha(x)))
                 and the multi-sample average of Section 5.1 (SMP), as planes
                 or as the per-element sum of the decoded samples.
* ``int4``    -- uniform INT4 round-to-nearest quantizer for weights and
                 activations (Section 3.3 rounding rule; Appendix A.1 scale
                 alpha = Delta / (2^b - 1)).
* ``gemm``    -- the backward and update GEMMs of Eqs. backward / update,
                 computed exactly on decoded integer codes in float64 and
                 scaled by the per-tensor scales once (Appendix A.1).
* ``im2col``  -- the 3x3 convolution lowering used by the ResNet-style
                 workload, on packed codes.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP library
and never imports it.  Where the paper is ambiguous the readings adopted are
listed in each module's header.
"""

from . import philox, luq, int4, gemm, im2col  # noqa: F401
