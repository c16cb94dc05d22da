"""CPU oracle for the FP8 linear-layer path (test infrastructure only).

This package is a plain, slow, deliberately unoptimised CPU statement of what
the FP8 linear layer of the paper computes (Section 3.2, "FP8 Mixed-Precision
Training", and Appendix C, "FP8 implementation pipeline"):

* ``fp8``    -- the OCP E4M3 / E5M2 codecs (decode table, round-to-nearest-even
                encode with saturation);
* ``quant``  -- amax, per-tensor and power-of-two block scales, and the
                quantisers (per-tensor, 1x128 rows, 128x1 columns, 128x128);
* ``gemm``   -- the scaled FP8 GEMM as an FP64 triple loop (plain C, OpenMP
                over output rows), plus a pure-Python exact-rational version
                for tiny inputs;
* ``linear`` -- the linear layer's forward and backward composed from the
                above;
* ``bf16``   -- BF16 bit helpers used to state expected outputs;
* ``swiglu`` -- the MLP's SwiGLU, whose BF16 output the down projection
                quantises (the fused SwiGLU + quantise operation);
* ``rmsnorm`` -- the RMSNorm whose BF16 output the QKV and gate/up
                projections quantise (the fused RMSNorm + quantise
                operation);
* ``lm_head`` -- the language-model head with its cross-entropy loss,
                forward and backward;
* ``muonh``  -- the MuonH optimiser step of one matrix: momentum,
                Newton-Schulz orthogonalisation and the hyperball update.

It is test infrastructure: only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import it. It shares no code with
the HIP library and never imports it.
"""

from . import bf16, fp8, quant, gemm, linear, rmsnorm, swiglu, lm_head, muonh  # noqa: F401
