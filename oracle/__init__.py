"""Reference oracle for VBQ packed weights and the fused dequantize-and-multiply.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check in
``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` may import this
package.  The product path (``paper_2607_02893_amd``) never imports it and
shares no code with it: this is a plain, slow, double-precision CPU
restatement of what the method computes, written from the paper
(arxiv 2607.02893, "Variable Bit-width Quantization"), used to check the HIP
kernels element by element.

Modules
  quant    -- the per-group quantizer: paper section 3.1, Eq. (1) for
              b in {2,4,8} and the sign/absmean rule for b = 1.
  layout   -- the packed byte format (version 1) written out independently of
              the C++ packer: pack / unpack / byte sizes.
  matmul   -- dequantization w_hat = s*q and the fp64 GEMV / small GEMM that the
              fused kernels must reproduce (paper section 6).
  storage  -- packed-storage accounting, params * mean_bits / 8 (paper
              section 4, "Training", and Table 1).
  qat      -- differentiable bit selection: the Gumbel-Softmax mix of the four
              candidate reconstructions, the expected bit cost, the hardened
              widths and the logit-step gradient (paper sections 3.2-3.3 and
              Algorithm 1).

Readings of the paper that the oracle fixes (every one is listed, with its
justification, in the design notes of the repository):
  * round() is round-half-to-even.
  * The codes are computed against the scale after it is rounded to fp16.
  * Scales are IEEE fp16, computed in double and rounded once.
  * sign(0) = +1 for the 1-bit rule.
  * The 1-bit absmean is the sequential double sum over the group / 64.
  * An all-zero group has s = 0 and q = 0 for b >= 2.
  * K % 64 == 0 is required.

Parity status: every function here is pinned by CPU tests against values the
method fixes (hand-computed groups from Eq. (1), closed forms, invariants,
brute force on tiny inputs); none is "parity unpinned".
"""

from . import quant, layout, matmul, storage, qat  # noqa: F401

__all__ = ["quant", "layout", "matmul", "storage", "qat"]
