"""CPU oracle for the rotated W2A4 quantized linear (Qift, arXiv 2606.02823).

TEST INFRASTRUCTURE ONLY.  This package is the plain, slow, obviously correct
definition of what the GPU path computes, written from the paper in NumPy.
Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import it; the product path never does, and it shares no code with the HIP
library (its own Hadamard construction, quantizers, packer and integer dot).

Modules, each citing the passage it follows:

* :mod:`oracle.levels`   - the fixed four-level sets (Sec. 1, Sec. 3.3, Sec. 3.4)
* :mod:`oracle.hadamard` - Sylvester Hadamard matrix by formula, block-diagonal
                           rotation of activations (exact) and weights (Sec. 3.1,
                           Sec. 4.1 "Quantization configuration")
* :mod:`oracle.quant`    - per-token INT4 activation quantizer; per-output-channel
                           weight quantizers for MNZ, PoT-MNZ and W4 (Eq. (1),
                           Sec. 3.3, Sec. 3.5, Sec. 4.5.1)
* :mod:`oracle.pack`     - the canonical 2-bit (QW2v1) and 4-bit (QW4v1) word
                           layouts, with their decoders
* :mod:`oracle.linear`   - exact int32 accumulator and the fp16 epilogue with the
                           per-channel and per-token scales (Sec. 1, Sec. 3.6)

Pinned by the ``-m "not gpu"`` tests against the paper's printed constants and
tables, closed forms, invariants and brute force.  Readings of points where the
paper is silent are listed in each function's docstring.
"""
from . import levels, hadamard, quant, pack, linear  # noqa: F401
