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
* :mod:`oracle.quant`    - per-token INT4 activation quantizer (fp16 exact, and the
                           staged fp64 reading for bf16); per-output-channel weight
                           quantizers for MNZ, PoT-MNZ, W4 and the mirror family
                           G(r); the ratio scan (Eq. (1), Sec. 3.3, Sec. 3.4 Eq. (18),
                           Sec. 3.5, Sec. 4.5.1, Sec. 4.5.3)
* :mod:`oracle.pack`     - the canonical 2-bit (QW2v1) and 4-bit (QW4v1) word
                           layouts, with their decoders
* :mod:`oracle.linear`   - exact int32 accumulator and the fp16 epilogue with the
                           per-channel and per-token scales (Sec. 1, Sec. 3.6)
* :mod:`oracle.lut`      - the linear over a four-level fp16 table (the reference
                           grids of Sec. 3.3)
* :mod:`oracle.kv4`      - asymmetric 4-bit KV cache and decode attention over it
                           (Sec. 4.1)

Pinned by the ``-m "not gpu"`` tests against the paper's printed constants and
tables, closed forms, invariants and brute force.  Readings of points where the
paper is silent are listed in each function's docstring.
"""
from . import levels, hadamard, quant, pack, linear  # noqa: F401
