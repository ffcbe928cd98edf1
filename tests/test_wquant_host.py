"""Host checks of the GPU weight quantizer's fixed constants (no GPU).

The kernel generates the 64 PoT candidate scale factors as j * ((1 - 0.2) / 63) + 0.2 for j < 63
and exactly 1 for the last (the evaluation order of linspace(0.2, 1, 64)); the oracle takes them
from numpy's linspace.  Both must be the same doubles, or the scale search would compare different
candidates.
"""
import numpy as np

from oracle import quant


def test_pot_candidates_are_linspace_bit_for_bit():
    step = (1.0 - 0.2) / 63.0
    kernel = np.array([j * step + 0.2 for j in range(63)] + [1.0])
    assert np.array_equal(kernel.view(np.uint64), quant.POT_CANDIDATES.view(np.uint64))
    assert kernel[0] == 0.2 and kernel[-1] == 1.0
