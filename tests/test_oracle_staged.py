"""Pins of the oracle's staged fp64 reading of the rotation for activations off the 2^-24 grid
(oracle.hadamard.rotate_act_staged, oracle.quant.act_quant_staged), checked against values worked out
by hand and against the exact transform where every partial sum is exact."""
import numpy as np
import pytest

from oracle import hadamard, quant
from paper_2606_02823_amd import synth


def test_stage_order_by_hand():
    # b = 4, x = [1, 2^-53, 2^-53, 0].  Bit 0: (1 + 2^-53 -> 1 (a tie, to even), 1 - 2^-53, 2^-53, 2^-53);
    # bit 1: (1 + 2^-53 -> 1, (1 - 2^-53) + 2^-53 = 1, 1 - 2^-53, 1 - 2^-52).  The exact transform is
    # [1 + 2^-52, 1, 1, 1 - 2^-52]; taking bit 1 first would give [1, 1 - 2^-53, 1, 1 - 2^-52].
    x = np.array([[1.0, 2.0 ** -53, 2.0 ** -53, 0.0]])
    X = hadamard.rotate_act_staged(x, 4)
    assert X.tolist() == [[1.0, 1.0, 1.0 - 2.0 ** -53, 1.0 - 2.0 ** -52]]


@pytest.mark.parametrize("K,b", [(256, 2), (512, 256), (4096, 4096), (8192, 8192), (11008, 64)])
def test_equals_the_exact_rotation_on_the_fp16_grid(K, b):
    c = synth.CONFIGS[1]
    x = synth.config_activations(c, 3, 0, 3, K)
    q0, s0, m0, X0 = quant.act_quant(x, b)
    q1, s1, m1, X1 = quant.act_quant_staged(x, b)
    assert np.array_equal(X1, X0.astype(np.float64) * 2.0 ** -24)
    assert np.array_equal(q1, q0) and np.array_equal(s1.view(np.uint32), s0.view(np.uint32))
    assert np.array_equal(m1, m0)


def test_off_grid_ties_by_hand():
    # b = 2 blocks [a, c] -> [a + c, a - c], exact here.  Block 0: [4.75, 2.25] 2^-100 -> [7, 2.5] 2^-100,
    # block 1: [0.25, -3.25] 2^-100 -> [-3, 3.5] 2^-100; A = 7 2^-100, v = 7 |X| / A = |X| / 2^-100:
    # 7 -> 7, 2.5 -> 2 (tie, even), -3 -> -3, 3.5 -> 4 (tie, even).  With clip 9/10, v = 70 |X| / 63 2^-100:
    # 7 -> 7 (clamped), 2.5 -> 25/9 = 2.78 -> 3, 3 -> 10/3 -> 3, 3.5 -> 35/9 = 3.89 -> 4.
    u = 2.0 ** -100
    x = np.array([[4.75 * u, 2.25 * u, 0.25 * u, -3.25 * u]])
    q, s, m, X = quant.act_quant_staged(x, 2)
    assert X.tolist() == [[7 * u, 2.5 * u, -3 * u, 3.5 * u]]
    assert q.tolist() == [[7, 2, -3, 4]] and m.tolist() == [10]
    q, _, _, _ = quant.act_quant_staged(x, 2, clip=(9, 10))
    assert q.tolist() == [[7, 3, -3, 4]]


def test_tiny_and_huge_tokens():
    # a single nonzero bf16 value spreads to +-x at every position of its block: all codes +-7, and
    # s_x = x / (7 sqrt(b)) for the smallest bf16 subnormal and for a large bf16 value
    for v in (2.0 ** -133, -(2.0 ** 100)):
        x = np.zeros((1, 64))
        x[0, 5] = v
        q, s, m, X = quant.act_quant_staged(x, 64)
        H = hadamard.hadamard(64)[:, 5]
        assert np.array_equal(q[0], (7 * np.sign(v) * H).astype(np.int8))
        assert s[0] == np.float32((abs(v) * 1.0) / (7.0 * 8.0))
        assert m[0] == int(7 * np.sign(v) * H.sum())
