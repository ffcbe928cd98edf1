"""Pins of the oracle's integer dot product, epilogue and end-to-end linear."""
import numpy as np
import pytest

from oracle import hadamard, levels, linear, pack, quant
from paper_2606_02823_amd import synth


def test_int_dot_equals_python_loops():
    rng = np.random.default_rng(21)
    L = np.array(levels.MNZ_HALF, dtype=np.int8)[rng.integers(0, 4, size=(5, 64))]
    Q = rng.integers(-7, 8, size=(3, 64)).astype(np.int8)
    assert linear.int_dot(L, Q).tolist() == linear.int_dot_loops(L, Q)


def test_int_dot_extreme_magnitudes():
    # |acc| reaches 4*7*K for PoT and 7*7*K for W4 at the largest K of the workloads
    K = 14336
    L = np.full((2, K), 4, dtype=np.int8)
    L[1] = -4
    Q = np.full((1, K), -7, dtype=np.int8)
    assert linear.int_dot(L, Q).tolist() == [[-4 * 7 * K, 4 * 7 * K]]
    W4 = np.full((1, K), 7, dtype=np.int8)
    assert linear.int_dot(W4, -Q).tolist() == [[7 * 7 * K]]


def test_dequantized_dense_product():
    rng = np.random.default_rng(22)
    L = np.array(levels.POT, dtype=np.int8)[rng.integers(0, 4, size=(7, 128))]
    Q = rng.integers(-7, 8, size=(4, 128)).astype(np.int8)
    s_w = rng.uniform(0.001, 0.02, 7).astype(np.float16)
    s_x = rng.uniform(0.01, 1.0, 4).astype(np.float32)
    dense = (s_x.astype(np.float64)[:, None] * Q) @ (s_w.astype(np.float64)[:, None] * L).T
    acc = linear.int_dot(L, Q)
    got = acc * s_x.astype(np.float64)[:, None] * s_w.astype(np.float64)[None, :]
    assert np.max(np.abs(dense - got)) <= 1e-12 * np.max(np.abs(dense))


def test_epilogue_fp32_within_tolerance_of_fp64():
    rng = np.random.default_rng(23)
    acc = rng.integers(-400_000, 400_000, size=(16, 300))
    acc[0, :5] = [0, 1, -1, 2 ** 24 - 1, -(2 ** 24 - 1)]
    s_x = (10.0 ** rng.uniform(-3, 1, 16)).astype(np.float32)
    s_w = (10.0 ** rng.uniform(-4, -1, 300)).astype(np.float16)
    y32 = linear.epilogue_fp32(acc, s_x, s_w)
    y64 = linear.epilogue_ref(acc, s_x, s_w)
    assert linear.max_abs_rel(y32, y64) <= linear.TOL_REL
    assert np.mean(y32 == y64) > 0.95
    # overflow goes to inf on both sides
    big = linear.epilogue_ref(np.array([[400_000]]), np.array([1.0], np.float32), np.array([1.0], np.float16))
    assert np.isinf(big[0, 0])
    assert linear.max_abs_rel(big, big) == 0.0


def test_max_abs_rel_criterion():
    r = np.array([1.0, 2.0 ** -20, 0.0], dtype=np.float16)
    assert linear.max_abs_rel(r, r) == 0.0
    y = r.copy()
    y[0] = np.nextafter(np.float16(1.0), np.float16(2.0))
    assert linear.max_abs_rel(y, r) == pytest.approx(2.0 ** -10)
    y = r.copy()
    y[2] = np.float16(2.0 ** -10)
    assert linear.max_abs_rel(y, r) > linear.TOL_REL


@pytest.mark.parametrize("fmt", [levels.FMT_W2_MNZ, levels.FMT_W2_POT, levels.FMT_W4_SYM])
def test_end_to_end_reconstructs_float_linear(fmt):
    # the quantized linear approximates the float W x of the unrotated layer: a dropped 1/sqrt(b),
    # a transposed operand or a sign slip anywhere in the chain breaks this by a wide margin
    c = synth.CONFIGS[0]
    shp = c.linears[0]
    W = synth.weights_fp32(0, 0, "lin", shp.N, shp.K)
    x = synth.config_activations(c, 0, 0, 4, shp.K)
    Wr = hadamard.rotate_weights(W, shp.block)
    L, s_w = quant.quantize_weights(Wr, fmt)
    P = pack.pack(L, fmt)
    q, s_x, _, _ = quant.act_quant(x, shp.block)
    y, acc = linear.linear(P, s_w, fmt, shp.K, q, s_x)
    ref = x.astype(np.float64) @ W.astype(np.float64).T
    rel = np.linalg.norm(y.astype(np.float64) - ref) / np.linalg.norm(ref)
    bound = {levels.FMT_W2_MNZ: 0.5, levels.FMT_W2_POT: 0.5, levels.FMT_W4_SYM: 0.25}[fmt]
    assert 0.0 < rel < bound, rel
    assert np.array_equal(acc, linear.int_dot(L, q))
