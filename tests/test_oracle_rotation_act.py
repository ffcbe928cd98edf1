"""Pins of the oracle's Hadamard rotation and per-token INT4 activation quantizer."""
import numpy as np
import pytest

from oracle import hadamard, quant


def _sylvester(b):
    H = np.array([[1]], dtype=np.int64)
    while H.shape[0] < b:
        H = np.block([[H, H], [H, -H]])
    return H


@pytest.mark.parametrize("b", [2, 4, 8, 64, 256, 1024])
def test_formula_matches_sylvester_recursion(b):
    assert np.array_equal(hadamard.hadamard(b), _sylvester(b))


def test_h2_literal_and_orthogonality():
    assert hadamard.hadamard(2).tolist() == [[1, 1], [1, -1]]
    for b in (16, 512, 4096):
        H = hadamard.hadamard(b)
        assert np.array_equal(H, H.T)
        Hf = H.astype(np.float64)          # entries +-1, sums <= 4096: exact in fp64
        assert np.array_equal(Hf @ Hf.T, b * np.eye(b))


def _fwht_int(v):
    """In-place iterative butterflies with Python integers (independent of the oracle's matrix)."""
    v = [int(a) for a in v]
    h = 1
    while h < len(v):
        for i in range(0, len(v), 2 * h):
            for j in range(i, i + h):
                a, b = v[j], v[j + h]
                v[j], v[j + h] = a + b, a - b
        h *= 2
    return v


def test_exact_rotation_adversarial_fp16():
    # extremes of fp16: max normal, smallest subnormal, mixed magnitudes
    b = 4096
    rng = np.random.default_rng(3)
    mags = 10.0 ** rng.uniform(-6, 3, size=b)
    x = (mags * rng.choice([-1, 1], size=b)).astype(np.float16)
    x[0] = np.float16(65504.0)
    x[1] = np.float16(-65504.0)
    x[2] = np.float16(2.0 ** -24)
    x[3] = np.float16(-(2.0 ** -24))
    X = hadamard.rotate_act_units(x[None, :], b)[0]
    units = [int(v) for v in (x.astype(np.float64) * 2.0 ** 24)]
    assert X.tolist() == _fwht_int(units)


def test_block_diagonal_rotation():
    b, nblk = 64, 5
    rng = np.random.default_rng(4)
    x = rng.standard_normal((3, b * nblk)).astype(np.float16)
    X = hadamard.rotate_act_units(x, b)
    for m in range(3):
        for j in range(nblk):
            seg = (x[m, j * b:(j + 1) * b].astype(np.float64) * 2.0 ** 24).astype(np.int64)
            assert X[m, j * b:(j + 1) * b].tolist() == _fwht_int(seg)


@pytest.mark.parametrize("b,nblk", [(64, 4), (256, 2), (16, 7)])
def test_rotation_semantics_weights_and_activations_agree(b, nblk):
    # W x == W_rot (H x / sqrt(b)): weight and activation rotations agree in orientation,
    # block order and normalisation (QuaRot-style invariance, Sec. 3.1)
    K = b * nblk
    rng = np.random.default_rng(5)
    W = rng.standard_normal((9, K))
    x = rng.standard_normal((4, K)).astype(np.float16)
    Wr = hadamard.rotate_weights(W, b)
    Xn = hadamard.rotate_act_units(x, b).astype(np.float64) * 2.0 ** -24 / np.sqrt(b)
    lhs = x.astype(np.float64) @ W.T
    rhs = Xn @ Wr.T
    assert np.max(np.abs(lhs - rhs)) <= 1e-12 * np.max(np.abs(lhs))
    assert np.allclose(hadamard.rotate_act_float(x, b), Xn, rtol=0, atol=1e-12)


def test_rotation_rejects_bad_blocks():
    x = np.zeros((1, 96), dtype=np.float16)
    with pytest.raises(ValueError):
        hadamard.rotate_act_units(x, 48)      # not a power of two
    with pytest.raises(ValueError):
        hadamard.rotate_act_units(x, 64)      # does not divide K


# --------------------------------------------------------------------------- activations


def test_act_quant_invariants():
    rng = np.random.default_rng(6)
    K, b = 1024, 256
    x = (rng.standard_normal((8, K)) * np.where(rng.random(K) < 0.01, 30, 1)).astype(np.float16)
    q, s_x, sq, X = quant.act_quant(x, b)
    assert q.dtype == np.int8 and s_x.dtype == np.float32 and sq.dtype == np.int32
    A = np.abs(X).max(axis=1)
    v = 7.0 * X.astype(np.float64) / A[:, None].astype(np.float64)
    assert np.all(np.abs(v - q) <= 0.5 + 1e-12)               # nearest integer
    assert np.all(np.abs(q) <= 7)
    for m in range(8):
        assert abs(q[m, np.argmax(np.abs(X[m]))]) == 7
    # away from exact halves the rounding equals fp64 rint of 7X/A
    far = np.abs(np.abs(v - np.floor(v)) - 0.5) > 1e-9
    assert np.array_equal(q[far], np.rint(v[far]).astype(np.int8))
    assert np.array_equal(sq, q.astype(np.int64).sum(axis=1))
    # per-token scale is max|H x / sqrt(b)| / 7 of the normalised rotation
    Xn = hadamard.rotate_act_float(x, b)
    want = np.abs(Xn).max(axis=1) / 7.0
    assert np.allclose(s_x, want, rtol=2 ** -23, atol=0)
    # dequantized activations are within half a step of the rotated token
    assert np.all(np.abs(Xn - s_x[:, None].astype(np.float64) * q) <= 0.5 * s_x[:, None] * (1 + 1e-6))


def test_act_quant_exact_ties_round_to_even():
    u = 2.0 ** -10
    # b=2: X = (x0 + x1, x0 - x1); A = 14u makes 7|X|/A = |X| / (2u)
    cases = [((9.5, 4.5), (7, 2)),     # X = (14u, 5u): 2.5 -> 2
             ((10.5, 3.5), (7, 4)),    # X = (14u, 7u): 3.5 -> 4
             ((7.5, 6.5), (7, 0)),     # X = (14u, 1u): 0.5 -> 0
             ((8.5, 5.5), (7, 2)),     # X = (14u, 3u): 1.5 -> 2
             ((4.5, 9.5), (7, -2))]    # X = (14u, -5u): -2.5 -> -2
    for (a, bb), want in cases:
        x = np.array([[a * u, bb * u]], dtype=np.float16)
        q, _, _, _ = quant.act_quant(x, 2)
        assert q[0].tolist() == list(want)


def test_act_quant_clip_ratio_nine_tenths():
    rng = np.random.default_rng(11)
    x = rng.standard_normal((4, 256)).astype(np.float16)
    q, s_x, _, X = quant.act_quant(x, 256, clip=(9, 10))
    A = np.abs(X).max(axis=1).astype(np.float64)
    v = 70.0 * np.abs(X) / (9.0 * A[:, None])
    far = np.abs(np.abs(v - np.floor(v)) - 0.5) > 1e-9
    want = np.minimum(np.rint(v), 7) * np.sign(X)
    assert np.array_equal(q[far], want[far].astype(np.int8))
    assert np.all(np.abs(q) <= 7)
    assert np.allclose(s_x, 0.9 * np.abs(hadamard.rotate_act_float(x, 256)).max(axis=1) / 7, rtol=2 ** -22)


def test_act_quant_zero_token():
    x = np.zeros((2, 128), dtype=np.float16)
    x[1, 5] = np.float16(1.0)
    q, s_x, sq, _ = quant.act_quant(x, 64)
    assert not q[0].any() and s_x[0] == 0 and sq[0] == 0
    # a single spike spreads to +-1 * 1 over its block: every entry hits |q| = 7
    assert np.all(np.abs(q[1, :64]) == 7) and not q[1, 64:].any()


def _bf16(a):
    """Round float32 values to bf16 (nearest even on the upper 16 bits) and return them as float32."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16 << 16
    return u.astype(np.uint32).view(np.float32)


def test_act_quant_bf16_inputs_on_the_grid():
    """bf16 activations (a deployment variant; the paper's reference is fp16) on the 2^-24 grid rotate exactly: the
    results equal the fp16 path's on the same values (every such bf16 is also an fp16), and the
    rounding decisions stay exact integers; values off the grid are refused."""
    rng = np.random.default_rng(5)
    x = _bf16(rng.normal(0, 1, (6, 512)) * rng.uniform(1e-3, 300, (6, 1)))
    x[np.abs(x) < 2.0 ** -17] = 0.0                       # keep every value on the grid
    x[0, :4] = [2.0 ** -17, -(2.0 ** -17), 65280.0, -3.0]   # grid ends: bf16 min on the grid, max below 2^16
    assert np.array_equal(x.astype(np.float16).astype(np.float32), x)   # exact in fp16 as well
    for clip in ((1, 1), (9, 10)):
        a = quant.act_quant(x, 128, clip)
        c = quant.act_quant(x.astype(np.float16), 128, clip)
        for u, v in zip(a, c):
            assert np.array_equal(u, v)
    with pytest.raises(ValueError):
        quant.act_quant(np.full((1, 128), 2.0 ** -25, dtype=np.float32), 128)   # half a grid step
    with pytest.raises(ValueError):
        quant.act_quant(np.full((1, 128), 65536.0, dtype=np.float32), 128)      # 2^16
