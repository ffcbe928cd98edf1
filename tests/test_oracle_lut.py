"""Pins of the level-table linear (the reference grids of Sec. 3.3 read through an fp16 table)."""
import numpy as np
import pytest

from oracle import levels, linear, lut, pack


def test_integer_tables_reduce_to_the_integer_linear():
    """With the MNZ (half scale) or PoT levels as the table, t is the pinned integer accumulator."""
    rng = np.random.default_rng(1)
    N, K, M = 7, 192, 3
    codes = rng.integers(0, 4, (N, K))
    q = rng.integers(-7, 8, (M, K))
    for grid in (levels.MNZ_HALF, levels.POT):
        L = np.asarray(grid)[codes]
        assert np.array_equal(lut.lut_dot(codes, grid, q), linear.int_dot(L, q).astype(np.float64))


@pytest.mark.parametrize("grid", [levels.LLOYD, levels.NF2, (-256.0, -(2.0 ** -24), 2.0 ** -14, 255.9),
                                  (0.1, 0.1, -0.3, 7.0)])
def test_exact_against_fractions(grid):
    rng = np.random.default_rng(2)
    codes = rng.integers(0, 4, (5, 64))
    q = rng.integers(-7, 8, (4, 64))
    q[0] = 7                                       # extreme accumulations
    codes[0] = 3
    t = lut.lut_dot(codes, grid, q)
    ref = lut.lut_dot_loops(codes, grid, q)
    assert all(t[m, n] == float(ref[m][n]) for m in range(4) for n in range(5))
    assert all(float(ref[m][n]) == ref[m][n] for m in range(4) for n in range(5))   # fits fp64


def test_bit_plane_decomposition():
    """t = L0 S + (L1 - L0) P0 + (L2 - L0) P1 + (L3 - L2 - L1 + L0) P01 with the integer sums
    S = sum q, P0 = sum b0 q, P1 = sum b1 q, P01 = sum b0 b1 q of the code bits c = b0 + 2 b1."""
    rng = np.random.default_rng(3)
    codes = rng.integers(0, 4, (9, 256))
    q = rng.integers(-7, 8, (6, 256))
    L = lut.table(levels.LLOYD).astype(np.float64)
    b0, b1 = codes & 1, codes >> 1
    S = q.sum(axis=1)[:, None]
    P0, P1, P01 = q @ b0.T, q @ b1.T, q @ (b0 & b1).T
    t = L[0] * S + (L[1] - L[0]) * P0 + (L[2] - L[0]) * P1 + (L[3] - L[2] - L[1] + L[0]) * P01
    assert np.array_equal(t, lut.lut_dot(codes, L, q))


def test_packed_codes_round_trip_and_linear():
    rng = np.random.default_rng(4)
    N, K, M = 6, 128, 2
    codes = rng.integers(0, 4, (N, K)).astype(np.int8)
    P = pack.pack_qw2(codes, levels.FMT_W2_LUT)
    assert np.array_equal(pack.unpack_qw2(P, levels.FMT_W2_LUT, K), codes)
    q = rng.integers(-7, 8, (M, K))
    s_x = rng.uniform(0.01, 0.1, M).astype(np.float32)
    s_w = rng.uniform(0.01, 0.1, N).astype(np.float16)
    y, y_ref, t = lut.lut_linear(P, levels.NF2, s_w, K, q, s_x)
    assert np.array_equal(t, lut.lut_dot(codes, levels.NF2, q))
    assert linear.max_abs_rel(y, y_ref) <= linear.TOL_REL


def test_table_bounds():
    with pytest.raises(ValueError):
        lut.table((0.0, 1.0, 2.0, 257.0))
    with pytest.raises(ValueError):
        lut.table((0.0, 1.0, 2.0, np.inf))
    with pytest.raises(ValueError):
        lut.table((0.0, 1.0, 2.0))
    assert lut.table(levels.LLOYD).dtype == np.float16
