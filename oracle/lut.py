"""Quantized linear over a four-level grid read through a level table.

Test infrastructure: a plain CPU statement of what the GPU path computes (only tests and the
benchmark's CPU leg use it).

The reference grids of Sec. 3.3 -- Lloyd-Max (Eq. (9)) and NF2 (Eq. (10)) -- have non-integer
levels, so the integer accumulation of the W2 formats does not carry over.  With the four levels
held as fp16 values in a table indexed by the 2-bit code (code c = the c-th entry; the paper
leaves the code assignment free, Sec. 3.3):

    t[m, n] = sum_k lut[c[n, k]] * q[m, k]            (exact)
    y[m, n] = fp16(fp32(fp32(t) * s_x[m]) * fp32(s_w[n]))

i.e. the epilogue of the integer formats (Sec. 3.6) with t in place of the accumulator.  t is
exact: every fp16 table entry of magnitude at most 256 is an integer multiple of 2^-24 below
2^32 units, so with |q| <= 7 and K <= 2^14 every term and partial sum is an integer number of
units below 2^53.  Readings: the table is fp16 (the levels as the caller rounds them), t is
rounded once to fp32 before the scales.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

from . import levels, linear, pack

UNIT = 2.0 ** -24
LUT_MAX = 256.0


def table(grid) -> np.ndarray:
    """The fp16 level table of a four-level grid (each level rounded once to fp16)."""
    t = np.asarray(grid, dtype=np.float64).astype(np.float16)
    if t.shape != (4,) or not np.all(np.isfinite(t)) or np.any(np.abs(t.astype(np.float64)) > LUT_MAX):
        raise ValueError("a level table is four finite fp16 values of magnitude <= 256")
    return t


def lut_dot(codes: np.ndarray, lut: np.ndarray, q: np.ndarray) -> np.ndarray:
    """t[m, n] = sum_k lut[codes[n, k]] q[m, k], exact, as fp64 [M, N] (integer units of 2^-24)."""
    lut = table(lut)
    units = (lut.astype(np.float64) / UNIT).astype(np.int64)
    assert np.array_equal(units.astype(np.float64) * UNIT, lut.astype(np.float64))
    W = units[np.asarray(codes, dtype=np.int64)]                     # [N, K] integer units
    Q = np.asarray(q, dtype=np.int64)
    K = W.shape[1]
    assert int(np.abs(W).max(initial=0)) * int(np.abs(Q).max(initial=0)) * K < 2 ** 53
    acc = Q.astype(np.float64) @ W.astype(np.float64).T              # exact: integers below 2^53
    assert np.array_equal(acc, np.round(acc))
    return acc * UNIT


def lut_dot_loops(codes, lut, q):
    """The same with Fractions and Python loops (tiny shapes only)."""
    vals = [Fraction(float(v)) for v in table(lut)]
    C = [[int(c) for c in row] for row in np.asarray(codes)]
    Q = [[int(v) for v in row] for row in np.asarray(q)]
    return [[sum(vals[c] * v for c, v in zip(crow, qrow)) for crow in C] for qrow in Q]


def lut_linear(P: np.ndarray, lut: np.ndarray, s_w: np.ndarray, K: int, q: np.ndarray, s_x: np.ndarray):
    """From packed QW2v1 code words: returns (y fp16 [M, N] by the fp32 epilogue, y_ref fp16 of the
    fp64 product, t fp64 [M, N])."""
    codes = pack.unpack_qw2(P, levels.FMT_W2_LUT, K)
    t = lut_dot(codes, lut, q)
    return linear.epilogue_fp32(t, s_x, s_w), linear.epilogue_ref(t, s_x, s_w), t
