"""Integer dot product and fp16 epilogue of the quantized linear.

``y[m, n] = s_w[n] * s_x[m] * sum_k level[n, k] * q[m, k]``: decoded small signed
integer weight levels times INT4 activations, accumulated exactly, with the
per-output-channel scale and the per-token scale applied afterwards in the
epilogue (Sec. 1 last paragraph before the contributions; Sec. 3.6).

Reading of the epilogue's precision: the reference value is the fp64 product
rounded once to fp16; the GPU's fp32 expression ``fp16(fp32(fp32(acc) * s_x) *
fp32(s_w))`` is also given here (``epilogue_fp32``) because the tests expect
it bit for bit.  Pass criterion on y: max over elements of
``|y - y_ref| / max(|y_ref|, 2^-14) <= 1e-3``.
"""
from __future__ import annotations

import numpy as np

from . import pack

TOL_REL = 1e-3
TOL_FLOOR = 2.0 ** -14


def int_dot_loops(L, Q):
    """acc[m][n] = sum_k L[n][k] * Q[m][k] with Python integers (tiny shapes only)."""
    L = [[int(v) for v in row] for row in np.asarray(L)]
    Q = [[int(v) for v in row] for row in np.asarray(Q)]
    return [[sum(a * b for a, b in zip(Lrow, Qrow)) for Lrow in L] for Qrow in Q]


def int_dot(L: np.ndarray, Q: np.ndarray) -> np.ndarray:
    """acc = Q @ L^T as int64 via an fp64 matmul of the integer-valued operands.

    Every product and partial sum is an integer of magnitude below 2^53, so the
    fp64 result is exact whatever the summation order; integrality is asserted.
    """
    L = np.asarray(L)
    Q = np.asarray(Q)
    K = L.shape[1]
    bound = int(np.abs(L).max(initial=0)) * int(np.abs(Q).max(initial=0)) * K
    assert bound < 2 ** 53
    acc = Q.astype(np.float64) @ L.astype(np.float64).T
    out = acc.astype(np.int64)
    assert np.array_equal(out.astype(np.float64), acc)
    assert np.all(np.abs(out) < 2 ** 31)
    return out


def epilogue_ref(acc: np.ndarray, s_x: np.ndarray, s_w: np.ndarray) -> np.ndarray:
    """fp16 of the fp64 product ``acc * s_x[m] * s_w[n]`` (IEEE rounding, overflow to inf)."""
    v = np.asarray(acc, np.float64) * np.asarray(s_x, np.float64)[:, None] * \
        np.asarray(s_w, np.float64)[None, :]
    with np.errstate(over="ignore"):
        return v.astype(np.float16)


def epilogue_fp32(acc: np.ndarray, s_x: np.ndarray, s_w: np.ndarray) -> np.ndarray:
    """``fp16(fp32(fp32(acc) * s_x) * fp32(s_w))`` with each fp32 product rounded."""
    a = np.asarray(acc).astype(np.float32)
    t = a * np.asarray(s_x, np.float32)[:, None]
    v = t * np.asarray(s_w, np.float16).astype(np.float32)[None, :]
    with np.errstate(over="ignore"):
        return v.astype(np.float16)


def max_abs_rel(y: np.ndarray, y_ref: np.ndarray) -> float:
    """Max of ``|y - y_ref| / max(|y_ref|, 2^-14)``; matching infinities count as equal."""
    y = np.asarray(y, np.float64)
    r = np.asarray(y_ref, np.float64)
    same = (y == r)
    with np.errstate(invalid="ignore"):
        err = np.abs(y - r) / np.maximum(np.abs(r), TOL_FLOOR)
    err = np.where(same, 0.0, err)
    if np.any(np.isnan(err)):
        return float("inf")
    return float(err.max(initial=0.0))


def linear(P: np.ndarray, s_w: np.ndarray, fmt: int, K: int, q: np.ndarray, s_x: np.ndarray):
    """The whole quantized linear from packed words: returns (y_ref fp16 [M,N], acc int64 [M,N])."""
    L = pack.unpack(P, fmt, K)
    acc = int_dot(L, q)
    return epilogue_ref(acc, s_x, s_w), acc
