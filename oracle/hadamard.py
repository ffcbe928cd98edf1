"""Hadamard rotation (Sec. 3.1; Sec. 4.1 "Quantization configuration").

The paper rotates with the default (deterministic) Hadamard matrix of a
QuaRot-style pipeline and samples no random rotation.  Readings used here:

* ``H_b[i, j] = (-1)^popcount(i & j)``: the Sylvester matrix in natural order,
  built entry by entry from that formula (symmetric, ``H_b H_b^T = b I``).
* For an input width K that is not a power of two the rotation is
  block-diagonal, ``I_{K/b} (x) H_b``, with a power-of-two block ``b | K``.
* The orthonormal rotation is ``H_b / sqrt(b)``.  Weights are rotated with it
  offline; activations are rotated online *unnormalised* (an exact integer
  combination of the fp16 inputs) and the ``1/sqrt(b)`` goes into the
  per-token scale, so that ``W x = W_rot (H x / sqrt(b))``.
"""
from __future__ import annotations

import functools

import numpy as np

FP16_UNIT = 2.0 ** -24   # every finite fp16 value is an integer multiple of this


def check_block(K: int, b: int) -> None:
    if b < 2 or b & (b - 1):
        raise ValueError(f"Hadamard block {b} is not a power of two >= 2")
    if K % b:
        raise ValueError(f"K={K} is not a multiple of the block {b}")


@functools.lru_cache(maxsize=8)
def hadamard(b: int) -> np.ndarray:
    """Sylvester Hadamard matrix of order ``b`` from the entry formula (int64)."""
    check_block(b, b)
    i = np.arange(b, dtype=np.int64)
    parity = np.bitwise_count(i[:, None] & i[None, :]) & 1
    H = 1 - 2 * parity.astype(np.int64)
    H.setflags(write=False)
    return H


def rotate_act_units(x: np.ndarray, b: int) -> np.ndarray:
    """Exact ``X = (I (x) H_b) x`` per token, in integer units of 2^-24.

    ``x`` is fp16 [M, K], or any float array whose values lie on the same grid
    (multiples of 2^-24 of magnitude below 2^16: every fp16, and every bf16 of
    magnitude in [2^-17, 2^16) or zero, bf16 having 8 significant bits).  Each
    value times 2^24 is then an integer of magnitude below 2^40, so every
    partial sum of at most 2^13 of them stays below 2^53 and the fp64 product
    below is exact in any summation order.  Returns int64 [M, K].
    """
    x = np.asarray(x)
    if x.dtype.kind != "f":
        raise TypeError("activations must be floating point")
    M, K = x.shape
    check_block(K, b)
    if b > 8192:
        raise ValueError("block above 8192 would break fp64 exactness")
    xu = x.astype(np.float64) * 2.0 ** 24
    if not np.all(np.isfinite(xu)):
        raise ValueError("non-finite activation")
    if x.dtype != np.float16 and not (np.all(xu == np.round(xu)) and np.all(np.abs(xu) < 2.0 ** 40)):
        raise ValueError("activation off the 2^-24 grid or not below 2^16 in magnitude")
    H = hadamard(b).astype(np.float64)
    X = (xu.reshape(M, K // b, b) @ H).reshape(M, K)   # H symmetric: x_blk @ H == H @ x_blk
    Xi = X.astype(np.int64)
    assert np.array_equal(Xi.astype(np.float64), X), "rotation left the exact integer grid"
    return Xi


def rotate_act_staged(x: np.ndarray, b: int) -> np.ndarray:
    """``X = (I (x) H_b) x`` per token in fp64, one butterfly stage per index bit, bits in ascending order.

    Stage j pairs the elements whose block index differs only in bit j and replaces (a, c) by
    (a + c, a - c), each rounded to fp64 (round to nearest, ties to even).  After the L = log2(b)
    stages every element holds its +-1 combination of the block (Sylvester ordering).  Inputs are any
    finite floats (fp16 or bf16 values, converted to fp64 exactly); on the 2^-24 grid of
    :func:`rotate_act_units` every partial sum is exact and this equals that transform times 2^-24.
    Returns fp64 [M, K].
    """
    x = np.asarray(x)
    if x.dtype.kind != "f":
        raise TypeError("activations must be floating point")
    M, K = x.shape
    check_block(K, b)
    X = x.astype(np.float64).reshape(M, K // b, b)
    if not np.all(np.isfinite(X)):
        raise ValueError("non-finite activation")
    h = 1
    while h < b:
        Y = X.reshape(M, K // b, b // (2 * h), 2, h)
        lo, hi = Y[:, :, :, 0, :], Y[:, :, :, 1, :]
        X = np.stack([lo + hi, lo - hi], axis=3).reshape(M, K // b, b)
        h *= 2
    return X.reshape(M, K)


def rotate_weights(W: np.ndarray, b: int) -> np.ndarray:
    """Offline rotation of weight rows: ``W_rot[n, :] = (I (x) H_b) W[n, :] / sqrt(b)`` (fp64)."""
    W = np.asarray(W, dtype=np.float64)
    N, K = W.shape
    check_block(K, b)
    H = hadamard(b).astype(np.float64)
    return (W.reshape(N, K // b, b) @ H).reshape(N, K) / np.sqrt(float(b))


def rotate_act_float(x: np.ndarray, b: int) -> np.ndarray:
    """Normalised rotation ``(I (x) H_b) x / sqrt(b)`` of any float array [M, K] in fp64."""
    x = np.asarray(x, dtype=np.float64)
    M, K = x.shape
    check_block(K, b)
    H = hadamard(b).astype(np.float64)
    return (x.reshape(M, K // b, b) @ H).reshape(M, K) / np.sqrt(float(b))
