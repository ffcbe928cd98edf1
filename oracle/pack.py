"""Canonical packed weight words (the bytes the GPU packer must reproduce).

The paper fixes the four levels and leaves the code assignment to the
implementation (Sec. 3.3); this project's layouts are:

QW2v1 (2-bit; MNZ and PoT-MNZ), ``uint32 P[N][K/16]``, little-endian, row-major:
    code ``c`` = index of the level in the ascending level list;
    weight ``k = 16 j + 4 t + beta`` (t, beta in 0..3) sits in bits
    ``[8 beta + 2 t, 8 beta + 2 t + 1]`` of word ``j``.

QW4v1 (4-bit; symmetric W4), ``uint32 P[N][K/8]``:
    stored nibble ``u = q + 8`` in 1..15;
    weight ``k = 8 j + 4 t + beta`` (t in 0..1, beta in 0..3) sits in bits
    ``[8 beta + 4 t, 8 beta + 4 t + 3]`` of word ``j``.

Both require ``K % 64 == 0``.
"""
from __future__ import annotations

import numpy as np

from . import levels


def codes_from_levels(L: np.ndarray, fmt: int) -> np.ndarray:
    """2-bit codes (uint32) of decoded levels; raises on a level outside the set."""
    table = levels.CODE_LEVELS[fmt]
    L = np.asarray(L)
    c = np.full(L.shape, -1, dtype=np.int64)
    for code, lev in enumerate(table):
        c[L == lev] = code
    if np.any(c < 0):
        raise ValueError("level outside the format's level set")
    return c.astype(np.uint32)


def pack_qw2(L: np.ndarray, fmt: int) -> np.ndarray:
    N, K = L.shape
    if K % 64:
        raise ValueError("K must be a multiple of 64")
    c = codes_from_levels(L, fmt).reshape(N, K // 16, 4, 4)   # [n, j, t, beta]
    P = np.zeros((N, K // 16), dtype=np.uint32)
    for t in range(4):
        for beta in range(4):
            P |= c[:, :, t, beta] << np.uint32(8 * beta + 2 * t)
    return P


def unpack_qw2(P: np.ndarray, fmt: int, K: int) -> np.ndarray:
    N = P.shape[0]
    table = np.asarray(levels.CODE_LEVELS[fmt], dtype=np.int8)
    c = np.empty((N, K // 16, 4, 4), dtype=np.uint32)
    for t in range(4):
        for beta in range(4):
            c[:, :, t, beta] = (P >> np.uint32(8 * beta + 2 * t)) & np.uint32(3)
    return table[c.reshape(N, K)]


def pack_qw4(q: np.ndarray) -> np.ndarray:
    N, K = q.shape
    if K % 64:
        raise ValueError("K must be a multiple of 64")
    q = np.asarray(q, dtype=np.int64)
    if np.any(q < -7) or np.any(q > 7):
        raise ValueError("W4 level outside -7..7")
    u = (q + 8).astype(np.uint32).reshape(N, K // 8, 2, 4)    # [n, j, t, beta]
    P = np.zeros((N, K // 8), dtype=np.uint32)
    for t in range(2):
        for beta in range(4):
            P |= u[:, :, t, beta] << np.uint32(8 * beta + 4 * t)
    return P


def unpack_qw4(P: np.ndarray, K: int) -> np.ndarray:
    N = P.shape[0]
    u = np.empty((N, K // 8, 2, 4), dtype=np.int64)
    for t in range(2):
        for beta in range(4):
            u[:, :, t, beta] = (P >> np.uint32(8 * beta + 4 * t)) & np.uint32(15)
    return (u.reshape(N, K) - 8).astype(np.int8)


def pack(L: np.ndarray, fmt: int) -> np.ndarray:
    return pack_qw4(L) if fmt == levels.FMT_W4_SYM else pack_qw2(L, fmt)


def unpack(P: np.ndarray, fmt: int, K: int) -> np.ndarray:
    return unpack_qw4(P, K) if fmt == levels.FMT_W4_SYM else unpack_qw2(P, fmt, K)


def packed_bytes(fmt: int, N: int, K: int) -> int:
    return N * K // 2 if fmt == levels.FMT_W4_SYM else N * K // 4
