"""Quantizers: per-token INT4 activations and per-output-channel weights.

Activations (Sec. 4.1 "Quantization configuration": symmetric 4-bit):
    per token, ``q = clip(round(X / s_x), -7, 7)`` on the rotated token with
    ``s_x = c * max|X| / 7``.  Readings: rounding is round-half-to-even; the
    range is the symmetric -7..7; the clip ratio ``c`` defaults to 1 (``c = 9/10``
    is the paper's setting and is supported as an exact rational).

Weights (Sec. 3.3, Sec. 3.5, Sec. 4.5.1): one scale per output channel and the
nearest level of a fixed set, no zero-point, no groups.  Scale rules:

* MNZ:  ``s = RMS(row)``; stored half scale ``s_w = fp16(s / 2)`` (Eq. (14)).
* PoT-MNZ: first minimiser of the squared error over 64 candidate scales
  ``linspace(0.2, 1.0, 64) * max|row| / 4``; ``s_w = fp16(best)``.
* W4: ``s_w = fp16(max|row| / 7)``; ``q = clip(round(w / s_w), -7, 7)`` (Eq. (1)).

Levels are always assigned against the *stored* fp16 scale.  Tie reading for the
four-level sets: a value exactly on the midpoint between an inner and an outer
level takes the inner level; zero takes the positive inner level.
"""
from __future__ import annotations

import numpy as np

from . import hadamard, levels

# ---------------------------------------------------------------------------
# activations
# ---------------------------------------------------------------------------


def act_scale_denominator(b: int, clip=(1, 1)) -> float:
    """``(den * 7) * sqrt(b)`` in fp64, the fixed divisor of the per-token scale."""
    num, den = clip
    return (float(den) * 7.0) * float(np.sqrt(np.float64(b)))


def act_quant(x: np.ndarray, b: int, clip=(1, 1)):
    """Rotate and quantize fp16 tokens [M, K] to INT4.

    Steps per token m (unnormalised rotation, see :mod:`oracle.hadamard`):

    1. ``X = (I (x) H_b) x_m`` exactly, in integer units ``u = 2^-24``.
    2. ``A = max_k |X_k|``.
    3. ``q_k = sign(X_k) * min(7, rne(7 |X_k| / (c A)))`` with ``c = num/den``,
       evaluated in exact integer arithmetic:
       ``t = 14 den |X|``, ``d = 2 num A``, ``q0 = floor((t + num A) / d)``, and
       when ``t + num A`` is a multiple of ``d`` (an exact half) an odd ``q0`` is
       lowered by one.  ``A = 0`` gives ``q = 0``.
    4. ``s_x = fp32( (A u num) / ((den 7) sqrt(b)) )``, i.e. ``c max|X| / (7 sqrt(b))``
       of the normalised rotation, each fp64 operation rounded in that order.
    5. ``sum_q = sum_k q_k`` (int32).

    Returns ``(q int8 [M,K], s_x fp32 [M], sum_q int32 [M], X int64 [M,K])``.
    """
    num, den = int(clip[0]), int(clip[1])
    if not (1 <= num <= den <= 16):
        raise ValueError("clip ratio must be num/den with 1 <= num <= den <= 16")
    X = hadamard.rotate_act_units(x, b)
    M, K = X.shape
    absX = np.abs(X)
    A = absX.max(axis=1) if K else np.zeros(M, dtype=np.int64)
    assert np.all(A < 2 ** 53)
    q = np.zeros((M, K), dtype=np.int64)
    for m in range(M):
        a = int(A[m])
        if a == 0:
            continue
        t = 14 * den * absX[m] + num * a
        d = 2 * num * a
        q0 = t // d
        tie = (t % d) == 0
        q0 = q0 - (tie & (q0 % 2 == 1))
        q0 = np.minimum(q0, 7)
        q[m] = np.where(X[m] < 0, -q0, q0)
    numer = A.astype(np.float64) * 2.0 ** -24 * float(num)
    s_x = (numer / act_scale_denominator(b, (num, den))).astype(np.float32)
    return q.astype(np.int8), s_x, q.sum(axis=1).astype(np.int32), X


def act_quant_staged(x: np.ndarray, b: int, clip=(1, 1)):
    """Rotate and quantize tokens [M, K] of any finite binary floats (bf16 activations included).

    Reading for inputs off the 2^-24 grid (bf16 values below 2^-17 or from 2^16 in magnitude), where
    the paper fixes no precision and an fp64 rotation is not exact in general: ``X`` is the fp64 value
    of the unnormalised block transform computed stage by stage over the index bits 0, 1, ..., L - 1
    (:func:`oracle.hadamard.rotate_act_staged`); then, exactly on those fp64 numbers taken as
    rationals, ``A = max |X|``, ``q = sign(X) min(7, rne(7 den |X| / (num A)))`` (a half rounds to the
    even integer), ``s_x = fp32(fp64(A num) / ((den 7) sqrt(b)))`` and ``sum_q``.  On the 2^-24 grid
    every partial sum is exact, so this is :func:`act_quant` there.

    Returns ``(q int8 [M,K], s_x fp32 [M], sum_q int32 [M], X fp64 [M,K])``.
    """
    from fractions import Fraction
    num, den = int(clip[0]), int(clip[1])
    if not (1 <= num <= den <= 16):
        raise ValueError("clip ratio must be num/den with 1 <= num <= den <= 16")
    X = hadamard.rotate_act_staged(x, b)
    M, K = X.shape
    q = np.zeros((M, K), dtype=np.int64)
    A = np.abs(X).max(axis=1) if K else np.zeros(M)
    for m in range(M):
        a = Fraction(float(A[m]))
        if a == 0:
            continue
        for k in range(K):
            t = 14 * den * abs(Fraction(float(X[m, k]))) + num * a
            d = 2 * num * a
            q0 = t // d
            if t % d == 0 and q0 % 2 == 1:
                q0 -= 1
            q0 = min(int(q0), 7)
            q[m, k] = -q0 if X[m, k] < 0 else q0
    s_x = ((A.astype(np.float64) * float(num)) / act_scale_denominator(b, (num, den))).astype(np.float32)
    return q.astype(np.int8), s_x, q.sum(axis=1).astype(np.int32), X


# ---------------------------------------------------------------------------
# nearest level
# ---------------------------------------------------------------------------


def nearest_mirror(u: np.ndarray, inner: float, outer: float) -> np.ndarray:
    """Nearest level of ``{-outer, -inner, +inner, +outer}`` to ``u``.

    Sign from ``u >= 0`` (zero goes positive); the outer magnitude only when
    ``|u|`` lies strictly beyond the midpoint ``(inner + outer) / 2``.
    """
    u = np.asarray(u, dtype=np.float64)
    mag = np.where(np.abs(u) > 0.5 * (inner + outer), outer, inner)
    return np.where(u >= 0, mag, -mag)


def nearest_bruteforce(u: np.ndarray, levels_) -> np.ndarray:
    """Nearest level by exhaustive search (first minimum); used by pins and diagnostics."""
    L = np.asarray(levels_, dtype=np.float64)
    u = np.asarray(u, dtype=np.float64)
    return L[np.argmin(np.abs(u[..., None] - L), axis=-1)]


def fp16_scale(s: np.ndarray) -> np.ndarray:
    """Stored per-channel scale: fp64 value rounded once to fp16."""
    return np.asarray(s, dtype=np.float64).astype(np.float16)


# ---------------------------------------------------------------------------
# weights (offline, per output channel)
# ---------------------------------------------------------------------------


def quantize_mnz_rms(W_rot: np.ndarray):
    """MNZ with the row-RMS scale at half scale.  Returns (levels int8 in {-3,-1,1,3}, s_w fp16).

    ``s = sqrt(mean_k W_rot[n,k]^2)``; ``s_w = fp16(s/2)``; level = nearest of
    ``{-3,-1,+1,+3}`` to ``W_rot / s_w`` (midpoints at 0 and +-2).  A row whose
    stored scale is 0 gets level +1 everywhere.
    """
    W = np.asarray(W_rot, dtype=np.float64)
    s = np.sqrt(np.mean(W * W, axis=1))
    s_w = fp16_scale(s / 2.0)
    sw64 = s_w.astype(np.float64)
    L = np.ones(W.shape, dtype=np.int8)
    nz = sw64 > 0
    u = W[nz] / sw64[nz, None]
    L[nz] = nearest_mirror(u, 1.0, 3.0).astype(np.int8)
    return L, s_w


POT_CANDIDATES = np.linspace(0.2, 1.0, 64)


def pot_level(w: np.ndarray, s: np.ndarray) -> np.ndarray:
    """PoT-MNZ level of ``w`` against scale ``s``: sign(w) * (4 if |w|/s > 2.5 else 1), sign(0) = +."""
    return nearest_mirror(np.asarray(w, np.float64) / np.asarray(s, np.float64), 1.0, 4.0)


def quantize_pot_mse(W_rot: np.ndarray):
    """PoT-MNZ with the 64-candidate MSE scale search.  Returns (levels int8 in {-4,-1,1,4}, s_w fp16)."""
    W = np.asarray(W_rot, dtype=np.float64)
    N, K = W.shape
    a = np.abs(W).max(axis=1)
    L = np.ones((N, K), dtype=np.int8)
    s_w = np.zeros(N, dtype=np.float16)
    for n in range(N):
        if a[n] == 0.0:
            continue
        cand = POT_CANDIDATES * a[n] / 4.0
        err = np.empty(len(cand))
        for j, s in enumerate(cand):
            lev = pot_level(W[n], s)
            err[j] = np.sum((W[n] - s * lev) ** 2)
        best = cand[int(np.argmin(err))]
        s_w[n] = fp16_scale(best)
        if s_w[n] > 0:
            L[n] = pot_level(W[n], float(s_w[n])).astype(np.int8)
    return L, s_w


def quantize_mirror_mse(W_rot: np.ndarray, r: float):
    """Mirror-family set ``G(r) = {-1, -r, +r, +1}`` (Sec. 3.4 Eq. (18)) with the 64-candidate MSE scale of
    the PoT rule: ``s`` over ``linspace(0.2, 1.0, 64) * max|row|`` (the outer level is 1), first
    minimiser of ``sum (w - s * level(w, s))^2``, stored ``s_w = fp16(best)``, levels by
    :func:`nearest_mirror` against the stored scale (inner/outer midpoint ``(1 + r) / 2``, zero to the
    positive inner level).  Returns (codes int8 in 0..3 for the ascending levels -1, -r, +r, +1; s_w
    fp16).  A row whose stored scale is 0 gets code 2 (+r)."""
    levels.mirror_family(r)   # validates r
    W = np.asarray(W_rot, dtype=np.float64)
    N, K = W.shape
    a = np.abs(W).max(axis=1)
    codes = np.full((N, K), 2, dtype=np.int8)
    s_w = np.zeros(N, dtype=np.float16)
    for n in range(N):
        if a[n] == 0.0:
            continue
        cand = POT_CANDIDATES * a[n]
        err = np.empty(len(cand))
        for j, s in enumerate(cand):
            lev = nearest_mirror(W[n] / s, r, 1.0)
            err[j] = np.sum((W[n] - s * lev) ** 2)
        s_w[n] = fp16_scale(cand[int(np.argmin(err))])
        codes[n] = mirror_codes(W[n], float(s_w[n]), r)
    return codes, s_w


def mirror_codes(w: np.ndarray, s: float, r: float) -> np.ndarray:
    """Codes 0..3 (ascending levels -1, -r, +r, +1) of :func:`nearest_mirror` of ``w / s`` with
    inner ``r`` and outer 1; all 2 (+r) when ``s == 0``."""
    w = np.asarray(w, dtype=np.float64)
    if s == 0:
        return np.full(w.shape, 2, dtype=np.int8)
    lev = nearest_mirror(w / s, r, 1.0)
    return np.where(lev >= 0, np.where(lev == 1.0, 3, 2), np.where(lev == -1.0, 0, 1)).astype(np.int8)


def ratio_scan(x: np.ndarray, ratios, cands):
    """Ratio-scan diagnostic (Sec. 4.5.3): for each mirror ratio r, the squared error of ``G(r)`` on the
    samples x at every scale ``c * max|x|`` of the candidate clip ratios ``cands`` (levels by
    :func:`nearest_mirror` of ``x / s``), and the best-scale NMSE ``min_c sse / sum x^2`` (first
    minimiser).  Returns (sse [n_ratios, n_cands], nmse [n_ratios], best index [n_ratios], (max|x|,
    sum x^2)).  All-zero samples have no error: sse and nmse 0; nmse is 0 too where sum x^2 is 0 (squares
    below the fp64 range)."""
    x = np.asarray(x, dtype=np.float64).ravel()
    a = float(np.abs(x).max())
    sx2 = float(np.sum(x * x))
    sse = np.zeros((len(ratios), len(cands)))
    if a == 0.0:
        return sse, np.zeros(len(ratios)), np.zeros(len(ratios), dtype=np.int64), (a, sx2)
    for i, r in enumerate(ratios):
        for j, c in enumerate(cands):
            s = float(c) * a
            lev = nearest_mirror(x / s, float(r), 1.0)
            sse[i, j] = np.sum((x - s * lev) ** 2)
    best = np.argmin(sse, axis=1)
    nmse = sse[np.arange(len(ratios)), best] / sx2 if sx2 > 0 else np.zeros(len(ratios))
    return sse, nmse, best, (a, sx2)


def rne(v: np.ndarray) -> np.ndarray:
    """Round half to even, written out on |v| (the rounding is odd-symmetric): f = floor(|v|) and the
    fractional part |v| - f, which is exact in fp64; round up when it exceeds 1/2, or equals 1/2 with
    f odd.  (Adding 1/2 before the floor would itself round for |v| within an ulp below a half.)"""
    v = np.asarray(v, dtype=np.float64)
    a = np.abs(v)
    f = np.floor(a)
    frac = a - f
    up = (frac > 0.5) | ((frac == 0.5) & (np.mod(f, 2.0) == 1.0))
    return np.copysign(f + up, v)


def quantize_w4_absmax(W_rot: np.ndarray):
    """Symmetric W4 (Eq. (1), b=4, range -7..7): ``s_w = fp16(max|row|/7)``.  Returns (q int8, s_w fp16)."""
    W = np.asarray(W_rot, dtype=np.float64)
    s_w = fp16_scale(np.abs(W).max(axis=1) / 7.0)
    sw64 = s_w.astype(np.float64)
    q = np.zeros(W.shape, dtype=np.int8)
    nz = sw64 > 0
    q[nz] = np.clip(rne(W[nz] / sw64[nz, None]), -7, 7).astype(np.int8)
    return q, s_w


def quantize_weights(W_rot: np.ndarray, fmt: int):
    if fmt == levels.FMT_W2_MNZ:
        return quantize_mnz_rms(W_rot)
    if fmt == levels.FMT_W2_POT:
        return quantize_pot_mse(W_rot)
    if fmt == levels.FMT_W4_SYM:
        return quantize_w4_absmax(W_rot)
    raise ValueError(f"unknown format {fmt}")


def mse_scale_search(w: np.ndarray, grid, ratios=np.linspace(0.05, 1.0, 400)):
    """Reference RTN: best scale for ``grid`` over clip ratios of ``max|w| / max|grid|`` (Sec. 4.5.1).

    Used by the statistical pins only.  Returns (best scale, dequantized values).
    """
    w = np.asarray(w, dtype=np.float64)
    gmax = max(abs(g) for g in grid)
    a = np.abs(w).max()
    best = (np.inf, None, None)
    for r in ratios:
        s = r * a / gmax
        wq = s * nearest_bruteforce(w / s, grid)
        e = np.sum((w - wq) ** 2)
        if e < best[0]:
            best = (e, s, wq)
    return best[1], best[2]
