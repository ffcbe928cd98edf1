"""Validity rule for weight-quantizer results whose rotation is inexact (test helper).

The quantizer rotates fp32 rows, w = (I (x) H_b) W / sqrt(b), in fp64.  The sums are not exact, and
two implementations that add in different orders (the oracle's dense product, the GPU's butterflies)
can differ in the last bits of w.  A decision taken on such bits may then go either way: a level whose
w lies within rounding of a level threshold, a scale whose unrounded value lies within rounding of an
fp16 rounding midpoint, or a PoT scale where two candidates' squared errors lie within rounding of each
other (Sec. 3.3, Eqs. (13)-(14) and (17); Eq. (1)).

Bound.  Either side's rotated value differs from the exact one by at most
    e = (b + log2(b) + 8) u S / sqrt(b),   u = 2^-53,   S = sum over the block of |W|,
which covers a b-term fp64 sum in any order ((b - 1) u S for a sequential order, less for butterflies),
the scaling by 1/sqrt(b) and a margin; so the two sides differ by at most d = 2e.

Rule.  A result (levels L, fp16 scales s) is valid for a row when:
  * its scale equals the oracle's, or both are adjacent fp16 values whose rounding midpoint lies within
    the propagated bound of the oracle's unrounded scale (MNZ: RMS / 2; W4: max / 7), or, for PoT, the
    scale is the fp16 rounding of a candidate whose squared error is within the propagated bound of the
    oracle's minimum (and whose unrounded value maps to that fp16 within the bound);
  * every level equals the oracle's level against that scale, except where the oracle's w lies within d
    (plus the division's rounding) of the threshold between the two levels, which must be adjacent.
The mirror family G(r) = {-1, -r, +r, +1} (Sec. 3.4 Eq. (18), fmt MIRROR with its ratio r) takes the PoT
rule with outer level 1 (candidates c max|w|, threshold (1 + r) / 2) and is checked on its codes 0..3.
Everything here uses the oracle's functions; nothing comes from the GPU but the result under test.
"""
from __future__ import annotations

import numpy as np

from oracle import hadamard, levels, quant

U = 2.0 ** -53

MIRROR = "mirror"

LEVELS = {levels.FMT_W2_MNZ: np.array([-3, -1, 1, 3]), levels.FMT_W2_POT: np.array([-4, -1, 1, 4]),
          levels.FMT_W4_SYM: np.arange(-7, 8), MIRROR: np.arange(4)}
# thresholds in units of the scale between consecutive levels of LEVELS[fmt]
THRESH = {levels.FMT_W2_MNZ: np.array([-2.0, 0.0, 2.0]), levels.FMT_W2_POT: np.array([-2.5, 0.0, 2.5]),
          levels.FMT_W4_SYM: np.arange(-7, 7) + 0.5}


def _thresh(fmt, r):
    if fmt == MIRROR:
        t = 0.5 * (r + 1.0)
        return np.array([-t, 0.0, t])
    return THRESH[fmt]


def _oracle_quantize(fmt, w, r):
    if fmt == MIRROR:
        return quant.quantize_mirror_mse(w, r)
    return quant.quantize_weights(w, fmt)


def rotation_bound(W: np.ndarray, b: int) -> np.ndarray:
    """d[n, k]: bound on the difference between two sides' fp64 rotated values of W[n, k]."""
    W = np.asarray(W, np.float64)
    N, K = W.shape
    S = np.abs(W).reshape(N, K // b, b).sum(axis=2) * (1.0 + 2.0 * b * U)
    e = (b + np.log2(b) + 8.0) * U * S / np.sqrt(b) * 1.01
    return 2.0 * np.repeat(e, b, axis=1)


def levels_against(fmt, w: np.ndarray, s: float, r: float | None = None) -> np.ndarray:
    """The oracle's levels (G(r): codes) of the rotated row w against the fp16 scale s."""
    if fmt == MIRROR:
        return quant.mirror_codes(w, s, r).astype(np.int64)
    if s == 0:
        return np.full(w.shape, 0 if fmt == levels.FMT_W4_SYM else 1, dtype=np.int64)
    if fmt == levels.FMT_W2_MNZ:
        return quant.nearest_mirror(w / s, 1.0, 3.0).astype(np.int64)
    if fmt == levels.FMT_W2_POT:
        return quant.pot_level(w, s).astype(np.int64)
    return np.clip(quant.rne(w / s), -7, 7).astype(np.int64)


def levels_valid(fmt, w: np.ndarray, d: np.ndarray, s: float, L: np.ndarray, r: float | None = None) -> str | None:
    """None if the levels L of row w against scale s satisfy the rule, else a reason."""
    ref = levels_against(fmt, w, s, r)
    bad = np.nonzero(np.asarray(L, np.int64) != ref)[0]
    if bad.size == 0:
        return None
    if s == 0:
        return "levels of a zero-scale row"
    lv, th = LEVELS[fmt], _thresh(fmt, r)
    for k in bad:
        i, j = np.searchsorted(lv, int(L[k])), np.searchsorted(lv, int(ref[k]))
        if i >= lv.size or lv[i] != L[k] or abs(int(i) - int(j)) != 1:
            return f"element {k}: level {int(L[k])} is not next to the oracle's {int(ref[k])}"
        t = th[min(i, j)]
        u = w[k] / s
        du = d[k] / s + 4.0 * U * abs(u) + 4.0 * U
        if abs(u - t) > du:
            return f"element {k}: w/s = {u!r} is {abs(u - t):.3e} from the threshold {t}, beyond {du:.3e}"
    return None


def _adjacent_midpoint(s_a: np.float16, s_b: np.float16):
    """Rounding midpoint between two adjacent fp16 values, or None if they are not adjacent."""
    ia, ib = int(np.float16(s_a).view(np.uint16)), int(np.float16(s_b).view(np.uint16))
    if (ia >> 15) != (ib >> 15) or abs(ia - ib) != 1:
        return None
    return 0.5 * (float(s_a) + float(s_b))


def _rounding_ok(x: float, bound: float, s_ref: np.float16, s_got: np.float16) -> str | None:
    """The unrounded scale x (oracle) within bound of the midpoint between the oracle's and the result's
    fp16 values."""
    m = _adjacent_midpoint(s_ref, s_got)
    if m is None:
        return f"scale {float(s_got)!r} is not adjacent to the oracle's {float(s_ref)!r}"
    if abs(x - m) > bound:
        return f"unrounded scale {x!r} is {abs(x - m):.3e} from the midpoint {m!r}, beyond {bound:.3e}"
    return None


def _search(fmt, r):
    """(candidate factor, level function of (w, s), threshold in units of s, outer - inner magnitude) of
    the 64-candidate search: PoT levels 1, 4 at c max / 4, G(r) levels r, 1 at c max."""
    if fmt == MIRROR:
        return 1.0, (lambda w, s: quant.nearest_mirror(w / s, r, 1.0)), 0.5 * (r + 1.0), 1.0 - r
    return 0.25, quant.pot_level, 2.5, 3.0


def _pot_errors(w, d, a, da, fmt=levels.FMT_W2_POT, rr=None):
    """Squared errors of the 64 candidates on row w (oracle arithmetic) and a bound on how far either
    side's value of each can be from the exact one."""
    K = w.size
    f, level_fn, thr, jump = _search(fmt, rr)
    errs, bounds, cands = [], [], []
    for c in quant.POT_CANDIDATES:
        s = c * a * f
        ds = c * da * f + 4.0 * U * s
        lev = level_fn(w, s)
        r = w - s * lev
        err = float(np.sum(r * r))
        dr = d + np.abs(lev) * ds
        # a level that flips within d of the threshold changes that term continuously (both residuals
        # are equal at the threshold): at most 2 |r| dr + 2 (outer - inner) s dr there
        near = np.abs(np.abs(w) - thr * s) <= d + thr * ds
        bound = float(np.sum(2.0 * np.abs(r) * dr + dr * dr) + np.sum(2.0 * jump * s * dr[near])
                      + 4.0 * K * U * err) + 1e-300
        errs.append(err)
        bounds.append(bound)
        cands.append(s)
    return np.array(errs), np.array(bounds), np.array(cands)


def row_valid(fmt, w: np.ndarray, d: np.ndarray, s_got: np.float16, L_got: np.ndarray,
              r: float | None = None) -> str | None:
    """None if (s_got, L_got) is a valid result for the oracle-rotated row w with difference bound d."""
    w = np.asarray(w, np.float64)
    K = w.size
    _, s_ref = _oracle_quantize(fmt, w[None, :], r)
    s_ref = s_ref[0]
    s_got = np.float16(s_got)
    if s_got.view(np.uint16) != s_ref.view(np.uint16):
        if fmt == levels.FMT_W2_MNZ:
            ss = float(np.sum(w * w))
            dss = float(np.sum(2.0 * np.abs(w) * d + d * d)) + 4.0 * K * U * ss
            rms = np.sqrt(ss / K)
            bound = (dss / (2.0 * K * max(rms, 1e-300))) / 2.0 + 8.0 * U * rms
            why = _rounding_ok(rms / 2.0, bound, s_ref, s_got)
        elif fmt == levels.FMT_W4_SYM:
            a = float(np.abs(w).max())
            why = _rounding_ok(a / 7.0, float(d.max()) / 7.0 + 4.0 * U * a, s_ref, s_got)
        else:
            a = float(np.abs(w).max())
            da = float(d.max())
            errs, bounds, cands = _pot_errors(w, d, a, da, fmt, r)
            f = _search(fmt, r)[0]
            jr = int(np.argmin(errs))
            why = "no PoT candidate rounds to the scale within its bound"
            for j in range(len(cands)):
                # the candidate's unrounded value may round to s_got ...
                m_lo = float(s_got) - abs(float(s_got)) * 2.0 ** -11 - 2.0 ** -25
                m_hi = float(s_got) + abs(float(s_got)) * 2.0 ** -11 + 2.0 ** -25
                slack = quant.POT_CANDIDATES[j] * da * f + 4.0 * U * cands[j]
                if not (m_lo - slack <= cands[j] <= m_hi + slack):
                    continue
                # ... and its error is within the bounds of the oracle's minimum
                if errs[j] - errs[jr] <= bounds[j] + bounds[jr]:
                    why = None
                    break
        if why is not None:
            return "scale: " + why
    return levels_valid(fmt, w, d, float(s_got), L_got, r)


def check_rows(fmt, W: np.ndarray, b: int, L_got: np.ndarray, s_got: np.ndarray, r: float | None = None):
    """Oracle result for the fp32 rows W, and the rows where the result under test differs from it but
    satisfies the rule.  Raises AssertionError at the first row that violates the rule."""
    W = np.asarray(W, np.float32)
    w = hadamard.rotate_weights(W.astype(np.float64), b)
    L_ref, s_ref = _oracle_quantize(fmt, w, r)
    differ = np.nonzero((np.asarray(s_got).view(np.uint16) != s_ref.view(np.uint16)) |
                        np.any(np.asarray(L_got) != L_ref, axis=1))[0]
    if differ.size:
        d = rotation_bound(W, b)
        for n in differ:
            why = row_valid(fmt, w[n], d[n], s_got[n], L_got[n], r)
            assert why is None, f"row {n}: {why}"
    return L_ref, s_ref, differ
