"""Four-level W2 reconstruction level sets and the W4 set.

* SYM-INT ``{-2,-1,0,+1}``: the b=2 case of the symmetric integer quantizer,
  Sec. 1 Eqs. (1)-(2).
* MNZ ``{-1.5,-0.5,+0.5,+1.5}``: the proposed mirror no-zero set, Sec. 1 Eq. (3)
  and Sec. 3.3 Eq. (13); written as odd integers ``{-3,-1,+1,+3}`` times a
  half scale ``s/2`` (Sec. 3.3 Eq. (14)).
* PoT-MNZ ``{-4,-1,+1,+4}``: Sec. 1 Eq. (4), Sec. 3.3 Eq. (17).
* Reference grids Lloyd-Max, NF2 and Far-MNZ: Sec. 3.3 Eqs. (9), (10), (12).
* Mirror family ``G(r) = {-1,-r,+r,+1}``: Sec. 3.4 Eq. (18).
* W4: Eq. (1) with b=4, used here on the symmetric range -7..7 (the -8 code
  is never produced; see the readings in the design notes).

The implementation assigns 2-bit code ``c`` to the c-th level of the ascending
list (the paper leaves the code-to-level assignment free, Sec. 3.3).  For MNZ
this is the unsigned code of the asymmetric quantizer with the fractional
midpoint ``z = 1.5`` (Sec. 3.3 Eqs. (15)-(16)): level = 2c - 3 at half scale.
"""
from __future__ import annotations

SYM = (-2.0, -1.0, 0.0, 1.0)
MNZ = (-1.5, -0.5, 0.5, 1.5)
MNZ_HALF = (-3, -1, 1, 3)
POT = (-4, -1, 1, 4)
LLOYD = (-1.5104, -0.4528, 0.4528, 1.5104)
NF2 = (-1.0, -0.2525685, 0.2525685, 1.0)
FAR_MNZ = (-2.0, -1.0, 1.0, 2.0)
W4 = tuple(range(-7, 8))

# format ids shared with the C ABI's numbering (a plain enumeration)
FMT_W2_MNZ = 0
FMT_W2_POT = 1
FMT_W4_SYM = 2
# any four levels read through a table indexed by the 2-bit code (the reference grids of Sec. 3.3,
# which are not integers): the packed "levels" are the codes themselves
FMT_W2_LUT = 3

CODE_LEVELS = {FMT_W2_MNZ: MNZ_HALF, FMT_W2_POT: POT, FMT_W2_LUT: (0, 1, 2, 3)}


def mirror_family(r: float):
    """``G(r) = {-1, -r, +r, +1}`` with outer magnitude normalised to one (Eq. (18))."""
    if not 0.0 < r < 1.0:
        raise ValueError("ratio must lie in (0, 1)")
    return (-1.0, -r, r, 1.0)


def inner_outer_ratio(levels) -> float:
    """Inner/outer centroid ratio of a mirror no-zero set (Sec. 3.4)."""
    mags = sorted({abs(v) for v in levels})
    if len(mags) != 2 or mags[0] == 0.0:
        raise ValueError("not a mirror no-zero four-level set")
    return mags[0] / mags[1]


def code_to_level(fmt: int, c: int) -> int:
    """Level of 2-bit code ``c`` under the ascending-index assignment."""
    return CODE_LEVELS[fmt][c]
