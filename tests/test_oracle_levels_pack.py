"""Pins of the oracle's level sets and packers against the paper's constants and hand-derived words."""
import json
import os

import numpy as np
import pytest

from oracle import levels, pack


def _load(golden_dir, name):
    with open(os.path.join(golden_dir, name)) as f:
        return json.load(f)


def test_level_sets_match_paper(golden_dir):
    g = _load(golden_dir, "level_sets.json")
    assert levels.SYM == tuple(g["SYM"])
    assert levels.MNZ == tuple(g["MNZ"])
    assert levels.MNZ_HALF == tuple(g["MNZ_half_scale_odd_levels"])
    assert levels.LLOYD == tuple(g["LLOYD"])
    assert levels.NF2 == tuple(g["NF2"])
    assert levels.POT == tuple(g["POT"])
    assert levels.FAR_MNZ == tuple(g["FAR_MNZ"])


def test_half_scale_identity():
    # {-1.5,-0.5,0.5,1.5} * s == {-3,-1,1,3} * s/2 for any scale
    for s in (1.0, 0.37, 2.0 ** -7, 123.5):
        assert [v * s for v in levels.MNZ] == [v * (s / 2) for v in levels.MNZ_HALF]


def test_midpoint_identity_gives_code_assignment(golden_dir):
    # unsigned codes {0,1,2,3} minus the midpoint z=1.5 are exactly MNZ; doubled they are the
    # half-scale odd levels, i.e. the ascending-index code assignment level = 2c - 3
    g = _load(golden_dir, "level_sets.json")
    z = g["asym_midpoint_z"]
    assert [c - z for c in g["asym_unsigned_codes"]] == list(levels.MNZ)
    for c in range(4):
        assert levels.code_to_level(levels.FMT_W2_MNZ, c) == 2 * c - 3
    # PoT: sign bit is c>>1, outer magnitude iff both bits agree
    for c in range(4):
        lev = levels.code_to_level(levels.FMT_W2_POT, c)
        assert (lev > 0) == bool(c >> 1)
        assert (abs(lev) == 4) == ((c >> 1) == (c & 1))


def test_inner_outer_ratios_match_table(golden_dir):
    rows = _load(golden_dir, "ratio_table.json")["rows"]
    for name in ("LLOYD", "MNZ", "NF2", "POT", "FAR_MNZ"):
        r = levels.inner_outer_ratio(getattr(levels, name))
        assert round(r, 4) == pytest.approx(rows[name]["r"], abs=1e-4), name
    assert levels.inner_outer_ratio(levels.MNZ) == pytest.approx(1 / 3)
    assert levels.inner_outer_ratio(levels.POT) == 0.25
    with pytest.raises(ValueError):
        levels.inner_outer_ratio(levels.SYM)          # has a zero level
    assert levels.mirror_family(0.25) == (-1.0, -0.25, 0.25, 1.0)


def _case_levels(case):
    L = np.full((1, case["K"]), case["default"], dtype=np.int8)
    for k, v in case["set"]:
        L[0, k] = v
    return L


def test_pack_hand_derived_words(golden_dir):
    for case in _load(golden_dir, "pack_examples.json")["cases"]:
        L = _case_levels(case)
        P = pack.pack(L, case["fmt"])
        want = np.array([int(w, 16) for w in case["words"]], dtype=np.uint32)
        assert P.dtype == np.uint32
        assert np.array_equal(P[0], want), case["why"]
        assert np.array_equal(pack.unpack(P, case["fmt"], case["K"]), L)


def _unpack_bruteforce_qw2(P, fmt, K):
    """Per-element bit extraction with Python integers (independent decoder)."""
    out = []
    for row in P:
        vals = []
        for k in range(K):
            j, r = divmod(k, 16)
            t, beta = divmod(r, 4)
            c = (int(row[j]) >> (8 * beta + 2 * t)) & 3
            vals.append(levels.CODE_LEVELS[fmt][c])
        out.append(vals)
    return np.array(out, dtype=np.int8)


def _unpack_bruteforce_qw4(P, K):
    out = []
    for row in P:
        vals = []
        for k in range(K):
            j, r = divmod(k, 8)
            t, beta = divmod(r, 4)
            vals.append(((int(row[j]) >> (8 * beta + 4 * t)) & 15) - 8)
        out.append(vals)
    return np.array(out, dtype=np.int8)


@pytest.mark.parametrize("fmt", [levels.FMT_W2_MNZ, levels.FMT_W2_POT])
def test_qw2_roundtrip_bruteforce(fmt):
    rng = np.random.default_rng(7)
    table = np.array(levels.CODE_LEVELS[fmt], dtype=np.int8)
    L = table[rng.integers(0, 4, size=(5, 128))]
    P = pack.pack_qw2(L, fmt)
    assert P.shape == (5, 8)
    assert np.array_equal(_unpack_bruteforce_qw2(P, fmt, 128), L)
    assert np.array_equal(pack.unpack_qw2(P, fmt, 128), L)


def test_qw4_roundtrip_bruteforce():
    rng = np.random.default_rng(8)
    q = rng.integers(-7, 8, size=(5, 128)).astype(np.int8)
    P = pack.pack_qw4(q)
    assert P.shape == (5, 16)
    assert np.array_equal(_unpack_bruteforce_qw4(P, 128), q)
    assert np.array_equal(pack.unpack_qw4(P, 128), q)


def test_byte_lane_property_of_qw2():
    # (P >> 2t) & 0x03030303 holds the codes of k = 16j+4t .. 16j+4t+3 in byte lanes 0..3
    rng = np.random.default_rng(9)
    L = np.array(levels.MNZ_HALF, dtype=np.int8)[rng.integers(0, 4, size=(3, 64))]
    P = pack.pack_qw2(L, levels.FMT_W2_MNZ)
    codes = (L.astype(np.int64) + 3) // 2
    for n in range(3):
        for j in range(4):
            for t in range(4):
                w = (int(P[n, j]) >> (2 * t)) & 0x03030303
                lanes = [(w >> (8 * b)) & 0xFF for b in range(4)]
                assert lanes == list(codes[n, 16 * j + 4 * t: 16 * j + 4 * t + 4])


def test_pack_rejects_bad_levels_and_shapes():
    with pytest.raises(ValueError):
        pack.pack_qw2(np.zeros((1, 64), dtype=np.int8), levels.FMT_W2_MNZ)   # 0 is not an MNZ level
    with pytest.raises(ValueError):
        pack.pack_qw2(np.full((1, 64), 3, dtype=np.int8), levels.FMT_W2_POT)  # 3 is not a PoT level
    with pytest.raises(ValueError):
        pack.pack_qw4(np.full((1, 64), -8, dtype=np.int8))                   # -8 outside -7..7
    with pytest.raises(ValueError):
        pack.pack_qw2(np.ones((1, 48), dtype=np.int8), levels.FMT_W2_MNZ)    # K % 64 != 0


def test_average_bits_of_mixed_schedule(golden_dir):
    # packed bytes of an L-layer W4 / (32-L)-layer W2 stack reproduce b_avg = 2 + L/16
    g = _load(golden_dir, "mixed_l.json")
    N, K = 512, 256
    for L, bavg in g["cases"]:
        total = L * pack.packed_bytes(levels.FMT_W4_SYM, N, K) + \
            (g["layers"] - L) * pack.packed_bytes(levels.FMT_W2_MNZ, N, K)
        assert 8 * total / (g["layers"] * N * K) == pytest.approx(bavg)
