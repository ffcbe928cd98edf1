"""Pins of the weight quantizer's validity rule (tests/wquant_rule.py) on the CPU: the oracle's own
result passes; a level moved away from the oracle's where the rotated value is not near a threshold, a
level two steps away, and a scale that is not the rounding of a value near a midpoint are rejected;
the other side of an exact threshold is accepted."""
import numpy as np
import pytest

from oracle import hadamard, levels, quant
from paper_2606_02823_amd import synth
from wquant_rule import check_rows, row_valid, rotation_bound

FMTS = [levels.FMT_W2_MNZ, levels.FMT_W2_POT, levels.FMT_W4_SYM]


def _oracle(W, b, fmt):
    return quant.quantize_weights(hadamard.rotate_weights(np.asarray(W, np.float64), b), fmt)


@pytest.mark.parametrize("fmt", FMTS)
def test_oracle_result_passes(fmt):
    W = synth.weights_fp32(97, 0, "q", 24, 512)
    L, s = _oracle(W, 256, fmt)
    _, _, differ = check_rows(fmt, W, 256, L, s)
    assert differ.size == 0


@pytest.mark.parametrize("fmt", FMTS)
def test_planted_level_far_from_threshold_is_rejected(fmt):
    W = synth.weights_fp32(97, 1, "q", 8, 256)
    L, s = _oracle(W, 256, fmt)
    w = hadamard.rotate_weights(W.astype(np.float64), 256)
    lv = {levels.FMT_W2_MNZ: [-3, -1, 1, 3], levels.FMT_W2_POT: [-4, -1, 1, 4]}.get(fmt, list(range(-7, 8)))
    # the element of row 3 farthest (relative to the scale) from every threshold: any other level is wrong
    k = int(np.argmin(np.abs(w[3] / float(s[3]) - np.round(w[3] / float(s[3])))))
    bad = L.copy()
    i = lv.index(int(L[3, k]))
    bad[3, k] = lv[i + 1] if i + 1 < len(lv) else lv[i - 1]
    with pytest.raises(AssertionError, match="row 3"):
        check_rows(fmt, W, 256, bad, s)


@pytest.mark.parametrize("fmt", FMTS)
def test_planted_scale_is_rejected(fmt):
    W = synth.weights_fp32(97, 2, "q", 8, 256)
    L, s = _oracle(W, 256, fmt)
    for step in (1, 2):
        bad = s.copy()
        bad[5] = np.uint16(int(s[5].view(np.uint16)) + step).view(np.float16)
        with pytest.raises(AssertionError, match="row 5"):
            check_rows(fmt, W, 256, L, bad)


def _one(c, p=5):
    r = np.zeros(64, np.float32)
    r[p] = c
    return r


def _two(a, d):
    r = np.zeros(64, np.float32)
    r[3], r[9] = a, d
    return r


@pytest.mark.parametrize("fmt,row,flips", [
    # MNZ: one nonzero 16 rotates to +-2 everywhere, RMS 2, s = 1: w/s = +-2 sits on the threshold
    (levels.FMT_W2_MNZ, _one(16.0), {1: 3, -1: -3}),
    # W4: (38, 18) rotates to +-7 and +-2.5 with s = 1: 2.5 is a rounding tie (to 2; 3 across it)
    (levels.FMT_W4_SYM, _two(38.0, 18.0), {2: 3, -2: -3}),
])
def test_other_side_of_an_exact_threshold_is_accepted(fmt, row, flips):
    W = row[None, :]
    L, s = _oracle(W, 64, fmt)
    w = hadamard.rotate_weights(W.astype(np.float64), 64)[0]
    d = rotation_bound(W, 64)[0]
    moved = np.array([flips.get(int(v), int(v)) for v in L[0]])
    assert np.any(moved != L[0])
    assert row_valid(fmt, w, d, s[0], moved) is None
    # two steps away is not
    far = np.array([int(v) + (2 if int(v) in flips and flips[int(v)] > int(v) else 0) for v in L[0]])
    if fmt == levels.FMT_W4_SYM:
        assert row_valid(fmt, w, d, s[0], far) is not None


# ----------------------------------------------------------------------------- mirror family G(r)

from wquant_rule import MIRROR   # noqa: E402

RATIOS = [0.3, 1.0 / 3.0, 0.5]


def _oracle_mirror(W, b, r):
    return quant.quantize_mirror_mse(hadamard.rotate_weights(np.asarray(W, np.float64), b), r)


@pytest.mark.parametrize("r", RATIOS)
def test_mirror_oracle_result_passes(r):
    W = synth.weights_fp32(98, 0, "q", 16, 512)
    C, s = _oracle_mirror(W, 256, r)
    _, _, differ = check_rows(MIRROR, W, 256, C, s, r)
    assert differ.size == 0


@pytest.mark.parametrize("r", RATIOS)
def test_mirror_planted_code_and_scale_are_rejected(r):
    W = synth.weights_fp32(98, 1, "q", 8, 256)
    C, s = _oracle_mirror(W, 256, r)
    w = hadamard.rotate_weights(W.astype(np.float64), 256)
    # the element of row 2 farthest from both thresholds (0 and (1 + r) / 2) in units of the scale
    u = np.abs(w[2] / float(s[2]))
    k = int(np.argmax(np.minimum(u, np.abs(u - 0.5 * (r + 1.0)))))
    bad = C.copy()
    bad[2, k] = C[2, k] + 1 if C[2, k] < 3 else C[2, k] - 1
    with pytest.raises(AssertionError, match="row 2"):
        check_rows(MIRROR, W, 256, bad, s, r)
    # a code two steps away (across zero) where the row is not near zero
    bad = C.copy()
    bad[2, k] = (C[2, k] + 2) % 4
    with pytest.raises(AssertionError, match="row 2"):
        check_rows(MIRROR, W, 256, bad, s, r)
    for step in (1, 2):
        bs = s.copy()
        bs[4] = np.uint16(int(s[4].view(np.uint16)) + step).view(np.float16)
        with pytest.raises(AssertionError, match="row 4"):
            check_rows(MIRROR, W, 256, C, bs, r)


def test_mirror_quarter_is_accepted_from_the_pot_result():
    # at r = 1/4 the PoT levels as codes, with 4 times the PoT scale, are the mirror result
    W = synth.weights_fp32(98, 2, "q", 12, 256)
    L, s = _oracle(W, 256, levels.FMT_W2_POT)
    codes = np.searchsorted(np.array([-4, -1, 1, 4]), L).astype(np.int8)
    _, _, differ = check_rows(MIRROR, W, 256, codes, (4.0 * s.astype(np.float64)).astype(np.float16), 0.25)
    assert differ.size == 0
