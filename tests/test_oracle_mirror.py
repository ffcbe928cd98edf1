"""Pins of the mirror-family weight quantizer (oracle.quant.quantize_mirror_mse, Sec. 3.4 Eq. (18)) and
of the ratio-scan diagnostic (oracle.quant.ratio_scan, Sec. 4.5.3): at r = 1/4 the mirror quantizer is
the PoT quantizer (levels +-1, +-4 at scale s are +-1/4, +-1 at scale 4 s, an exact power-of-two
rescaling of every candidate, quotient and error); the scan reproduces the paper's ratio table
(tests/golden/ratio_table.json) on Gaussian samples and puts its optimum inside the effective band."""
import json
import os

import numpy as np
import pytest

from oracle import levels, quant


def test_quarter_ratio_is_the_pot_quantizer():
    rows = np.random.default_rng(21).standard_normal((12, 1024)) * 0.02
    rows[3] = 0.0
    c, s = quant.quantize_mirror_mse(rows, 0.25)
    L, sp = quant.quantize_pot_mse(rows)
    assert np.array_equal(np.array([-4, -1, 1, 4])[c], L)
    assert np.array_equal(s.astype(np.float64), 4.0 * sp.astype(np.float64))
    assert np.all(c[3] == 2) and s[3] == 0


def test_mirror_levels_by_hand():
    # one row [4, 2.6, 2.4, -1, 0]: the candidate grid gives some s; then against s_w the codes follow
    # the midpoint (1 + r) / 2 of u = w / s_w exactly (ties to the inner level, zero positive)
    r = 0.5
    w = np.array([[4.0, 3.0, 2.9, -3.0, -2.0, 0.0, 1.0, -0.5]])
    c, s = quant.quantize_mirror_mse(w, r)
    u = w[0] / float(s[0])
    expect = [3 if v > 0.75 else 2 if v >= 0 else 0 if v < -0.75 else 1 for v in u]
    assert c[0].tolist() == expect
    # the scale is the fp16 of one of the 64 candidates c * max|w|
    assert np.any(np.float16(quant.POT_CANDIDATES * 4.0) == s[0])


def _table():
    with open(os.path.join(os.path.dirname(__file__), "golden", "ratio_table.json")) as f:
        return json.load(f)


def test_ratio_scan_reproduces_the_paper_table():
    rows = _table()["rows"]
    x = np.random.default_rng(22).standard_normal(1 << 17)
    cands = np.linspace(0.15, 0.65, 201)
    ratios = [rows["MNZ"]["r"], rows["POT"]["r"], rows["FAR_MNZ"]["r"]]
    _, nmse, best, _ = quant.ratio_scan(x, ratios, cands)
    for name, v in zip(("MNZ", "POT", "FAR_MNZ"), nmse):
        assert v == pytest.approx(rows[name]["nmse"], rel=8e-3), name
    assert np.all((best > 0) & (best < len(cands) - 1))   # the optimum lies inside the candidate range


def test_ratio_scan_optimum_in_the_effective_band():
    g = _table()
    x = np.random.default_rng(23).standard_normal(1 << 16)
    rs = np.arange(0.15, 0.55 + 1e-9, 0.02)
    _, nmse, _, _ = quant.ratio_scan(x, rs, np.linspace(0.15, 0.65, 101))
    lo, hi = g["effective_band"]
    assert lo - 0.02 <= rs[int(np.argmin(nmse))] <= hi + 0.02
    assert nmse.min() == pytest.approx(g["scan_optimum"]["nmse"], rel=1.5e-2)
