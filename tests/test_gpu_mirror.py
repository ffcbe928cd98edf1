"""GPU mirror-family quantizer (qift_quantize_weights_mirror, G(r) = {-1, -r, +r, +1} of Sec. 3.4
Eq. (18)) and the ratio scan (qift_ratio_scan, Sec. 4.5.3) against the oracle, through the C ABI.

* The quantizer rotates fp32 rows in fp64 like the PoT quantizer, so its results are checked with the
  validity rule of tests/wquant_rule.py (the oracle's result, or a different one only within the
  rotation-error bound of the deciding threshold); rows built to rotate exactly must agree bit for
  bit.  At r = 1/4 its codes and scales are the PoT quantizer's levels and 4 x scales, bit for bit.
  Its codes, packed with the level-table format, drive the level-table linear with the table
  {-1, -r, +r, +1}: y bit-exact against the oracle's table linear.
* The scan forms every term with the same rounded fp64 operations as the oracle; only the order of
  the n-term sums differs, so sse, nmse and the statistics agree within 2 n ulps of the sums, and the
  chosen candidate's oracle error lies within that bound of the oracle's minimum.
"""
import numpy as np
import pytest
import torch

from oracle import hadamard, levels, linear as olin, lut as olut, pack as opack, quant
from paper_2606_02823_amd import synth
from wquant_rule import MIRROR, check_rows

pytestmark = pytest.mark.gpu

U = 2.0 ** -53
RATIOS = [0.2526, 0.3, 1.0 / 3.0, 0.5, 0.9]


@pytest.fixture(scope="module")
def Q():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_02823_amd import qift
    qift.lib()
    return qift


def run_mirror(Q, W, b, r):
    C, s = Q.quantize_weights_mirror(torch.from_numpy(np.ascontiguousarray(W, dtype=np.float32)).cuda(), b, r)
    torch.cuda.synchronize()
    return C.cpu().numpy(), s.cpu().numpy()


@pytest.mark.parametrize("r", RATIOS)
@pytest.mark.parametrize("N,K,b", [(40, 256, 256), (24, 4096, 4096), (12, 11008, 64), (8, 14336, 2048),
                                   (5, 16384, 4096), (17, 1088, 64)])
def test_mirror_quantizer_seeded(Q, r, N, K, b):
    W = synth.weights_fp32(101, K, "q", N, K)
    print(f"mirror r={r} N={N} K={K} b={b}", flush=True)
    C, s = run_mirror(Q, W, b, r)
    _, _, differ = check_rows(MIRROR, W, b, C, s, r)
    print(f"  {differ.size} rows differ within the rule", flush=True)
    assert set(np.unique(C).tolist()) <= {0, 1, 2, 3}


@pytest.mark.parametrize("r", [0.3, 0.5])
def test_mirror_quantizer_rule_many_rows(Q, r):
    W = synth.weights_fp32(102, 0, "gate", 4000, 4096)
    C, s = run_mirror(Q, W, 4096, r)
    _, _, differ = check_rows(MIRROR, W, 4096, C, s, r)
    print(f"mirror r={r}: 4000 rows, {differ.size} differ within the rule", flush=True)


def test_mirror_quantizer_exact_rows(Q):
    # K = b = 64: rows of one or two nonzeros rotate exactly (sqrt(64) = 8), a zero row, tiny rows
    rows = []
    for a, d in ((16, 0), (38, 18), (42, 14), (-38, 18), (16, 16), (24, 8), (3, 1), (1e-3, 0), (5e-7, 0)):
        r_ = np.zeros(64)
        r_[3], r_[9] = a, d
        rows.append(r_)
    rows.append(np.zeros(64))
    W = np.array(rows, dtype=np.float32)
    w = hadamard.rotate_weights(W.astype(np.float64), 64)
    for r in (0.25, 0.3, 0.5, 0.75):
        C, s = run_mirror(Q, W, 64, r)
        C_ref, s_ref = quant.quantize_mirror_mse(w, r)
        assert np.array_equal(s.view(np.uint16), s_ref.view(np.uint16)), f"scales r={r}"
        assert np.array_equal(C, C_ref), f"codes r={r}"
        assert np.all(C[-1] == 2) and s[-1] == 0


def test_mirror_quarter_is_the_pot_quantizer(Q):
    # the same rotated values and the same candidate errors up to the exact factor 4
    W = synth.weights_fp32(103, 0, "o", 64, 4096)
    C, s = run_mirror(Q, W, 4096, 0.25)
    L, sp = Q.quantize_weights(torch.from_numpy(W).cuda(), 4096, levels.FMT_W2_POT)
    L, sp = L.cpu().numpy(), sp.cpu().numpy()
    assert np.array_equal(np.array([-4, -1, 1, 4])[C], L)
    assert np.array_equal(s.astype(np.float64), 4.0 * sp.astype(np.float64))


@pytest.mark.parametrize("r", [0.3, 0.5])
def test_mirror_codes_through_the_table_linear(Q, r):
    # quantize -> pack (level-table format) -> rotate_quant_act -> table linear, y against the oracle
    N, K, b, M = 96, 4096, 4096, 5
    W = synth.weights_fp32(104, 0, "up", N, K)
    Cg, sg = Q.quantize_weights_mirror(torch.from_numpy(W).cuda(), b, r)
    pk = Q.pack_w2(Cg, sg, Q.W2_LUT)
    grid = (-1.0, -r, r, 1.0)
    x = synth.activations_fp16(104, 0, 0, M, K, 5, 20.0)
    act = Q.rotate_quant_act(torch.from_numpy(x).cuda(), b)
    y = Q.w2a4_lut_linear(pk, grid, act)
    torch.cuda.synchronize()
    C, s = Cg.cpu().numpy(), sg.cpu().numpy()
    check_rows(MIRROR, W, b, C, s, r)
    P = opack.pack_qw2(C, levels.FMT_W2_LUT)
    assert np.array_equal(pk.words.cpu().numpy().view(np.uint32), P)
    y32, yref, _ = olut.lut_linear(P, olut.table(grid), s, K, act.q.cpu().numpy(), act.scale.cpu().numpy())
    got = y.cpu().numpy()
    assert np.array_equal(got.view(np.uint16), y32.view(np.uint16))
    assert olin.max_abs_rel(got, yref) <= olin.TOL_REL


# ----------------------------------------------------------------------------- ratio scan

def _scan_check(Q, x, ratios, cands):
    sse, nmse, best, stats = Q.ratio_scan(torch.from_numpy(x).cuda(), ratios, cands)
    torch.cuda.synchronize()
    sse, nmse, best, stats = sse.cpu().numpy(), nmse.cpu().numpy(), best.cpu().numpy(), stats.cpu().numpy()
    sse_ref, nmse_ref, best_ref, (a, sx2) = quant.ratio_scan(x, ratios, cands)
    n = x.size
    assert stats[0] == a                                       # a maximum is exact
    assert abs(stats[1] - sx2) <= 2.0 * n * U * sx2
    tol = 2.0 * n * U * sse_ref + 1e-300
    assert np.all(np.abs(sse - sse_ref) <= tol), "sse"
    rows = np.arange(len(ratios))
    # the chosen candidate is a minimiser within the summation bound
    assert np.all(sse_ref[rows, best] - sse_ref[rows, best_ref] <= tol[rows, best] + tol[rows, best_ref])
    same = best == best_ref
    if sx2 > 0:
        assert np.all(np.abs(nmse[same] - nmse_ref[same]) <= 4.0 * n * U * nmse_ref[same] + 1e-300)
    else:
        assert np.all(nmse == 0) and np.all(sse == 0)
    return nmse, best


def test_ratio_scan_gaussian(Q):
    x = np.random.default_rng(31).standard_normal(1 << 17)
    ratios = [0.25, 0.2526, 0.2998, 1.0 / 3.0, 0.5]
    cands = np.linspace(0.15, 0.65, 201)
    nmse, best = _scan_check(Q, x, ratios, cands)
    assert np.all((best > 0) & (best < len(cands) - 1))
    assert int(np.argmin(nmse)) == 2                        # the Lloyd-Max ratio is the best of these


def test_ratio_scan_many_ratios_and_weights(Q):
    # pooled rotated Student-t weights (the study's input), 81 ratios (three launches of the table), the
    # 64 PoT candidates, and a ragged sample count
    W = synth.weights_fp32(105, 0, "gate", 24, 4096)
    x = hadamard.rotate_weights(W.astype(np.float64), 4096).ravel()[: 24 * 4096 - 37]
    ratios = np.linspace(0.1, 0.9, 81)
    _scan_check(Q, np.ascontiguousarray(x), ratios, quant.POT_CANDIDATES)


def test_ratio_scan_edges(Q):
    # one sample; all-zero samples (no error); exact ties on the threshold; extreme magnitudes
    _scan_check(Q, np.array([0.7]), [0.5], [0.2, 1.0, 0.7])
    _scan_check(Q, np.zeros(1000), [0.3, 0.6], [0.5, 1.0])
    x = np.array([1.0, -1.0, 0.75, -0.75, 0.5, 0.0, -0.0, 0.25] * 33)
    _scan_check(Q, x, [0.5, 0.25], [1.0, 0.5, 0.25])
    rng = np.random.default_rng(32)
    _scan_check(Q, rng.standard_normal(5000) * 1e-300, [0.3], np.linspace(0.2, 1.0, 64))
    _scan_check(Q, rng.standard_normal(5000) * 1e150, [0.3], np.linspace(0.2, 1.0, 256))
