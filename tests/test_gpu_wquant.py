"""GPU weight quantizer (qift_quantize_weights) against the oracle, through the C ABI.

The oracle rotates with a dense fp64 product, then applies quant.quantize_weights.  The rotation of
an fp32 row is not exact, so the two sides can differ in the last bits of a rotated value, and a
decision taken on such bits (a value within rounding of a level threshold, an unrounded scale within
rounding of an fp16 midpoint, two PoT candidates within rounding of each other) may go either way.
Every result is therefore checked with the validity rule of tests/wquant_rule.py: equal to the
oracle's, or different only where the oracle's values lie within the rotation-error bound of the
deciding threshold.  10^4 Student-t rows per format, and rows built to sit on thresholds with
perturbations below fp64 rounding (where the two sides' sums may round differently), go through it.
Rows built to rotate exactly put scales on fp16 rounding ties and values on level thresholds, where
both sides decide on identical numbers and must agree bit for bit.
"""
import numpy as np
import pytest
import torch

from oracle import hadamard, levels, quant
from paper_2606_02823_amd import synth
from wquant_rule import check_rows

pytestmark = pytest.mark.gpu

FMTS = [levels.FMT_W2_MNZ, levels.FMT_W2_POT, levels.FMT_W4_SYM]


@pytest.fixture(scope="module")
def Q():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_02823_amd import qift
    qift.lib()
    return qift


def run_gpu(Q, W, b, fmt):
    L, s = Q.quantize_weights(torch.from_numpy(np.ascontiguousarray(W, dtype=np.float32)).cuda(), b, fmt)
    torch.cuda.synchronize()
    return L.cpu().numpy(), s.cpu().numpy()


def check(Q, W, b, fmt, exact=False):
    """GPU result against the oracle: bit for bit where the rotation is exact, else by the rule."""
    W = np.asarray(W, dtype=np.float32)
    L, s = run_gpu(Q, W, b, fmt)
    if exact:
        L_ref, s_ref = quant.quantize_weights(hadamard.rotate_weights(W.astype(np.float64), b), fmt)
        assert np.array_equal(s.view(np.uint16), s_ref.view(np.uint16)), "scales"
        assert np.array_equal(L, L_ref), "levels"
    else:
        _, _, differ = check_rows(fmt, W, b, L, s)
        print(f"fmt {fmt}: {W.shape[0]} rows, {differ.size} differ from the oracle within the rule", flush=True)
    return L, s


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("N,K,b", [(48, 256, 256), (33, 4096, 4096), (20, 11008, 64), (12, 14336, 2048),
                                   (9, 16384, 4096), (5, 64, 64), (17, 1088, 64), (7, 8192, 128)])
def test_quantize_weights_seeded(Q, fmt, N, K, b):
    # Student-t(5) * 0.02 rows as in the configs; every tile count, ragged tiles, a run-time block
    W = synth.weights_fp32(95, K, "q", N, K)
    L, s = check(Q, W, b, fmt)
    allowed = {levels.FMT_W2_MNZ: {-3, -1, 1, 3}, levels.FMT_W2_POT: {-4, -1, 1, 4}}.get(fmt, set(range(-7, 8)))
    assert set(np.unique(L).tolist()) <= allowed


@pytest.mark.parametrize("fmt", FMTS)
def test_quantize_weights_exact_rows(Q, fmt):
    # K = b = 64 (sqrt(b) = 8): one nonzero c at p rotates to +-c/8 in every column, two nonzeros
    # a, d to +-(a + d)/8 and +-(a - d)/8, all exact
    def one(c, p=5):
        r = np.zeros(64)
        r[p] = c
        return r

    def two(a, d):
        r = np.zeros(64)
        r[3], r[9] = a, d
        return r

    rows = [np.zeros(64),
            one(16 * (1 + 2 ** -11)),       # MNZ s/2 = 1 + 2^-11: a tie, to the even 1.0
            one(16 * (1 + 3 * 2 ** -11)),   # a tie, up to 1 + 2^-9; |w| / s_w just above 2
            one(-16 * (1 + 2 ** -11)),
            one(56 * (1 + 2 ** -11)),       # W4 max/7 = 1 + 2^-11: a tie
            one(3.0), one(1e-3),
            one(5e-7),                      # scales in the fp16 subnormal range
            two(38, 18), two(42, 14), two(-38, 18),   # W4: 7 and +-2.5 (to 2), 7 and 3.5 (to 4)
            two(16, 16), two(24, 8)]        # a zero and an exact midpoint after rotation
    check(Q, np.array(rows), 64, fmt, exact=True)


def test_quantize_weights_then_pack(Q):
    # the quantizer's outputs are the packer's inputs: packed words equal the oracle's packing
    from oracle import pack as opack
    W = synth.weights_fp32(96, 0, "gate", 40, 4096)
    for fmt in FMTS:
        Lg, sg = Q.quantize_weights(torch.from_numpy(W).cuda(), 4096, fmt)
        pk = Q.pack_w4(Lg, sg) if fmt == levels.FMT_W4_SYM else Q.pack_w2(Lg, sg, fmt)
        torch.cuda.synchronize()
        L_ref, _ = quant.quantize_weights(hadamard.rotate_weights(W.astype(np.float64), 4096), fmt)
        assert np.array_equal(pk.words.cpu().numpy().view(np.uint32), opack.pack(L_ref, fmt))


@pytest.mark.parametrize("fmt", FMTS)
def test_quantize_weights_rule_ten_thousand_rows(Q, fmt):
    W = synth.weights_fp32(98, 0, "gate", 10000, 4096)
    check(Q, W, 4096, fmt)


@pytest.mark.parametrize("fmt", FMTS)
def test_quantize_weights_rule_near_thresholds(Q, fmt):
    # K = b = 64: rows whose large entries rotate exactly onto level thresholds, rounding ties and
    # PoT candidate boundaries, plus entries 2^-47 .. 2^-58 times as large in the other positions,
    # which move the exact rotated values off those points by less than fp64 rounding, so that
    # the two sides' sums (dense product, butterflies) may round to either side
    rng = np.random.default_rng(99 + fmt)
    bases = []
    for a, dd in ((38, 18), (42, 14), (-38, 18), (16, 16), (24, 8), (20, 0), (16, 0), (40, 16), (36, 20)):
        r = np.zeros(64)
        r[3], r[9] = a, dd
        bases.append(r)
    rows = []
    for base in bases:
        for _ in range(40):
            r = base.copy()
            free = np.setdiff1d(np.arange(64), [3, 9])
            pos = rng.choice(free, size=int(rng.integers(1, 20)), replace=False)
            r[pos] = rng.choice([-1.0, 1.0], pos.size) * 40.0 * 2.0 ** -rng.integers(47, 59, pos.size)
            rows.append(r)
    check(Q, np.array(rows, dtype=np.float32), 64, fmt)
