"""GPU level-table linear (qift_w2a4_lut_linear: the reference grids of Sec. 3.3 through an fp16
table) against the oracle, through the C ABI.  Bit-exact: the packed code words, and y against the
oracle's exact t with the fp32 epilogue; within the 1e-3 criterion of the fp64 epilogue."""
import numpy as np
import pytest
import torch

from oracle import levels, linear as olin, lut as olut, pack as opack
from paper_2606_02823_amd import synth

pytestmark = pytest.mark.gpu

ADVERSARIAL = (-256.0, -(2.0 ** -24), 2.0 ** -14, 255.875)


@pytest.fixture(scope="module")
def Q():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_02823_amd import qift
    qift.lib()
    return qift


def _case(Q, M, N, K, grid, seed):
    rng = np.random.default_rng(seed)
    codes = rng.integers(0, 4, (N, K)).astype(np.int8)
    codes[0] = 3                                           # a row at the top level
    if N > 1:
        codes[1] = 0
    s_w = rng.uniform(0.005, 0.05, N).astype(np.float16)
    b = 4096 if K % 4096 == 0 else 256
    x = synth.activations_fp16(seed, 0, 0, M, K, 5, 20.0)
    act = Q.rotate_quant_act(torch.from_numpy(x).cuda(), b)
    pk = Q.pack_w2(torch.from_numpy(codes).cuda(), torch.from_numpy(s_w.view(np.int16)).cuda().view(torch.float16),
                   Q.W2_LUT)
    y = Q.w2a4_lut_linear(pk, grid, act)
    torch.cuda.synchronize()
    P = opack.pack_qw2(codes, levels.FMT_W2_LUT)
    assert np.array_equal(pk.words.cpu().numpy().view(np.uint32), P)
    q, s_x = act.q.cpu().numpy(), act.scale.cpu().numpy()
    y32, yref, _ = olut.lut_linear(P, olut.table(grid), s_w, K, q, s_x)
    got = y.cpu().numpy()
    assert np.array_equal(got.view(np.uint16), y32.view(np.uint16))
    assert olin.max_abs_rel(got, yref) <= olin.TOL_REL
    return pk, act, got


@pytest.mark.parametrize("grid", [levels.LLOYD, levels.NF2, ADVERSARIAL], ids=["lloyd", "nf2", "adversarial"])
@pytest.mark.parametrize("M,N,K", [(1, 4096, 4096), (3, 1000, 512), (17, 300, 11008), (64, 64, 14336),
                                   (1, 22016, 4096), (100, 48, 1024)])
def test_lut_linear(Q, M, N, K, grid):
    _case(Q, M, N, K, grid, seed=M * 1009 + N + K)


def test_mnz_table_equals_integer_linear(Q):
    """The MNZ levels at half scale as the table give the integer linear's result bit for bit."""
    M, N, K = 4, 256, 4096
    pk, act, got = _case(Q, M, N, K, levels.MNZ_HALF, seed=7)
    rng = np.random.default_rng(7)
    codes = rng.integers(0, 4, (N, K)).astype(np.int8)
    codes[0], codes[1] = 3, 0
    L = np.asarray(levels.MNZ_HALF, dtype=np.int8)[codes]
    pk2 = Q.pack_w2(torch.from_numpy(L).cuda(), pk.scales, Q.W2_MNZ)
    y2 = Q.w2a4_linear(pk2, act)
    assert np.array_equal(y2.cpu().numpy().view(np.uint16), got.view(np.uint16))
