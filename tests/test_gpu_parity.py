"""GPU parity: libqift's HIP path against the CPU oracle, through the C ABI.

Bit-exact: packed words, act_q, act_sum, act_scale, int32 accumulators and
the fp16 output against the oracle's fp32 epilogue expression; within the
max-abs-rel 1e-3 criterion against the oracle's fp64 epilogue.  Inputs come
from the seeded generators; expected values only from ``oracle``.  The
linears run with the per-token code sums computed in the kernels (the
boundary's call takes none) unless a test passes the quantizer's sums.
"""
import numpy as np
import pytest
import torch

from oracle import hadamard, levels, linear as olin, pack as opack, quant
from paper_2606_02823_amd import synth

pytestmark = pytest.mark.gpu

FMTS = [levels.FMT_W2_MNZ, levels.FMT_W2_POT, levels.FMT_W4_SYM]


@pytest.fixture(scope="module")
def Q():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_02823_amd import qift
    qift.lib()
    return qift


def dev(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint32:
        a = a.view(np.int32)
    return torch.from_numpy(a).cuda()


def host(t):
    return t.cpu().numpy()


def bits16(a):
    return np.ascontiguousarray(a).view(np.uint16)


def pack_dev(Q, L, s_w, fmt):
    if fmt == levels.FMT_W4_SYM:
        return Q.pack_w4(dev(L), dev(s_w))
    return Q.pack_w2(dev(L), dev(s_w), fmt)


def check_act(act, x, b, clip=(1, 1), tokens=None):
    q_ref, sx_ref, sum_ref, _ = quant.act_quant(x if tokens is None else x[tokens], b, clip)
    q, sx, sm = host(act.q), host(act.scale), host(act.sum)
    if tokens is not None:
        q, sx, sm = q[tokens], sx[tokens], sm[tokens]
    assert np.array_equal(q, q_ref)
    assert np.array_equal(sx.view(np.uint32), sx_ref.view(np.uint32))
    assert np.array_equal(sm, sum_ref)
    return q_ref, sx_ref


def check_linear(y, acc, L, q_ref, sx_ref, s_w, rows=None, tokens=None):
    y, acc = host(y), host(acc)
    if rows is not None:
        y, acc, L, s_w = y[:, rows], acc[:, rows], L[rows], s_w[rows]
    if tokens is not None:
        y, acc = y[tokens], acc[tokens]
    acc_ref = olin.int_dot(L, q_ref)
    assert np.array_equal(acc, acc_ref)
    assert np.array_equal(bits16(y), bits16(olin.epilogue_fp32(acc_ref, sx_ref, s_w)))
    assert olin.max_abs_rel(y, olin.epilogue_ref(acc_ref, sx_ref, s_w)) <= olin.TOL_REL


def run_linear(Q, pk, act, M, N, use_sum=False, workspace=None):
    acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
    y = Q.linear(pk, act, acc_out=acc, use_sum=use_sum, workspace=workspace)
    torch.cuda.synchronize()
    return y, acc


# ----------------------------------------------------------------------------- config 0


@pytest.mark.parametrize("fmt", FMTS)
def test_cfg0_pipeline(Q, fmt):
    c = synth.CONFIGS[0]
    shp = c.linears[0]
    N, K, b, M = shp.N, shp.K, shp.block, c.Ms[0]
    W = synth.weights_fp32(0, 0, "lin", N, K)
    L, s_w = quant.quantize_weights(hadamard.rotate_weights(W, b), fmt)
    pk = pack_dev(Q, L, s_w, fmt)
    assert np.array_equal(host(pk.words).view(np.uint32), opack.pack(L, fmt))
    x = synth.config_activations(c, 0, 0, M, K)
    act = Q.rotate_quant_act(dev(x), b)
    q_ref, sx_ref = check_act(act, x, b)
    y, acc = run_linear(Q, pk, act, M, N)
    check_linear(y, acc, L, q_ref, sx_ref, s_w)
    # the plain entry (no accumulator output) gives the same y
    y2 = Q.linear(pk, act)
    torch.cuda.synchronize()
    assert torch.equal(y2, y)


# ----------------------------------------------------------------------------- ragged tiles


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("M", [1, 5, 16, 17, 32, 47, 64, 65, 130])
def test_linear_ragged(Q, fmt, M):
    # N not a multiple of 16, K spanning a partial 1024-chunk, every token-tile count
    N, K, b = 1000, 1088, 64
    L = synth.draw_levels(fmt, N, K, cfg=90, layer=M)
    s_w = synth.draw_scales(fmt, N, cfg=90, layer=M)
    x = synth.activations_fp16(90, M, 0, M, K, 11, 30.0)
    pk = pack_dev(Q, L, s_w, fmt)
    assert np.array_equal(host(pk.words).view(np.uint32), opack.pack(L, fmt))
    act = Q.rotate_quant_act(dev(x), b)
    q_ref, sx_ref = check_act(act, x, b)
    y, acc = run_linear(Q, pk, act, M, N)
    check_linear(y, acc, L, q_ref, sx_ref, s_w)
    # the quantizer's sums passed in (qift_*_linear_ex) give the same results
    y2, acc2 = run_linear(Q, pk, act, M, N, use_sum=True)
    assert torch.equal(acc2, acc) and torch.equal(y2.view(torch.int16), y.view(torch.int16))
    # and so does the boundary's call without accumulators or sums
    y3 = Q.linear(pk, act)
    torch.cuda.synchronize()
    assert torch.equal(y3.view(torch.int16), y.view(torch.int16))


@pytest.mark.parametrize("fmt", [levels.FMT_W2_MNZ, levels.FMT_W2_POT])
@pytest.mark.parametrize("M,N,K", [(65, 1000, 1088), (130, 1000, 1088), (300, 1000, 4096), (200, 1000, 14336),
                                   (96, 1000, 4160), (320, 16400, 2048)])
def test_w2_prefill_int8_and_fp4_paths(Q, fmt, M, N, K):
    # W2 (MNZ, PoT) at M > 64, ragged rows and tokens, K with a partial last step; bit-identical to the
    # oracle on every path:
    #   no workspace: the int8 GEMM;
    #   a workspace of workspace_bytes where the 256 x 64 tiles are few: the int8 GEMM split over K
    #   (S = min(ceil(512 / tiles), 512 // tiles, steps // 4) >= 2 ranges of 256-k steps; K = 4160 has
    #   17 steps: ranges of 5, 5, 5 and 2, the last one ending in a partial step);
    #   otherwise the FP4 x FP6 GEMM (FP6 activations in the workspace; the MNZ codes as c / 2, the PoT
    #   levels +-1, +-4 as E2M1 values), itself split over K where S = min(ceil(512 / tiles),
    #   768 // tiles, steps // 4) >= 2 (16400 x 2048 at 320 tokens: 325 tiles, two ranges).
    b = 64
    L = synth.draw_levels(fmt, N, K, cfg=97, layer=M + fmt)
    s_w = synth.draw_scales(fmt, N, cfg=97, layer=M + fmt)
    x = synth.activations_fp16(97, M, 0, M, K, K // 100, 30.0)
    pk = pack_dev(Q, L, s_w, fmt)
    act = Q.rotate_quant_act(dev(x), b)
    q_ref, sx_ref = check_act(act, x, b)
    KT, tiles, N4 = -(-K // 256), -(-N // 256) * -(-M // 64), -(-N // 4) * 4

    def ranges(S):
        if S < 2:
            return 1
        us = -(-KT // S)
        return -(-KT // us)

    S8 = ranges(min(-(-512 // tiles), 512 // tiles, KT // 4))
    if S8 > 1:
        expect = -(-(S8 * M * N4 * 4) // 256) * 256 + S8 * M * 4
    else:
        expect = M * 3 * (K // 4) + 4 * M * (-(-(K // 32) // 256))
        S4 = ranges(min(-(-512 // tiles), 768 // tiles, KT // 4))
        if S4 > 1:
            expect = -(-expect // 256) * 256 + -(-(S4 * M * N4 * 4) // 256) * 256
    assert Q.workspace_bytes(pk, M) == expect
    for ws in (None, torch.empty(Q.workspace_bytes(pk, M), dtype=torch.uint8, device="cuda")):
        for use_sum in (False, True):
            y, acc = run_linear(Q, pk, act, M, N, use_sum=use_sum, workspace=ws)
            check_linear(y, acc, L, q_ref, sx_ref, s_w)


@pytest.mark.parametrize("M,N,K", [(65, 300, 4160), (200, 300, 4160), (128, 1000, 14336), (96, 4096, 1088),
                                   (130, 2064, 8192), (40, 16400, 4160), (64, 16384, 2048), (48, 4096, 14336),
                                   (24, 4096, 14336), (30, 28672, 4096)])
def test_w4_prefill_split_over_k(Q, M, N, K):
    # W4 above 64 tokens with a workspace of workspace_bytes: where the 256 x 64 tiles are few the int8
    # GEMM is split over K (S >= 3 ranges of at least 8 steps of 128 k, about 512 workgroups, at most 512):
    # K = 4160 has 33 steps (ranges of 9, 9, 9 and 6, the last step partial); K = 1088 has 9 steps, too
    # few to split (workspace_bytes 0).  From 24 tokens on a gate|up width (N >= 16384) or a down shape
    # (N >= 4096, K > 4096) takes the same split instead of the skinny kernel.  Bit-identical to the oracle and to the call without a
    # workspace, with and without the quantizer's code sums.
    fmt = levels.FMT_W4_SYM
    L = synth.draw_levels(fmt, N, K, cfg=95, layer=M)
    s_w = synth.draw_scales(fmt, N, cfg=95, layer=M)
    x = synth.activations_fp16(95, M, 0, M, K, 9, 30.0)
    pk = pack_dev(Q, L, s_w, fmt)
    act = Q.rotate_quant_act(dev(x), 64)
    q_ref, sx_ref = check_act(act, x, 64)
    KT, tiles = -(-K // 128), -(-N // 256) * -(-M // 64)
    S = min(-(-512 // tiles), 512 // tiles, KT // 8)
    need = Q.workspace_bytes(pk, M)
    if S >= 3:
        us = -(-KT // S)
        S = -(-KT // us)
        assert need == -(-(S * M * (-(-N // 4) * 4) * 4) // 256) * 256 + S * M * 4
    else:
        assert need == 0
    ws = torch.empty(max(need, 16), dtype=torch.uint8, device="cuda")
    for use_sum in (False, True):
        y, acc = run_linear(Q, pk, act, M, N, use_sum=use_sum, workspace=ws if need else None)
        check_linear(y, acc, L, q_ref, sx_ref, s_w)
        y0, acc0 = run_linear(Q, pk, act, M, N, use_sum=use_sum)
        assert torch.equal(acc, acc0) and torch.equal(y.view(torch.int16), y0.view(torch.int16))


@pytest.mark.parametrize("fmt", [levels.FMT_W2_MNZ, levels.FMT_W2_POT])
@pytest.mark.parametrize("M,N,K", [(17, 1000, 1088), (32, 1000, 14336), (33, 4096, 4096), (64, 1000, 14336),
                                   (64, 4096, 14336), (20, 2064, 8192), (40, 300, 16384), (64, 6144, 4096),
                                   (47, 28672, 4096), (16, 1000, 14336), (13, 4096, 14336), (16, 1000, 4096),
                                   (32, 28672, 4096), (40, 16400, 4160)])
def test_skinny_split_over_k(Q, fmt, M, N, K):
    # 17..64 tokens with a workspace of workspace_bytes, and up to 16 where the decode kernel's LDS does
    # not hold the codes (16 or 13 tokens of 14336): a linear with K > 4096 and few 16-row tiles runs
    # split over K (int32 partial sums of each K-range in the workspace, then added and the epilogue
    # applied); K <= 4096 needs no split (workspace_bytes 0).  From 33 tokens on a gate|up width (N >=
    # 16384) or a down shape (N >= 4096, K > 4096) takes the prefill GEMM split over K instead (S = min(ceil(512 / tiles), 512 // tiles,
    # steps // 4) ranges of 256-k steps over 256 x 64 tiles).  Bit-identical to the oracle and to the call
    # without a workspace, with and without the quantizer's code sums.
    b = 4096 if K % 4096 == 0 else (2048 if K % 2048 == 0 else 64)
    L = synth.draw_levels(fmt, N, K, cfg=98, layer=M + fmt)
    s_w = synth.draw_scales(fmt, N, cfg=98, layer=M + fmt)
    x = synth.activations_fp16(98, M, 0, M, K, max(1, K // 100), 30.0)
    pk = pack_dev(Q, L, s_w, fmt)
    act = Q.rotate_quant_act(dev(x), b)
    q_ref, sx_ref = check_act(act, x, b)
    need = Q.workspace_bytes(pk, M)
    if M >= 33 and (N >= 16384 or (N >= 4096 and K > 4096)):
        tiles, KT = -(-N // 256), -(-K // 256)
        S = min(-(-512 // tiles), 512 // tiles, KT // 4)
        S = -(-KT // -(-KT // S))
        assert need == -(-(S * M * (-(-N // 4) * 4) * 4) // 256) * 256 + S * M * 4
    else:
        # the skinny split rule: K > 4096, 4 tiles per workgroup, S = 256 / workgroups rounded, from S = 2
        gx = -(-(-(-N // 16)) // 4)
        assert (need > 0) == (K > 4096 and (256 + gx // 2) // gx >= 2)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda") if need else None
    y0, acc0 = run_linear(Q, pk, act, M, N)
    check_linear(y0, acc0, L, q_ref, sx_ref, s_w)
    for use_sum in (False, True):
        y, acc = run_linear(Q, pk, act, M, N, use_sum=use_sum, workspace=ws)
        assert torch.equal(acc, acc0) and torch.equal(y.view(torch.int16), y0.view(torch.int16))


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("M,K", [(1, 20480), (9, 20480), (16, 32768)])
def test_linear_long_k(Q, fmt, M, K):
    # K beyond the decode-on-codes kernel's limit: codes staged in LDS (M = 1) or read from HBM
    N, b = 300, 4096
    L = synth.draw_levels(fmt, N, K, cfg=91, layer=M)
    s_w = synth.draw_scales(fmt, N, cfg=91, layer=M)
    x = synth.activations_fp16(91, M, 0, M, K, K // 100, 30.0)
    pk = pack_dev(Q, L, s_w, fmt)
    act = Q.rotate_quant_act(dev(x), b)
    q_ref, sx_ref = check_act(act, x, b)
    y, acc = run_linear(Q, pk, act, M, N)
    check_linear(y, acc, L, q_ref, sx_ref, s_w)


@pytest.mark.parametrize("fmt", FMTS)
def test_linear_extremes(Q, fmt):
    # all-outer levels against all +-7 activations: the largest |acc| of each format
    N, K, b, M = 48, 14336, 2048, 3
    vals = {levels.FMT_W2_MNZ: (3, -3), levels.FMT_W2_POT: (4, -4), levels.FMT_W4_SYM: (7, -7)}[fmt]
    L = np.empty((N, K), dtype=np.int8)
    L[: N // 2] = vals[0]
    L[N // 2:] = vals[1]
    s_w = np.full(N, 0.5, dtype=np.float16)
    s_w[0] = np.float16(65504.0)          # overflow of the product goes to inf
    s_w[1] = 0                            # a zero scale
    x = np.zeros((M, K), dtype=np.float16)
    x[0, ::b] = 60000.0                   # one spike per block -> every q = +7, y overflows to inf
    x[1] = np.float16(2.0 ** -24)         # smallest subnormals
    x[2] = synth.activations_fp16(94, 0, 0, 1, K, 143, 30.0)[0]
    pk = pack_dev(Q, L, s_w, fmt)
    act = Q.rotate_quant_act(dev(x), b)
    q_ref, sx_ref = check_act(act, x, b)
    y, acc = run_linear(Q, pk, act, M, N)
    check_linear(y, acc, L, q_ref, sx_ref, s_w)


def test_pack_rejects_levels_outside_the_set(Q):
    # the pack calls validate every level and return QIFT_ERR_CODE (status -5)
    L = np.full((16, 64), 1, dtype=np.int8)
    L[3, 7] = 0
    s = np.ones(16, dtype=np.float16)
    for fmt, bad in ((Q.W2_MNZ, 0), (Q.W2_MNZ, 2), (Q.W2_POT, 3), (Q.W2_LUT, 4), (Q.W4_SYM, -8), (Q.W4_SYM, 8)):
        L[3, 7] = bad
        with pytest.raises(Q.QiftError, match="QIFT_ERR_CODE") as e:
            if fmt == Q.W4_SYM:
                Q.pack_w4(dev(L), dev(s))
            else:
                Q.pack_w2(dev(L), dev(s), fmt)
        assert e.value.status == -5
    # a clean call afterwards starts from a zero count
    L[3, 7] = 1
    Q.pack_w2(dev(L), dev(s), Q.W2_MNZ)
    Q.pack_w4(dev(L), dev(s))


# ----------------------------------------------------------------------------- activation quantizer


ACT_CASES = [(64, 2), (128, 4), (256, 8), (512, 16), (256, 32), (1024, 64), (11008, 64), (1024, 128),
             (768, 256), (4096, 512), (2048, 1024), (14336, 2048), (4096, 4096), (12288, 4096),
             (16384, 4096), (20480, 4096), (8192, 8192), (32768, 8192), (24576, 2048)]


@pytest.mark.parametrize("K,b", ACT_CASES)
def test_rotate_quant_act_blocks(Q, K, b):
    M = 4
    x = synth.activations_fp16(91, K // 64, b, M, K, max(1, K // 100), 30.0)
    x[1] = 0                                                # all-zero token
    rng = np.random.default_rng(K + b)
    mags = 10.0 ** rng.uniform(-7.5, 4.8, size=K)           # subnormals .. near fp16 max
    x[2] = (mags * rng.choice([-1, 1], size=K)).astype(np.float16)
    x[2, :2] = [65504.0, -65504.0]
    act = Q.rotate_quant_act(dev(x), b)
    check_act(act, x, b)


@pytest.mark.parametrize("M,K,b", [(1, 14336, 2048), (16, 11008, 64), (256, 14336, 2048), (257, 14336, 2048),
                                   (3, 12288, 4096), (64, 8192, 256)])
def test_rotate_quant_act_tile_parallel(Q, M, K, b):
    # up to 256 tokens of several 4096-tiles the tiles are rotated at once by groups of four waves,
    # one token per workgroup; from 257 tokens on by the persistent kernel: the same codes either way
    x = synth.activations_fp16(93, M, b, M, K, max(1, K // 100), 30.0)
    if M > 2:
        x[1] = 0                                            # all-zero token
    act = Q.rotate_quant_act(dev(x), b)
    check_act(act, x, b)


def test_rotate_quant_act_exact_ties(Q):
    u = 2.0 ** -10
    pairs = [(9.5, 4.5), (10.5, 3.5), (7.5, 6.5), (8.5, 5.5), (4.5, 9.5)]
    x = np.zeros((2, 64), dtype=np.float16)
    for i in range(32):
        a, bb = pairs[i % len(pairs)]
        x[0, 2 * i], x[0, 2 * i + 1] = a * u, bb * u
        x[1, 2 * i], x[1, 2 * i + 1] = -bb * u, -a * u
    act = Q.rotate_quant_act(dev(x), 2)
    q_ref, _ = check_act(act, x, 2)
    assert set(np.abs(q_ref[0, 1::2]).tolist()) == {0, 2, 4}


@pytest.mark.parametrize("clip", [(9, 10), (1, 2), (15, 16)])
def test_rotate_quant_act_clip_ratio(Q, clip):
    K, b = 4096, 4096
    x = synth.activations_fp16(92, 0, 0, 8, K, 41, 30.0)
    act = Q.rotate_quant_act(dev(x), b, clip=clip)
    check_act(act, x, b, clip)


def _bf16_any(rng, M, K, b):
    """bf16 activations across the finite bf16 range (no narrowing): rows of N(0, 1) at scales from
    2^-30 to 2^30 (values below 2^-17 and from 2^16 in magnitude among them), extreme values
    (subnormals, the largest finite magnitude), a row far below 2^-24, a row mixing 2^-120 and 2^100,
    and a block holding only two values, whose transform alternates 7 2^-100 and 2.5 2^-100 (a
    rounding tie off the fp16 grid)."""
    x = rng.normal(0, 1, (M, K)) * 2.0 ** rng.uniform(-30, 30, (M, 1))
    x[0] *= 2.0 ** -60
    if M > 1:
        x[1] = rng.normal(0, 1, K)
        x[1, ::2] *= 2.0 ** -120
        x[1, 1::2] *= 2.0 ** 100
    if M > 2:
        x[2] = 0
        x[2, 0], x[2, 1] = 4.75 * 2.0 ** -100, 2.25 * 2.0 ** -100   # block 0: [7, 2.5, 7, 2.5, ...] 2^-100
    ext = [2.0 ** -133, -(2.0 ** -126), 3.3e38, -(2.0 ** 100), 2.0 ** -17, 65280.0, 65536.0, 1e-30]
    for m in range(3, M):
        x[m, rng.choice(K, size=len(ext), replace=False)] = ext
    xb = torch.from_numpy(x).to(torch.bfloat16)
    assert torch.isfinite(xb.float()).all()
    return xb


def check_act_bf16(act, x, b, clip=(1, 1)):
    q_ref, sx_ref, sum_ref, _ = quant.act_quant_staged(x, b, clip)
    assert np.array_equal(host(act.q), q_ref)
    assert np.array_equal(host(act.scale).view(np.uint32), sx_ref.view(np.uint32))
    assert np.array_equal(host(act.sum), sum_ref)
    return q_ref, sx_ref


@pytest.mark.parametrize("M,K,b", [(5, 4096, 4096), (4, 11008, 64), (4, 8192, 128), (4, 32768, 4096),
                                   (4, 14336, 2048), (4, 256, 2)])
def test_rotate_quant_act_bf16(Q, M, K, b):
    """bf16 input (qift_rotate_quant_act_bf16) over the whole finite bf16 range: bit-exact against the
    oracle's staged fp64 reading (exact on the fp16 grid)."""
    rng = np.random.default_rng(M * 7919 + K)
    x = _bf16_any(rng, M, K, b)
    for clip in ((1, 1), (9, 10)):
        act = Q.rotate_quant_act(x.cuda(), b, clip=clip)
        check_act_bf16(act, x.float().numpy(), b, clip)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("M,N,K,b", [(1, 4096, 4096, 4096), (3, 1040, 4096, 4096), (4, 528, 14336, 2048),
                                     (2, 640, 11008, 64)])
def test_fused_rotate_quant_linear_bf16(Q, fmt, M, N, K, b):
    """bf16 tokens into the fused entry (QIFT_SPEC_BF16): codes, accumulators and y bit-exact."""
    rng = np.random.default_rng(N + K + fmt)
    x = _bf16_any(rng, M, K, b)
    L = synth.draw_levels(fmt, N, K, cfg=90, layer=fmt, slot=M)
    s_w = synth.draw_scales(fmt, N, cfg=90, layer=fmt, slot=M)
    pk = pack_dev(Q, L, s_w, fmt)
    aq = Q.alloc_act(M, K, torch.device("cuda"))
    acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
    y = Q.rotate_quant_linear(pk, x.cuda(), b, acc_out=acc, act_out=aq)
    torch.cuda.synchronize()
    q_ref, sx_ref = check_act_bf16(aq, x.float().numpy(), b)
    acc_ref = olin.int_dot(L, q_ref)
    assert np.array_equal(host(acc), acc_ref)
    assert np.array_equal(bits16(host(y)), bits16(olin.epilogue_fp32(acc_ref, sx_ref, s_w)))


# ----------------------------------------------------------------------------- full-size configs


def _config_linear(Q, cfg, layer, shp, fmt, M, rows=None, tokens=None):
    L = synth.draw_levels(fmt, shp.N, shp.K, cfg=cfg, layer=layer, slot=synth.LINEAR_ID[shp.name])
    s_w = synth.draw_scales(fmt, shp.N, cfg=cfg, layer=layer, slot=synth.LINEAR_ID[shp.name])
    c = synth.CONFIGS[cfg]
    x = synth.config_activations(c, layer, synth.SITE_OF[shp.name], M, shp.K)
    pk = pack_dev(Q, L, s_w, fmt)
    words = host(pk.words).view(np.uint32)
    if rows is None:
        assert np.array_equal(words, opack.pack(L, fmt))
    else:
        assert np.array_equal(words[rows], opack.pack(L[rows], fmt))
    act = Q.rotate_quant_act(dev(x), shp.block)
    q_ref, sx_ref = check_act(act, x, shp.block, tokens=tokens)
    y, acc = run_linear(Q, pk, act, M, shp.N)
    check_linear(y, acc, L, q_ref, sx_ref, s_w, rows=rows, tokens=tokens)


@pytest.mark.parametrize("name", ["q", "k", "v", "o", "gate", "up", "down"])
def test_cfg1_llama2_layer(Q, name):
    shp = next(s for s in synth.CONFIGS[1].linears if s.name == name)
    _config_linear(Q, 1, 0, shp, levels.FMT_W2_MNZ, 1)


@pytest.mark.parametrize("N", [12288, 22016])
def test_cfg1_row_concatenated(Q, N):
    # q|k|v and gate|up stacked along N, as the decode benchmark launches them
    shp = synth.LinearShape("q" if N == 12288 else "gate", N, 4096, 4096)
    _config_linear(Q, 1, 1, shp, levels.FMT_W2_MNZ, 1)


@pytest.mark.parametrize("M", [1, 4, 16])
@pytest.mark.parametrize("name", ["q", "k", "o", "gate", "down"])
def test_cfg2_llama31_decode(Q, M, name):
    shp = next(s for s in synth.CONFIGS[2].linears if s.name == name)
    _config_linear(Q, 2, 31 if name == "k" else 0, shp, levels.FMT_W2_MNZ, M)


@pytest.mark.parametrize("M", [1, 8, 64])
@pytest.mark.parametrize("name", ["gate", "up", "down"])
def test_cfg3_pot_mlp(Q, M, name):
    shp = next(s for s in synth.CONFIGS[3].linears if s.name == name)
    _config_linear(Q, 3, 0, shp, levels.FMT_W2_POT, M)


@pytest.mark.parametrize("fmt", [levels.FMT_W4_SYM, levels.FMT_W2_MNZ])
@pytest.mark.parametrize("name", ["q", "k", "gate", "down"])
def test_cfg4_prefill_sampled(Q, fmt, name):
    shp = next(s for s in synth.CONFIGS[4].linears if s.name == name)
    layer = 0 if fmt == levels.FMT_W4_SYM else 16
    rng = np.random.default_rng(hash((fmt, name)) & 0xFFFF)
    rows = np.sort(rng.choice(shp.N, size=96, replace=False))
    rows[-1] = shp.N - 1
    tokens = np.sort(rng.choice(2048, size=48, replace=False))
    tokens[-1] = 2047
    _config_linear(Q, 4, layer, shp, fmt, 2048, rows=rows, tokens=tokens)


@pytest.mark.parametrize("fmt", [levels.FMT_W4_SYM, levels.FMT_W2_MNZ])
def test_cfg4_row_concatenated(Q, fmt):
    # gate|up stacked along N (28672 rows), as the prefill benchmark launches it: the widest GEMM grid
    shp = synth.LinearShape("gate", 28672, 4096, 4096)
    layer = 1 if fmt == levels.FMT_W4_SYM else 17
    rng = np.random.default_rng(7 + fmt)
    rows = np.sort(rng.choice(shp.N, size=96, replace=False))
    rows[0], rows[-1] = 0, shp.N - 1
    tokens = np.sort(rng.choice(2048, size=48, replace=False))
    tokens[0], tokens[-1] = 0, 2047
    _config_linear(Q, 4, layer, shp, fmt, 2048, rows=rows, tokens=tokens)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("K", [64, 128, 320, 512, 576, 896])
def test_gemm_pipeline_tails(Q, fmt, K):
    # the prefill GEMM (M > 64, no workspace) over every count of k-steps that ends its pipeline
    # differently: W4 steps over 128 k with three stages (1, 1, 3, 4, 5, 7 steps: the unrolled loop
    # body, then one or two more, the last step partial at K = 64, 320, 576), W2 over 256 k with two
    # (1, 1, 2, 2, 3, 4 steps); 300 rows and 200 tokens leave partial tiles both ways
    N, M = 300, 200
    L = synth.draw_levels(fmt, N, K, cfg=96, layer=K)
    s_w = synth.draw_scales(fmt, N, cfg=96, layer=K)
    x = synth.activations_fp16(96, K, 0, M, K, 7, 30.0)
    pk = pack_dev(Q, L, s_w, fmt)
    act = Q.rotate_quant_act(dev(x), 64)
    q_ref, sx_ref = check_act(act, x, 64)
    for use_sum in (False, True):
        y, acc = run_linear(Q, pk, act, M, N, use_sum=use_sum)
        check_linear(y, acc, L, q_ref, sx_ref, s_w)


@pytest.mark.parametrize("fmt", FMTS)
def test_linear_wide_grid_ragged(Q, fmt):
    # a grid wide enough for the 128-token W4 tiles, with ragged rows, tokens and a half k-step
    N, K, b, M = 16400, 1088, 64, 2000
    L = synth.draw_levels(fmt, N, K, cfg=94)
    s_w = synth.draw_scales(fmt, N, cfg=94)
    x = synth.activations_fp16(94, 0, 0, M, K, 11, 30.0)
    pk = pack_dev(Q, L, s_w, fmt)
    act = Q.rotate_quant_act(dev(x), b)
    q_ref, sx_ref = check_act(act, x, b)
    y, acc = run_linear(Q, pk, act, M, N)
    check_linear(y, acc, L, q_ref, sx_ref, s_w)


def test_linear_deterministic(Q):
    N, K, M = 4096, 14336, 16
    L = synth.draw_levels(levels.FMT_W2_MNZ, N, K, cfg=93)
    s_w = synth.draw_scales(levels.FMT_W2_MNZ, N, cfg=93)
    x = synth.activations_fp16(93, 0, 0, M, K, 143, 30.0)
    pk = pack_dev(Q, L, s_w, levels.FMT_W2_MNZ)
    act = Q.rotate_quant_act(dev(x), 2048)
    y1, a1 = run_linear(Q, pk, act, M, N)
    y2, a2 = run_linear(Q, pk, act, M, N)
    assert torch.equal(a1, a2) and torch.equal(y1.view(torch.int16), y2.view(torch.int16))


# ----------------------------------------------------------------------------- decode paths


@pytest.mark.parametrize("M,K,b", [(8, 14336, 2048), (16, 14336, 2048), (16, 4096, 4096), (12, 11008, 64)])
def test_decode_activation_paths(Q, M, K, b):
    # activations staged in LDS (M*K small), above 64 KiB of LDS, or read from global (M*K large)
    N = 784
    fmt = levels.FMT_W2_MNZ
    L = synth.draw_levels(fmt, N, K, cfg=95, layer=M)
    s_w = synth.draw_scales(fmt, N, cfg=95, layer=M)
    x = synth.activations_fp16(95, M, 1, M, K, K // 100, 30.0)
    pk = pack_dev(Q, L, s_w, fmt)
    act = Q.rotate_quant_act(dev(x), b)
    q_ref, sx_ref = check_act(act, x, b)
    y, acc = run_linear(Q, pk, act, M, N)
    check_linear(y, acc, L, q_ref, sx_ref, s_w)


# N covers every tiles-per-workgroup count of the decode kernel (ceil(N/16/256) = 1..6)
FUSED_SHAPES = [(512, 256, 256), (1000, 1088, 64), (4096, 4096, 4096), (2064, 11008, 64),
                (4096, 14336, 2048), (1040, 16384, 4096), (784, 8192, 8), (8208, 4096, 4096),
                (12288, 4096, 4096), (16400, 2048, 2048), (22016, 4096, 4096), (24592, 1024, 1024),
                (1040, 2048, 32), (6144, 4096, 4096), (28672, 4096, 4096)]


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("N,K,b", FUSED_SHAPES)
@pytest.mark.parametrize("M", [1, 4])
def test_fused_rotate_quant_linear(Q, fmt, N, K, b, M):
    L = synth.draw_levels(fmt, N, K, cfg=96, layer=K + M)
    s_w = synth.draw_scales(fmt, N, cfg=96, layer=K + M)
    x = synth.activations_fp16(96, K + M, 2, M, K, max(1, K // 100), 30.0)
    pk = pack_dev(Q, L, s_w, fmt)
    xd = dev(x)
    act = Q.alloc_act(M, K)
    acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
    y = Q.rotate_quant_linear(pk, xd, b, acc_out=acc, act_out=act)
    torch.cuda.synchronize()
    q_ref, sx_ref = check_act(act, x, b)
    check_linear(y, acc, L, q_ref, sx_ref, s_w)
    # bit-identical to the two-call form
    act2 = Q.rotate_quant_act(xd, b)
    y2, acc2 = run_linear(Q, pk, act2, M, N)
    assert torch.equal(acc, acc2) and torch.equal(y.view(torch.int16), y2.view(torch.int16))


@pytest.mark.parametrize("M", [2, 3])
def test_fused_clip_and_no_act_output(Q, M):
    N, K, b = 1024, 4096, 4096
    fmt = levels.FMT_W2_POT
    L = synth.draw_levels(fmt, N, K, cfg=97, layer=M)
    s_w = synth.draw_scales(fmt, N, cfg=97, layer=M)
    x = synth.activations_fp16(97, M, 0, M, K, 41, 30.0)
    x[M - 1] = 0                                    # a zero token inside the batch
    pk = pack_dev(Q, L, s_w, fmt)
    y = Q.rotate_quant_linear(pk, dev(x), b, clip=(9, 10))
    torch.cuda.synchronize()
    q_ref, sx_ref, _, _ = quant.act_quant(x, b, (9, 10))
    acc_ref = olin.int_dot(L, q_ref)
    assert np.array_equal(bits16(host(y)), bits16(olin.epilogue_fp32(acc_ref, sx_ref, s_w)))


# ----------------------------------------------------------------------------- graph replay


def test_graph_replay_matches_eager(Q):
    # one decode layer slice captured as a hipGraph, replayed several times with eager work
    # and synchronizations in between; every replay must equal the eager result
    K, b = 4096, 4096
    shapes = [(3 * 1024, levels.FMT_W2_MNZ), (2048, levels.FMT_W2_POT), (1024, levels.FMT_W4_SYM)]
    pks = []
    for i, (N, fmt) in enumerate(shapes):
        L = synth.draw_levels(fmt, N, K, cfg=98, layer=i)
        pks.append(pack_dev(Q, L, synth.draw_scales(fmt, N, cfg=98, layer=i), fmt))
    x = dev(synth.activations_fp16(98, 0, 0, 1, K, 41, 30.0))
    xs = dev(synth.activations_fp16(98, 1, 0, 16, K, 41, 30.0))
    acts = Q.alloc_act(16, K)
    outs = [torch.empty((1, N), dtype=torch.float16, device="cuda") for N, _ in shapes]
    outs16 = [torch.empty((16, N), dtype=torch.float16, device="cuda") for N, _ in shapes]

    def step():
        for pk, o in zip(pks, outs):
            Q.rotate_quant_linear(pk, x, b, out=o)
        Q.rotate_quant_act(xs, b, out=acts)
        for pk, o in zip(pks, outs16):
            Q.linear(pk, acts, out=o)

    step()
    torch.cuda.synchronize()
    eager = [o.clone() for o in outs + outs16]
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    with torch.cuda.graph(g):
        step()
    for _ in range(4):
        for o in outs + outs16:
            o.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for o, e in zip(outs + outs16, eager):
            assert torch.equal(o.view(torch.int16), e.view(torch.int16))


@pytest.mark.parametrize("nwords", [4, 16_388, 262_156, 10_485_764])
def test_hbm_read_probe_reads_every_word(Q, nwords):
    # the bandwidth probe must touch every 32-bit word once: its per-segment XORs are the host's
    words = np.random.default_rng(nwords).integers(0, 2**32, size=nwords, dtype=np.uint64).astype(np.uint32)
    buf = dev(words)
    parts = torch.full((Q.read_probe_slots(4 * nwords),), -1, dtype=torch.int32, device="cuda")
    Q.hbm_read_probe(buf, parts)
    torch.cuda.synchronize()
    seg = Q.READ_PROBE_SEGMENT // 4
    expect = [np.bitwise_xor.reduce(words[i:i + seg]) for i in range(0, nwords, seg)]
    assert np.array_equal(host(parts).view(np.uint32), np.array(expect, dtype=np.uint32))
