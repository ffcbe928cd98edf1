"""The persistent decode chain (qift_chain_prepare / qift_decode_chain) against the oracle.

A chain runs a decode step of a layer stack as one launch: each link rotates and quantizes its input
(the chain input, or a slice of an earlier link's fp16 output) and applies its quantized linear.  The
oracle runs the same links one by one on the CPU: act_quant of the link's input, the integer dot
product, the fp32 epilogue (expected bit for bit), and feeds its own fp16 output to the next link.
Every run of a chain uses a new input, so a read of a stale copy of an earlier output (a cache not
refreshed across the XCDs) shows as a mismatch.  Expected values come only from ``oracle``.
"""
import numpy as np
import pytest
import torch

from oracle import levels, linear as olin, quant
from paper_2606_02823_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def Q():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_02823_amd import qift
    qift.lib()
    return qift


def _dev(a):
    a = np.ascontiguousarray(a)
    return torch.from_numpy(a).cuda()


class Spec:
    """One link on the host: levels, scales and the chain wiring."""

    def __init__(self, fmt, N, K, block, in_link, in_offset, seed, s_w=None):
        self.fmt, self.N, self.K, self.block = fmt, N, K, block
        self.in_link, self.in_offset = in_link, in_offset
        self.L = synth.draw_levels(fmt, N, K, cfg=80, layer=seed)
        if s_w is None:
            # keep the activations' magnitude about constant along the chain: |y| ~ s_w s_x sqrt(K E l^2 E q^2)
            # with s_x ~ 0.57 sigma_x and E q^2 ~ 2.5, i.e. a gain of about 0.9 sqrt(E l^2) per unit s_w sqrt(K)
            jitter = synth.draw_scales(fmt, N, cfg=80, layer=seed).astype(np.float64)
            jitter /= np.median(jitter)
            gain = {levels.FMT_W2_MNZ: 1.7, levels.FMT_W2_POT: 2.24, levels.FMT_W4_SYM: 1.75}[fmt]
            s_w = (jitter / (gain * np.sqrt(K))).astype(np.float16)
        self.s_w = s_w


def oracle_chain(specs, x):
    """fp16 outputs and int64 accumulators of every link, computed link by link."""
    ys, accs = [], []
    for sp in specs:
        xin = x if sp.in_link < 0 else ys[sp.in_link][:, sp.in_offset:sp.in_offset + sp.K]
        xin = np.ascontiguousarray(xin)
        assert np.isfinite(xin.astype(np.float32)).all()
        q, sx, _, _ = quant.act_quant(xin, sp.block)
        acc = olin.int_dot(sp.L, q)
        ys.append(olin.epilogue_fp32(acc, sx, sp.s_w))
        accs.append(acc)
    return ys, accs


def build(Q, specs, M, acc=True):
    pks = []
    for sp in specs:
        if sp.fmt == levels.FMT_W4_SYM:
            pks.append(Q.pack_w4(_dev(sp.L), _dev(sp.s_w)))
        else:
            pks.append(Q.pack_w2(_dev(sp.L), _dev(sp.s_w), sp.fmt))
    links = [Q.ChainLink(pk, sp.block, sp.in_link, sp.in_offset) for pk, sp in zip(pks, specs)]
    return Q.Chain(links, M, acc=acc), pks


def check_run(Q, chain, specs, x, acc=True):
    chain.run(_dev(x))
    torch.cuda.synchronize()
    ys, accs = oracle_chain(specs, x)
    for i, (y, a) in enumerate(zip(ys, accs)):
        if acc:
            assert np.array_equal(chain.accs[i].cpu().numpy(), a), f"link {i} accumulators"
        # bit-exact against the oracle's fp32 epilogue (within 1e-3 of its fp64 one: the parity tests)
        assert np.array_equal(chain.outs[i].cpu().numpy().view(np.uint16), y.view(np.uint16)), f"link {i} y"
    return ys


def llama31_layers(fmt, layers, seed0=0):
    """q|k|v, o, gate|up, down per layer (LLaMA-3.1-8B shapes): o reads the q part of q|k|v, down the
    gate part of gate|up, the next layer's q|k|v the down output (synthetic stand-ins for attention and
    the gated activation)."""
    specs = []
    for l in range(layers):
        base = len(specs)
        prev = base - 1
        specs.append(Spec(fmt, 6144, 4096, 4096, prev if l else -1, 0, seed0 + 4 * l))
        specs.append(Spec(fmt, 4096, 4096, 4096, base, 0, seed0 + 4 * l + 1))
        specs.append(Spec(fmt, 28672, 4096, 4096, base + 1, 0, seed0 + 4 * l + 2))
        specs.append(Spec(fmt, 4096, 14336, 2048, base + 2, 0, seed0 + 4 * l + 3))
    return specs


def test_chain_two_llama31_layers_mnz(Q):
    """Two LLaMA-3.1-8B decode layers chained (8 links, the real shapes and dependencies): bit-exact,
    on three runs with different inputs (the second and third would expose stale reads)."""
    M = 1
    specs = llama31_layers(levels.FMT_W2_MNZ, 2)
    chain, _ = build(Q, specs, M)
    for r in range(3):
        x = synth.activations_fp16(81, r, 0, M, 4096, 41, 30.0)
        check_run(Q, chain, specs, x)
    assert Q.device_error() == 0


def mixed_specs(fmt):
    """Shapes that exercise every path: workgroups without tiles (N/16 < CUs), K of 1, 3 and 4
    rotation tiles, blocks 64 / 256 / 2048 / 4096, tiles per workgroup above the chunk size (several
    chunks), inputs taken at an offset inside the producer's row."""
    return [Spec(fmt, 1040, 4096, 4096, -1, 0, 1),
            Spec(fmt, 11008, 1024, 256, 0, 8, 2),
            Spec(fmt, 4096, 11008, 64, 1, 0, 3),
            Spec(fmt, 20000, 4096, 4096, 2, 0, 4),
            Spec(fmt, 784, 14336, 2048, 3, 8, 5),
            Spec(fmt, 40000, 768, 256, 4, 16, 6),
            Spec(fmt, 2064, 8192, 2048, 5, 64, 7)]


def multi_token_specs(fmt):
    """Links with K <= 8192 (several tokens per call fit in LDS): 1 and 2 rotation tiles, every block,
    idle workgroups and several chunks."""
    return [Spec(fmt, 1040, 4096, 4096, -1, 0, 11),
            Spec(fmt, 8208, 1024, 256, 0, 8, 12),
            Spec(fmt, 20000, 8192, 2048, 1, 8, 13),
            Spec(fmt, 4112, 4096, 4096, 2, 4000, 14),
            Spec(fmt, 30000, 4096, 64, 3, 0, 15),
            Spec(fmt, 496, 8192, 4096, 4, 2048, 16)]


@pytest.mark.parametrize("fmt", [levels.FMT_W2_MNZ, levels.FMT_W2_POT, levels.FMT_W4_SYM])
def test_chain_mixed_shapes(Q, fmt):
    M = 1
    specs = mixed_specs(fmt)
    chain, _ = build(Q, specs, M)
    for r in range(2):
        x = synth.activations_fp16(82, 10 * fmt + r, 0, M, 4096, 41, 30.0)
        check_run(Q, chain, specs, x)
    assert Q.device_error() == 0


@pytest.mark.parametrize("fmt,M", [(levels.FMT_W2_MNZ, 4), (levels.FMT_W2_POT, 2), (levels.FMT_W4_SYM, 3)])
def test_chain_multi_token(Q, fmt, M):
    specs = multi_token_specs(fmt)
    chain, _ = build(Q, specs, M)
    for r in range(2):
        x = synth.activations_fp16(86, 10 * fmt + r, 0, M, 4096, 41, 30.0)
        check_run(Q, chain, specs, x)
    assert Q.device_error() == 0


@pytest.mark.parametrize("fmt,M", [(levels.FMT_W2_MNZ, 2), (levels.FMT_W2_POT, 3), (levels.FMT_W4_SYM, 2)])
def test_chain_multi_token_long_links(Q, fmt, M):
    """Several tokens through links of 3 and 4 rotation tiles (K = 11008, 14336), whose tiles the
    activation group and the two weight-wave groups rotate at once, one token after another."""
    specs = [Spec(fmt, 4096, 4096, 4096, -1, 0, 21),
             Spec(fmt, 11008, 4096, 4096, 0, 0, 22),
             Spec(fmt, 4096, 11008, 64, 1, 0, 23),
             Spec(fmt, 14336, 4096, 4096, 2, 0, 24),
             Spec(fmt, 2064, 14336, 2048, 3, 0, 25),
             Spec(fmt, 9000, 2048, 256, 4, 16, 26),
             Spec(fmt, 784, 12288, 4096, 3, 0, 27)]
    chain, _ = build(Q, specs, M)
    for r in range(2):
        x = synth.activations_fp16(87, 10 * fmt + r, 0, M, 4096, 41, 30.0)
        check_run(Q, chain, specs, x)
    assert Q.device_error() == 0


def test_chain_rejects_what_does_not_fit(Q):
    # four tokens next to a K = 14336 link exceed one workgroup's LDS; a block the kernel was not
    # compiled for is refused
    specs = llama31_layers(levels.FMT_W2_MNZ, 1, seed0=50)
    with pytest.raises(Q.QiftError, match="QIFT_ERR_SHAPE"):
        build(Q, specs, 4)
    specs = [Spec(levels.FMT_W2_MNZ, 512, 4096, 1024, -1, 0, 51)]
    with pytest.raises(Q.QiftError, match="QIFT_ERR_SPEC"):
        build(Q, specs, 1)


def test_chain_graph_replay(Q):
    """The chain step captured in a HIP graph and replayed with eager work and synchronizations in
    between: every replay equals the oracle for the input it saw."""
    specs = llama31_layers(levels.FMT_W2_MNZ, 1, seed0=40)
    chain, _ = build(Q, specs, 1, acc=False)
    xd = torch.empty((1, 4096), dtype=torch.float16, device="cuda")
    xd.copy_(_dev(synth.activations_fp16(83, 0, 0, 1, 4096, 41, 30.0)))
    chain.run(xd)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        chain.run(xd)
    torch.cuda.current_stream().wait_stream(s)
    with torch.cuda.graph(g):
        chain.run(xd)
    for r in range(1, 4):
        x = synth.activations_fp16(83, r, 0, 1, 4096, 41, 30.0)
        xd.copy_(_dev(x))
        for o in chain.outs:
            o.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        ys, _ = oracle_chain(specs, x)
        for i, y in enumerate(ys):
            assert np.array_equal(chain.outs[i].cpu().numpy().view(np.uint16), y.view(np.uint16)), (r, i)
    assert Q.device_error() == 0


def test_chain_wait_gives_up_and_is_reported(Q):
    """Host-forced: with a tiny wait limit the workgroups stop waiting for each other (and for their
    own waves), compute on whatever the buffers hold, and every kernel still exits; the error word
    reports it.  With the default limit the same chain is exact again and reports nothing."""
    specs = mixed_specs(levels.FMT_W2_MNZ)[:4]
    chain, _ = build(Q, specs, 1)
    for o in chain.outs:
        o.zero_()   # finite values for the links that read them early
    x = synth.activations_fp16(84, 0, 0, 1, 4096, 41, 30.0)
    Q.device_error(clear=True)
    Q.set_wait_limit(1)
    try:
        for _ in range(3):
            chain.run(_dev(x))
        bits = Q.device_error(clear=True)
    finally:
        Q.set_wait_limit(0)
    assert bits & (Q.DEVERR_CHAIN_WAIT | Q.DEVERR_GROUP_WAIT)
    check_run(Q, chain, specs, synth.activations_fp16(84, 1, 0, 1, 4096, 41, 30.0))
    assert Q.device_error() == 0


def test_chain_matches_fused_entry(Q):
    """Each link of a chain equals qift_rotate_quant_linear on the same input, bit for bit."""
    specs = multi_token_specs(levels.FMT_W2_POT)[:4]
    chain, pks = build(Q, specs, 2)
    x = synth.activations_fp16(85, 0, 0, 2, 4096, 41, 30.0)
    chain.run(_dev(x))
    torch.cuda.synchronize()
    for i, (sp, pk) in enumerate(zip(specs, pks)):
        xin = _dev(x) if sp.in_link < 0 else chain.outs[sp.in_link][:, sp.in_offset:sp.in_offset + sp.K].contiguous()
        y = Q.rotate_quant_linear(pk, xin, sp.block)
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int16), chain.outs[i].view(torch.int16)), i
