"""Full-size and end-to-end parity of the HIP path against the oracle.

* The LLaMA-3.1-8B prefill schedule at M = 2048 tokens: layer 15 (W4) chained into layer 16 (W2 MNZ),
  the mixed schedule of Sec. 4.4, Eq. (24) at the boundary where the format changes.  Each linear's
  input is an earlier linear's fp16 output (o reads the q part of q|k|v, gate|up reads o, down reads the
  gate part of gate|up, layer 16's q|k|v reads layer 15's down), and every output element (int32
  accumulator and fp16 y) of the 8 linears is compared, covering all seven shapes of both formats.
* The whole pipeline of Sec. 3 from each config's Student-t weights: the oracle's rotation and level
  quantization (RMS scale, 64-candidate MSE scale, absmax / 7), the GPU packer, rotate_quant_act and
  the linear, on a block of rows of every linear.
* A seeded random sweep over shapes, blocks, formats and fp16 extremes (stops at the first mismatch).

Expected values come only from ``oracle``; the GPU's bit-exact agreement on every linear is what
lets the next linear start from the oracle's own output.
"""
import numpy as np
import pytest
import torch

from oracle import hadamard, levels, linear as olin, pack as opack, quant
from paper_2606_02823_amd import synth

pytestmark = pytest.mark.gpu


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


def run_and_check(Q, L, s_w, fmt, x, b, check_words=True):
    """pack, rotate_quant_act and the linear on the GPU; every packed word, code, scale, code sum,
    accumulator and output against the oracle.  Returns the oracle's fp16 output."""
    M, K = x.shape
    N = L.shape[0]
    pk = pack_dev(Q, L, s_w, fmt)
    if check_words:
        assert np.array_equal(host(pk.words).view(np.uint32), opack.pack(L, fmt)), "packed words"
    act = Q.rotate_quant_act(dev(x), b)
    acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
    y = Q.linear(pk, act, acc_out=acc)
    torch.cuda.synchronize()
    q_ref, sx_ref, sum_ref, _ = quant.act_quant(x, b)
    assert np.array_equal(host(act.q), q_ref), "act_q"
    assert np.array_equal(host(act.scale).view(np.uint32), sx_ref.view(np.uint32)), "act_scale"
    assert np.array_equal(host(act.sum), sum_ref), "act_sum"
    acc_ref = olin.int_dot(L, q_ref)
    assert np.array_equal(host(acc), acc_ref), "accumulators"
    y_ref = olin.epilogue_fp32(acc_ref, sx_ref, s_w)
    assert np.array_equal(bits16(host(y)), bits16(y_ref)), "y"
    # the fp64 reading within the tolerance wherever it is finite (next to the fp16 overflow threshold
    # the two roundings may land on 65504 and inf)
    y64 = olin.epilogue_ref(acc_ref, sx_ref, s_w)
    fin = np.isfinite(y64.astype(np.float32))
    assert olin.max_abs_rel(host(y)[fin], y64[fin]) <= olin.TOL_REL
    return y_ref


# ----------------------------------------------------------------------------- cfg4 schedule

# gain of one linear on the activations' RMS per unit of s_w sqrt(K) for drawn levels: with
# s_w = jitter / (gain sqrt(K)) the magnitudes stay about constant along the chain
GAIN = {levels.FMT_W2_MNZ: 1.7, levels.FMT_W2_POT: 2.24, levels.FMT_W4_SYM: 1.75}
SCHEDULE = [(15, "qkv"), (15, "o"), (15, "gate_up"), (15, "down"),
            (16, "qkv"), (16, "o"), (16, "gate_up"), (16, "down")]
# (N, K, block) of the four launches of a layer (q|k|v and gate|up stacked along N)
SHAPES4 = {"qkv": (6144, 4096, 4096), "o": (4096, 4096, 4096), "gate_up": (28672, 4096, 4096),
           "down": (4096, 14336, 2048)}
SCHED_OUT = {}


def _schedule_input(step):
    c = synth.CONFIGS[4]
    layer, name = SCHEDULE[step]
    K = SHAPES4[name][1]
    if step == 0:
        return synth.config_activations(c, layer, 0, 2048, K)
    # every link reads the first K columns of the link before it (the q part of q|k|v, all of o,
    # the gate part of gate|up, all of down)
    return np.ascontiguousarray(SCHED_OUT[step - 1][:, :K])


@pytest.mark.parametrize("step", range(len(SCHEDULE)))
def test_cfg4_schedule_w4_into_w2_full(Q, step):
    if step > 0 and step - 1 not in SCHED_OUT:
        pytest.skip("the link before this one did not pass")
    c = synth.CONFIGS[4]
    layer, name = SCHEDULE[step]
    fmt = c.fmt_of_layer[layer]
    assert fmt == (levels.FMT_W4_SYM if layer < 16 else levels.FMT_W2_MNZ)   # the L = 16 boundary
    N, K, b = SHAPES4[name]
    print(f"cfg4 schedule step {step}: layer {layer} {name} fmt {fmt} N={N} K={K} M=2048", flush=True)
    x = _schedule_input(step)
    assert np.isfinite(x.astype(np.float32)).all()
    L = synth.draw_levels(fmt, N, K, cfg=4, layer=layer, slot=step)
    jit = synth.draw_scales(fmt, N, cfg=4, layer=layer, slot=step).astype(np.float64)
    s_w = (jit / np.median(jit) / (GAIN[fmt] * np.sqrt(K))).astype(np.float16)
    SCHED_OUT[step] = run_and_check(Q, L, s_w, fmt, x, b)


# ----------------------------------------------------------------------------- weights -> linear

PIPE_ROWS = 200   # a ragged block (12.5 tiles of 16 rows) of each linear


@pytest.mark.parametrize("cfg,layer,M", [(1, 0, 1), (2, 0, 4), (2, 31, 16), (3, 0, 8), (3, 5, 64),
                                         (4, 0, 256), (4, 16, 256)])
def test_pipeline_from_student_t_weights(Q, cfg, layer, M):
    c = synth.CONFIGS[cfg]
    fmt = c.fmt_of_layer[layer]
    for shp in c.linears:
        print(f"pipeline cfg{cfg} layer {layer} {shp.name} fmt {fmt} rows {PIPE_ROWS} K={shp.K} M={M}", flush=True)
        W = synth.weights_fp32(cfg, layer, shp.name, PIPE_ROWS, shp.K)
        L, s_w = quant.quantize_weights(hadamard.rotate_weights(W, shp.block), fmt)
        x = synth.config_activations(c, layer, synth.SITE_OF[shp.name], M, shp.K)
        run_and_check(Q, L, s_w, fmt, x, shp.block)


# ----------------------------------------------------------------------------- random sweep

FP16_EXTREMES = np.array([65504.0, -65504.0, 6.103515625e-05, -6.103515625e-05, 5.960464477539063e-08,
                          -5.960464477539063e-08, 0.0, -0.0, 1.0, -1.0, 0.5, 2048.0], dtype=np.float16)


def _sweep_case(rng):
    fmt = int(rng.choice([levels.FMT_W2_MNZ, levels.FMT_W2_POT, levels.FMT_W4_SYM]))
    M = int(rng.integers(1, 81))
    N = 64 * int(rng.integers(1, 65))
    K = 64 * int(rng.integers(1, 65))
    blocks = [b for b in (2, 4, 8, 16, 32, 64, 128, 256, 512, 1024, 2048, 4096) if K % b == 0]
    b = int(rng.choice(blocks))
    x = (rng.standard_normal((M, K)) * np.exp(rng.uniform(-6, 6))).astype(np.float16)
    x[~np.isfinite(x)] = 0
    # fp16 extremes at random places, one token of zeros and one token of a single extreme value
    n_ext = int(rng.integers(0, 9))
    x[rng.integers(0, M, n_ext), rng.integers(0, K, n_ext)] = rng.choice(FP16_EXTREMES, n_ext)
    if M > 2 and rng.random() < 0.5:
        x[int(rng.integers(0, M))] = 0
        t = int(rng.integers(0, M))
        x[t] = 0
        x[t, int(rng.integers(0, K))] = rng.choice(FP16_EXTREMES)
    vals = {levels.FMT_W2_MNZ: [-3, -1, 1, 3], levels.FMT_W2_POT: [-4, -1, 1, 4],
            levels.FMT_W4_SYM: list(range(-7, 8))}[fmt]
    L = rng.choice(np.array(vals, dtype=np.int8), size=(N, K))
    # per-row scales over a wide range (some overflowing the fp16 output to inf), a zero scale row
    s_w = np.exp(rng.uniform(-12, 2, N)).astype(np.float16)
    s_w[int(rng.integers(0, N))] = 0
    return fmt, M, N, K, b, x, L, s_w


def test_random_shape_sweep(Q):
    rng = np.random.default_rng(20261202)
    for case in range(48):
        fmt, M, N, K, b, x, L, s_w = _sweep_case(rng)
        print(f"sweep case {case}: fmt {fmt} M={M} N={N} K={K} block={b}", flush=True)
        run_and_check(Q, L, s_w, fmt, x, b)
        if M <= 4 and b <= 4096:
            # the fused entry on the same operands: the same y bit for bit
            pk = pack_dev(Q, L, s_w, fmt)
            y = Q.rotate_quant_linear(pk, dev(x), b)
            torch.cuda.synchronize()
            q_ref, sx_ref, _, _ = quant.act_quant(x, b)
            y_ref = olin.epilogue_fp32(olin.int_dot(L, q_ref), sx_ref, s_w)
            assert np.array_equal(bits16(host(y)), bits16(y_ref)), f"fused y, case {case}"
