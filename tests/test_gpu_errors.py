"""Device-side error reporting of the bounded waits, forced from the host.

The fused decode kernel's activation waves synchronize among themselves with a
bounded spin.  A test hook lowers the spin limit so that those waits give up:
every kernel must still exit normally, the per-device error word must report
the give-up, and with the default limit restored the same call must be exact
again and report nothing.  No kernel here faults or hangs: a wave that gives up
only computes on stale LDS values (every index stays in range).
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
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def test_group_wait_gives_up_and_is_reported(Q):
    N, K, b, M = 4096, 4096, 4096, 2
    fmt = levels.FMT_W2_MNZ
    L = synth.draw_levels(fmt, N, K, cfg=99, layer=1)
    s_w = synth.draw_scales(fmt, N, cfg=99, layer=1)
    x = synth.activations_fp16(99, 1, 0, M, K, 41, 30.0)
    pk = Q.pack_w2(_dev(L), _dev(s_w), Q.W2_MNZ)
    xd = _dev(x)
    y = torch.empty((M, N), dtype=torch.float16, device="cuda")
    Q.device_error(clear=True)                      # start from a clear word
    Q.rotate_quant_linear(pk, xd, b, out=y)
    assert Q.device_error() == 0                    # a normal call reports nothing
    Q.set_wait_limit(1)
    try:
        for _ in range(4):
            Q.rotate_quant_linear(pk, xd, b, out=y)
        bits = Q.device_error(clear=True)           # synchronizes: every kernel has exited
    finally:
        Q.set_wait_limit(0)
    assert bits & Q.DEVERR_GROUP_WAIT
    # default limit again: exact results, nothing reported
    acc = torch.empty((M, N), dtype=torch.int32, device="cuda")
    y = Q.rotate_quant_linear(pk, xd, b, acc_out=acc)
    bits = Q.device_error()
    q_ref, sx_ref, _, _ = quant.act_quant(x, b)
    acc_ref = olin.int_dot(L, q_ref)
    assert np.array_equal(acc.cpu().numpy(), acc_ref)
    assert np.array_equal(y.cpu().numpy().view(np.uint16),
                          olin.epilogue_fp32(acc_ref, sx_ref, s_w).view(np.uint16))
    assert bits == 0
