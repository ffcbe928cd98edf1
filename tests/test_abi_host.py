"""Host-only checks of libqift's C ABI: it loads, exports every declared symbol,
and rejects bad arguments with the documented status before any HIP call.

No call here reaches a kernel launch: every argument set fails validation
(the pointers passed are never dereferenced on the host or the device)."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2606_02823_amd import qift

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qift.h")

OK, E_NULL, E_SHAPE, E_SPEC, E_FORMAT, E_CODE, E_ALIGN, E_WS = 0, -1, -2, -3, -4, -5, -6, -8
A = 0x10000       # a 16-byte aligned fake device address (never dereferenced)
MIS = 0x10008     # an 8-byte aligned, not 16-byte aligned fake address


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(qift.LIB_PATH):
        pytest.skip("libqift.so not built")
    return qift.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(qift_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert len(names) == 28
    assert sorted(qift.EXPORTS) == names
    for n in names:
        assert hasattr(L, n), n


def test_version_and_status_strings(L):
    assert qift.version().startswith("qift")
    for code in (0, -1, -2, -3, -4, -5, -6, -7, -8):
        assert L.qift_status_string(code)
    assert L.qift_status_string(12345) == b"unknown status"


def test_packed_bytes(L):
    assert qift.packed_bytes(qift.W2_MNZ, 512, 256) == 512 * 256 // 4
    assert qift.packed_bytes(qift.W2_POT, 14336, 4096) == 14_680_064
    assert qift.packed_bytes(qift.W4_SYM, 4096, 14336) == 4096 * 14336 // 2
    assert qift.packed_bytes(qift.W2_MNZ, 4096, 100) == 0     # K % 64
    assert qift.packed_bytes(7, 4096, 4096) == 0              # unknown format
    assert qift.packed_bytes(qift.W2_MNZ, 0, 4096) == 0


def _spec(K=256, block=256, num=1, den=1, flags=None):
    return qift.HadamardSpec(K, block, qift.clip_flags(num, den) if flags is None else flags)


def test_spec_layout_and_clip_flags():
    # the boundary's spec is {int64 K; int32 block; int32 flags}: 16 bytes, flags 0 = clip 1
    assert ctypes.sizeof(qift.HadamardSpec) == 16
    assert qift.HadamardSpec.flags.offset == 12
    assert qift.clip_flags(1, 1) == 0
    assert qift.clip_flags(9, 10) == (9 << 8) | 10
    text = open(HEADER).read()
    assert "#define QIFT_CLIP(num, den) ((int32_t)((((num) & 0xFF) << 8) | ((den) & 0xFF)))" in text


def test_quantize_weights_validation(L):
    f = L.qift_quantize_weights
    mnz, pot, w4 = qift.W2_MNZ, qift.W2_POT, qift.W4_SYM
    assert f(None, 8, _spec(), mnz, A, A, None) == E_NULL
    assert f(A, 8, _spec(), pot, None, A, None) == E_NULL
    assert f(A, 8, _spec(), w4, A, None, None) == E_NULL
    assert f(A, 8, _spec(), 7, A, A, None) == E_FORMAT
    assert f(A, 0, _spec(), mnz, A, A, None) == E_SHAPE
    assert f(A, 8, _spec(K=100, block=4), mnz, A, A, None) == E_SHAPE
    assert f(A, 8, _spec(K=16448, block=64), mnz, A, A, None) == E_SHAPE     # K > 16384
    assert f(A, 1 << 18, _spec(K=8192, block=64), mnz, A, A, None) == E_SHAPE   # N K >= 2^31
    assert f(A, 8, _spec(block=48), mnz, A, A, None) == E_SPEC
    assert f(A, 8, _spec(K=8192, block=8192), mnz, A, A, None) == E_SPEC    # block above 4096
    assert f(A, 8, _spec(K=192, block=128), mnz, A, A, None) == E_SPEC      # block does not divide K
    assert f(A, 8, _spec(num=9, den=10), w4, A, A, None) == E_SPEC          # no clip on weights
    assert f(A, 8, _spec(flags=1 << 16), mnz, A, A, None) == E_SPEC
    assert f(MIS, 8, _spec(), mnz, A, A, None) == E_ALIGN
    assert f(A, 8, _spec(), mnz, MIS, A, None) == E_ALIGN


def test_quantize_weights_mirror_validation(L):
    f = L.qift_quantize_weights_mirror
    assert f(None, 8, _spec(), 0.3, A, A, None) == E_NULL
    assert f(A, 8, _spec(), 0.3, None, A, None) == E_NULL
    assert f(A, 8, _spec(), 0.3, A, None, None) == E_NULL
    assert f(A, 0, _spec(), 0.3, A, A, None) == E_SHAPE
    assert f(A, 8, _spec(K=16448, block=64), 0.3, A, A, None) == E_SHAPE
    assert f(A, 1 << 18, _spec(K=8192, block=64), 0.3, A, A, None) == E_SHAPE
    assert f(A, 8, _spec(block=48), 0.3, A, A, None) == E_SPEC
    assert f(A, 8, _spec(flags=1 << 16), 0.3, A, A, None) == E_SPEC
    for r in (0.0, 1.0, -0.3, 1.5, float("nan"), float("inf")):
        assert f(A, 8, _spec(), r, A, A, None) == E_SPEC, r
    assert f(MIS, 8, _spec(), 0.3, A, A, None) == E_ALIGN
    assert f(A, 8, _spec(), 0.3, A, MIS, None) == E_ALIGN


def test_ratio_scan_validation(L):
    f = L.qift_ratio_scan
    dv = lambda *v: (ctypes.c_double * len(v))(*v)
    r, c = dv(0.25, 0.3), dv(0.2, 0.5, 1.0)
    assert f(None, 100, r, 2, c, 3, A, A, A, A, None) == E_NULL
    assert f(A, 100, None, 2, c, 3, A, A, A, A, None) == E_NULL
    assert f(A, 100, r, 2, None, 3, A, A, A, A, None) == E_NULL
    for k in range(4):
        out = [A] * 4
        out[k] = None
        assert f(A, 100, r, 2, c, 3, *out, None) == E_NULL
    assert f(A, 0, r, 2, c, 3, A, A, A, A, None) == E_SHAPE
    assert f(A, 1 << 40, r, 2, c, 3, A, A, A, A, None) == E_SHAPE
    assert f(A, 100, r, 0, c, 3, A, A, A, A, None) == E_SHAPE
    assert f(A, 100, dv(*([0.5] * 1025)), 1025, c, 3, A, A, A, A, None) == E_SHAPE
    assert f(A, 100, r, 2, c, 0, A, A, A, A, None) == E_SHAPE
    assert f(A, 100, r, 2, dv(*([0.5] * 257)), 257, A, A, A, A, None) == E_SHAPE
    for bad in (0.0, 1.0, -0.1, float("nan")):
        assert f(A, 100, dv(0.3, bad), 2, c, 3, A, A, A, A, None) == E_SPEC, bad
    for bad in (0.0, -1.0, float("inf"), float("nan")):
        assert f(A, 100, r, 2, dv(0.5, bad), 2, A, A, A, A, None) == E_SPEC, bad
    for k in range(5):
        ptrs = [A] * 5
        ptrs[k] = MIS
        x, sse, nmse, best, stats = ptrs
        assert f(x, 100, r, 2, c, 3, sse, nmse, best, stats, None) == E_ALIGN


def test_kv4_validation(L):
    fq = L.qift_kv4_quant
    assert fq(None, 4, 128, A, A, A, None) == E_NULL
    assert fq(A, 4, 64, A, A, A, None) == E_SHAPE          # head_dim 128 only
    assert fq(A, 0, 128, A, A, A, None) == E_SHAPE
    assert fq(MIS, 4, 128, A, A, A, None) == E_ALIGN        # x: 16-byte loads
    assert fq(A, 4, 128, 0x10002, A, A, None) == E_ALIGN    # codes: 4-byte words
    assert fq(A, 4, 128, A, 0x10002, A, None) == E_ALIGN    # scales: fp32
    ws = L.qift_kv4_attention_workspace_bytes
    assert ws(2, 32, 8, 128, 1000) == 2 * 32 * 4 * 130 * 4   # 4 chunks of 256 tokens, 130 floats each
    assert ws(1, 32, 8, 64, 1000) == 0
    assert ws(1, 24, 8, 128, 1000) == 0                       # Hq / Hkv = 3
    f = L.qift_kv4_attention_decode
    good = ws(1, 32, 8, 128, 1000)
    for lay in (0, 1):                                        # token-major, head-major
        assert f(A, 1, 32, 8, 128, 1000, lay, A, A, A, A, A, None, A, A, good, None) == E_NULL
        assert f(A, 1, 32, 8, 128, 0, lay, A, A, A, A, A, A, A, A, good, None) == E_SHAPE
        assert f(A, 1, 32, 6, 128, 1000, lay, A, A, A, A, A, A, A, A, good, None) == E_SHAPE
        assert f(A, 1, 32, 8, 128, 1000, lay, A, A, A, A, A, A, A, A, good - 4, None) == E_WS
        assert f(A, 1, 32, 8, 128, 1000, lay, A, A, A, A, A, A, A, None, good, None) == E_WS
        assert f(A, 1, 32, 8, 128, 1000, lay, A, A, MIS, A, A, A, A, A, good, None) == E_ALIGN
    assert f(A, 1, 32, 8, 128, 1000, 2, A, A, A, A, A, A, A, A, good, None) == E_SPEC
    assert f(A, 1, 32, 8, 128, 1000, -1, A, A, A, A, A, A, A, A, good, None) == E_SPEC
    # the entry point without a workspace: the same checks, and calls beyond its 8 MiB array refused
    # (all before any HIP call)
    fn = L.qift_kv4_attention_decode_noalloc
    for lay in (0, 1):
        assert fn(A, 1, 32, 8, 128, 1000, lay, A, A, A, A, A, None, A, None) == E_NULL
        assert fn(A, 1, 32, 8, 128, 0, lay, A, A, A, A, A, A, A, None) == E_SHAPE
        assert fn(A, 1, 32, 8, 128, 1000, lay, A, A, MIS, A, A, A, A, None) == E_ALIGN
    assert fn(A, 1, 32, 8, 128, 1000, 2, A, A, A, A, A, A, A, None) == E_SPEC
    assert ws(1, 32, 8, 128, 129024) <= qift.KV4_SCRATCH_BYTES < ws(1, 32, 8, 128, 129025)
    assert fn(A, 1, 32, 8, 128, 129025, 1, A, A, A, A, A, A, A, None) == E_WS
    assert fn(A, 16, 32, 8, 128, 8192, 0, A, A, A, A, A, A, A, None) == E_WS


@pytest.mark.parametrize("entry", ["qift_rotate_quant_act", "qift_rotate_quant_act_bf16"])
def test_rotate_quant_act_validation(L, entry):
    f = getattr(L, entry)
    assert f(None, 4, _spec(), A, A, A, None) == E_NULL
    assert f(A, 4, _spec(), None, A, A, None) == E_NULL
    assert f(A, 4, _spec(), A, None, None, None) == E_NULL      # act_sum is optional, act_scale is not
    assert f(A, 0, _spec(), A, A, A, None) == E_SHAPE
    assert f(A, 4, _spec(K=100, block=4), A, A, A, None) == E_SHAPE
    assert f(A, 4, _spec(K=65536, block=4096), A, A, A, None) == E_SHAPE
    assert f(A, 4, _spec(block=48), A, A, A, None) == E_SPEC
    assert f(A, 4, _spec(block=1), A, A, A, None) == E_SPEC
    assert f(A, 4, _spec(K=16384, block=16384), A, A, A, None) == E_SPEC
    assert f(A, 4, _spec(K=192, block=128), A, A, A, None) == E_SPEC
    assert f(A, 4, _spec(num=0, den=1), A, A, A, None) == E_SPEC
    assert f(A, 4, _spec(num=3, den=2), A, A, A, None) == E_SPEC
    assert f(A, 4, _spec(num=9, den=17), A, A, A, None) == E_SPEC
    assert f(A, 4, _spec(flags=0x20101), A, A, A, None) == E_SPEC          # bits above the clip fields and the bf16 flag
    assert f(MIS, 4, _spec(), A, A, A, None) == E_ALIGN
    assert f(A, 4, _spec(), A, A, MIS, None) == E_ALIGN
    assert f(MIS, 4, _spec(), A, A, None, None) == E_ALIGN


def _pw(fmt=qift.W2_MNZ, N=512, K=256, packed=A, scales=A, layout=1):
    return qift.PackedW(fmt, layout, N, K, packed, scales)


def test_linear_validation(L):
    w2 = L.qift_w2a4_linear
    w4 = L.qift_w4a4_linear
    w2x = L.qift_w2a4_linear_ex
    w4x = L.qift_w4a4_linear_ex
    P = ctypes.byref
    # the base calls follow the boundary's w2a4_linear(packed_w, act_q, act_scale, out): no code sums
    assert w2(None, A, A, 4, A, None) == E_NULL
    assert w2(P(_pw()), None, A, 4, A, None) == E_NULL
    assert w2(P(_pw()), A, None, 4, A, None) == E_NULL
    assert w2(P(_pw()), A, A, 4, None, None) == E_NULL
    assert w2(P(_pw(packed=None)), A, A, 4, A, None) == E_NULL
    assert w2(P(_pw(scales=None)), A, A, 4, A, None) == E_NULL
    assert w2(P(_pw(fmt=qift.W4_SYM)), A, A, 4, A, None) == E_FORMAT
    assert w4(P(_pw(fmt=qift.W2_MNZ)), A, A, 4, A, None) == E_FORMAT
    assert w2(P(_pw(layout=2)), A, A, 4, A, None) == E_FORMAT
    assert w2(P(_pw(K=100)), A, A, 4, A, None) == E_SHAPE
    assert w2(P(_pw(N=0)), A, A, 4, A, None) == E_SHAPE
    assert w2(P(_pw()), A, A, 0, A, None) == E_SHAPE
    assert w2(P(_pw(packed=MIS)), A, A, 4, A, None) == E_ALIGN
    assert w2(P(_pw()), A, A, 4, MIS, None) == E_ALIGN
    assert w4(P(_pw(fmt=qift.W4_SYM)), MIS, A, 4, A, None) == E_ALIGN
    # _ex: the code sums are optional (NULL: summed in the kernel) and checked for alignment when given
    assert w2x(P(_pw()), A, A, MIS, 4, A, None, None, 0, None) == E_ALIGN
    assert w2x(P(_pw()), A, A, None, 4, A, MIS, None, 0, None) == E_ALIGN
    assert w2x(P(_pw()), A, A, A, 4, A, MIS, None, 0, None) == E_ALIGN
    assert w2x(P(_pw()), A, A, None, 4, A, None, None, 64, None) == E_WS
    assert w2x(P(_pw()), None, A, None, 4, A, None, None, 0, None) == E_NULL
    assert w4x(P(_pw(fmt=qift.W2_MNZ)), A, A, None, 4, A, None, None, 0, None) == E_FORMAT
    assert L.qift_workspace_bytes(P(_pw()), 4) == 0
    # the workspace that selects the FP4 x FP6 prefill kernel: MNZ and PoT at M > 64, M * 3K/4 bytes
    K = _pw().K
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W2_MNZ)), 64) == 0
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W2_MNZ)), 65) == 65 * 3 * (K // 4) + 65 * 4
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W2_POT)), 65) == 65 * 3 * (K // 4) + 65 * 4
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W4_SYM)), 65) == 0
    # 17..64 tokens: the skinny linear split over K when K > 4096 and its 16-row tiles are few (4 tiles
    # per workgroup, S ranges of K for about 256 workgroups, at most two 256-k units per K-slice):
    # S M N4 int32 partial sums (256-byte aligned), then S M int32 code sums; none for a gate|up width
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W2_POT, N=1000, K=14336)), 64) == 14 * 64 * 1000 * 4 + 14 * 64 * 4
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W2_MNZ, N=1000, K=14336)), 64) == 14 * 64 * 1000 * 4 + 14 * 64 * 4
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W2_POT, N=1000, K=14336)), 17) == 952064 + 14 * 17 * 4
    # a down shape (N >= 4096, K > 4096) from 33 tokens on: the prefill GEMM split over K (16 tiles -> S = 14)
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W2_MNZ, N=4096, K=14336)), 64) == 14 * 64 * 4096 * 4 + 14 * 64 * 4
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W2_MNZ, N=4096, K=14336)), 32) == 4 * 32 * 4096 * 4 + 4 * 32 * 4
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W2_MNZ, N=1000, K=4096)), 64) == 0
    # a gate|up width from 33 tokens on: the prefill GEMM split over K (112 tiles -> S = 4, W2 and W4);
    # 32 tokens keep the skinny kernel (no workspace)
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W2_MNZ, N=28672, K=4096)), 64) == 4 * 64 * 28672 * 4 + 4 * 64 * 4
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W2_MNZ, N=28672, K=4096)), 32) == 0
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W4_SYM, N=28672, K=4096)), 64) == 4 * 64 * 28672 * 4 + 4 * 64 * 4
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W4_SYM, N=28672, K=4096)), 32) == 4 * 32 * 28672 * 4 + 4 * 32 * 4
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W4_SYM, N=28672, K=4096)), 23) == 0
    # up to 16 tokens only where the decode kernel's LDS does not hold the codes (16 x 14336 does not,
    # 4 x 14336 and 16 x 4096 do)
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W2_MNZ, N=1000, K=14336)), 16) == 14 * 16 * 1000 * 4 + 14 * 16 * 4
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W2_MNZ, N=1000, K=14336)), 4) == 0
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W2_POT, N=1000, K=4096)), 16) == 0
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W4_SYM, N=1000, K=14336)), 64) == 0
    # above 64 tokens, where the 256 x 64 GEMM tiles are few, the int8 GEMM is split over K: S ranges of
    # at least 4 steps of 256 k, S = min(ceil(512 / tiles), 512 // tiles, steps // 4) when >= 2: S M N4
    # int32 partial sums (256-byte aligned), then S M int32 code sums
    W = L.qift_workspace_bytes
    # down at 128 tokens: 32 tiles, 56 steps -> S = 14
    assert W(P(_pw(fmt=qift.W2_MNZ, N=4096, K=14336)), 128) == 14 * 128 * 4096 * 4 + 14 * 128 * 4
    # gate|up at 65 tokens: 224 tiles -> S = 2
    assert W(P(_pw(fmt=qift.W2_POT, N=28672, K=4096)), 65) == 2 * 65 * 28672 * 4 + 2 * 65 * 4
    # ragged: 1000 rows (N4 = 1000), K = 4160 (17 steps, S = 4 of 5, 5, 5, 2), 96 tokens
    assert W(P(_pw(fmt=qift.W2_POT, N=1000, K=4160)), 96) == 4 * 96 * 1000 * 4 + 4 * 96 * 4
    # otherwise the FP4 x FP6 kernel's: FP6 codes and code sums, split over K itself where its tiles are
    # few (S = min(ceil(512 / tiles), 768 // tiles, steps // 4) when >= 2), the partial sums following
    # at the next multiple of 256 bytes.  q|k|v at 1024 tokens: 384 tiles -> S = 2; 65 x 5 tiles of
    # 16400 x 2048 at 320 tokens -> S = 2; 448 tiles (gate|up at 256) and 512 (down at 2048): unsplit
    assert W(P(_pw(fmt=qift.W2_MNZ, N=6144, K=4096)), 1024) == 1024 * 3072 + 1024 * 4 + 2 * 1024 * 6144 * 4
    assert W(P(_pw(fmt=qift.W2_MNZ, N=16400, K=2048)), 320) == 320 * 1536 + 320 * 4 + 2 * 320 * 16400 * 4
    assert W(P(_pw(fmt=qift.W2_MNZ, N=28672, K=4096)), 256) == 256 * 3072 + 256 * 4
    assert W(P(_pw(fmt=qift.W2_MNZ, N=4096, K=14336)), 2048) == 2048 * 10752 + 2048 * 2 * 4
    # W4 above 64 tokens: the int8 GEMM split over K where its tiles are few, S ranges of at least 8
    # steps of 128 k, S = min(ceil(512 / tiles), 512 // tiles, steps // 8) when >= 3: S M N4 int32
    # partial sums (256-byte aligned), then S M int32 code sums
    assert W(P(_pw(fmt=qift.W4_SYM, N=4096, K=14336)), 128) == 14 * 128 * 4096 * 4 + 14 * 128 * 4
    assert W(P(_pw(fmt=qift.W4_SYM, N=28672, K=4096)), 65) == 0        # 224 tiles: S = 2
    assert W(P(_pw(fmt=qift.W4_SYM, N=4096, K=4096)), 512) == 4 * 512 * 4096 * 4 + 4 * 512 * 4
    assert W(P(_pw(fmt=qift.W4_SYM, N=4096, K=14336)), 2048) == 0
    assert W(P(_pw(fmt=qift.W4_SYM, N=4096, K=14336)), 64) == 14 * 64 * 4096 * 4 + 14 * 64 * 4
    assert W(P(_pw(fmt=qift.W4_SYM, N=4096, K=14336)), 24) == 14 * 24 * 4096 * 4 + 14 * 24 * 4   # W4 from 24
    assert W(P(_pw(fmt=qift.W4_SYM, N=4096, K=14336)), 23) == 0
    # FP6 codes (M 3K/4 bytes), then one int32 code sum per token and 256 groups of 32 k
    need = 100 * 3 * (K // 4) + 100 * 4
    assert L.qift_workspace_bytes(P(_pw(fmt=qift.W2_MNZ)), 100) == need
    assert w2x(P(_pw(fmt=qift.W2_MNZ)), A, A, A, 100, A, None, A, need - 16, None) == E_WS
    assert w2x(P(_pw(fmt=qift.W2_MNZ)), A, A, A, 100, A, None, None, need, None) == E_WS
    assert w2x(P(_pw(fmt=qift.W2_MNZ)), A, A, A, 100, A, None, MIS, need, None) == E_ALIGN


def test_fused_validation(L):
    f = L.qift_rotate_quant_linear
    P = ctypes.byref
    sp = _spec(K=256, block=256)
    assert f(None, A, 1, sp, A, None, None, None, None, None) == E_NULL
    assert f(P(_pw()), A, 1, sp, A, None, A, None, None, None) == E_NULL       # act outputs: all or none
    assert f(P(_pw(layout=3)), A, 1, sp, A, None, None, None, None, None) == E_FORMAT
    assert f(P(_pw()), A, 5, sp, A, None, None, None, None, None) == E_SHAPE     # M > 4
    assert f(P(_pw(K=32768)), A, 1, _spec(K=32768, block=4096), A, None, None, None, None, None) == E_SHAPE
    assert f(P(_pw()), A, 1, _spec(K=512, block=256), A, None, None, None, None, None) == E_SPEC
    assert f(P(_pw(K=8192)), A, 1, _spec(K=8192, block=8192), A, None, None, None, None, None) == E_SPEC
    assert f(P(_pw()), A, 1, _spec(K=256, block=256, num=17, den=18), A, None, None, None, None, None) == E_SPEC
    assert f(P(_pw()), MIS, 1, sp, A, None, None, None, None, None) == E_ALIGN
    # the bf16 flag is accepted (validation reaches the alignment check); a bit above it is not
    bf = _spec(K=256, block=256, flags=qift.SPEC_BF16)
    assert f(P(_pw()), MIS, 1, bf, A, None, None, None, None, None) == E_ALIGN
    assert f(P(_pw()), A, 1, _spec(K=256, block=256, flags=1 << 17), A, None, None, None, None, None) == E_SPEC


def test_read_probe_validation(L):
    f = L.qift_hbm_read_probe
    assert f(None, 1024, A, None) == E_NULL
    assert f(A, 1024, None, None) == E_NULL
    assert f(A, 0, A, None) == E_SHAPE
    assert f(A, 1000, A, None) == E_SHAPE
    assert f(MIS, 1024, A, None) == E_ALIGN
    assert f(A, 1024, 0x10002, None) == E_ALIGN
    assert f(A, 1 << 50, A, None) == E_SHAPE     # more workgroups than a grid holds


def test_pack_validation(L):
    # the boundary's pack_w2(codes, scales, N, K, fmt, packed, out, stream); out-of-set levels are
    # QIFT_ERR_CODE (the call synchronizes to read them back), covered on the GPU
    f2, f4 = L.qift_pack_w2, L.qift_pack_w4
    assert f2(None, A, 512, 256, 0, A, None, None) == E_NULL
    assert f2(A, A, 512, 256, 0, None, None, None) == E_NULL
    assert f2(A, A, 512, 256, qift.W4_SYM, A, None, None) == E_FORMAT
    assert f2(A, A, 512, 100, 0, A, None, None) == E_SHAPE
    assert f2(A, A, 0, 256, 0, A, None, None) == E_SHAPE
    assert f2(MIS, A, 512, 256, 0, A, None, None) == E_ALIGN
    assert f2(A, MIS, 512, 256, 0, A, None, None) == E_ALIGN
    assert f4(A, A, 512, 256, None, None, None) == E_NULL
    assert f4(A, A, 512, 96, A, None, None) == E_SHAPE
    assert L.qift_status_string(E_CODE) == b"level outside the format's level set (nothing usable was packed)"


def test_device_error_api_validation(L):
    # host-side checks only: the read itself needs a GPU (covered by the GPU tests)
    assert L.qift_device_error(None, 1, None) == E_NULL
    assert L.qift_set_wait_limit(-1) == E_SHAPE
    assert L.qift_set_wait_limit(0) == OK     # back to the default


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(qift, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(qift, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        qift.lib()


def test_lut_linear_validation(L):
    f = L.qift_w2a4_lut_linear
    P = ctypes.byref
    half = lambda *v: (ctypes.c_uint16 * 4)(*[int(np.float16(x).view(np.uint16)) for x in v])
    good = half(-1.5104, -0.4528, 0.4528, 1.5104)
    lw = lambda **kw: _pw(fmt=qift.W2_LUT, K=kw.pop("K", 4096), **kw)
    assert L.qift_packed_bytes(qift.W2_LUT, 8, 4096) == 8 * 1024
    assert f(None, good, A, A, 4, A, None) == E_NULL
    assert f(P(lw()), None, A, A, 4, A, None) == E_NULL
    assert f(P(lw()), good, A, None, 4, A, None) == E_NULL
    assert f(P(_pw(fmt=qift.W2_MNZ, K=4096)), good, A, A, 4, A, None) == E_FORMAT   # integer formats: no table
    assert f(P(lw(K=4160)), good, A, A, 4, A, None) == E_SHAPE                     # K not a multiple of 256
    assert f(P(lw(K=16640)), good, A, A, 4, A, None) == E_SHAPE                    # K above 16384
    assert f(P(lw()), good, A, A, 0, A, None) == E_SHAPE
    assert f(P(lw()), half(0, 1, 2, 257), A, A, 4, A, None) == E_SPEC             # above 256
    assert f(P(lw()), half(0, 1, 2, np.inf), A, A, 4, A, None) == E_SPEC
    assert f(P(lw()), half(0, 1, np.nan, 2), A, A, 4, A, None) == E_SPEC
    assert f(P(lw()), good, A, A, 4, MIS, None) == E_ALIGN
    # the integer linears refuse the table format
    assert L.qift_w2a4_linear(P(lw()), A, A, 4, A, None) == E_FORMAT
