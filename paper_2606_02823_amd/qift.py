"""Python binding of libqift (ctypes): argument marshalling only.

Every function here checks tensor dtypes, shapes and devices, passes raw
device pointers and the current HIP stream to the C ABI declared in
``include/qift.h``, and raises on a non-zero status.  All arithmetic happens
in the library's HIP kernels; there is no fallback path.  PyTorch serves only
for device memory and streams.

Names follow the C entry points without the ``qift_`` prefix.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libqift.so")

W2_MNZ, W2_POT, W4_SYM, W2_LUT = 0, 1, 2, 3
FUSED_MAX_M = 4   # tokens per call of the fused rotate_quant_linear entry (limits in qift.h)
LAYOUT_V1 = 1

STATUS = {0: "QIFT_OK", -1: "QIFT_ERR_NULL", -2: "QIFT_ERR_SHAPE", -3: "QIFT_ERR_SPEC",
          -4: "QIFT_ERR_FORMAT", -5: "QIFT_ERR_CODE", -6: "QIFT_ERR_ALIGN", -7: "QIFT_ERR_HIP",
          -8: "QIFT_ERR_WORKSPACE"}
DEVERR_GROUP_WAIT, DEVERR_CHAIN_WAIT = 1, 2   # bits of the device error word (qift_device_error)

# every symbol declared in include/qift.h
EXPORTS = ("qift_packed_bytes", "qift_pack_w2", "qift_pack_w4", "qift_quantize_weights",
           "qift_quantize_weights_mirror", "qift_ratio_scan", "qift_kv4_quant",
           "qift_kv4_attention_workspace_bytes", "qift_kv4_attention_decode", "qift_kv4_attention_decode_noalloc", "qift_rotate_quant_act",
           "qift_rotate_quant_act_bf16",
           "qift_w2a4_linear", "qift_w2a4_linear_ex", "qift_w2a4_lut_linear", "qift_w4a4_linear", "qift_w4a4_linear_ex",
           "qift_rotate_quant_linear", "qift_hbm_read_probe", "qift_workspace_bytes", "qift_status_string",
           "qift_last_hip_error", "qift_device_error", "qift_set_wait_limit", "qift_chain_workspace_bytes",
           "qift_chain_prepare", "qift_decode_chain", "qift_version")


class QiftError(RuntimeError):
    def __init__(self, fn: str, status: int, lib):
        msg = lib.qift_status_string(status).decode()
        extra = f" (hipError {lib.qift_last_hip_error()})" if status == -7 else ""
        super().__init__(f"{fn}: {STATUS.get(status, status)}: {msg}{extra}")
        self.status = status


class PackedW(ctypes.Structure):
    _fields_ = [("fmt", ctypes.c_int32), ("layout", ctypes.c_int32), ("N", ctypes.c_int64),
                ("K", ctypes.c_int64), ("packed", ctypes.c_void_p), ("scales", ctypes.c_void_p)]


class HadamardSpec(ctypes.Structure):
    _fields_ = [("K", ctypes.c_int64), ("block", ctypes.c_int32), ("flags", ctypes.c_int32)]


def clip_flags(num: int, den: int) -> int:
    """The spec flags of clip ratio num/den (QIFT_CLIP; 0 for the plain absmax/7 scale)."""
    return 0 if (num, den) == (1, 1) else ((int(num) & 0xFF) << 8) | (int(den) & 0xFF)


SPEC_BF16 = 1 << 16   # QIFT_SPEC_BF16: the tokens are bf16 values


def spec(K: int, block: int, clip=(1, 1), bf16: bool = False) -> HadamardSpec:
    return HadamardSpec(K, block, clip_flags(*clip) | (SPEC_BF16 if bf16 else 0))


class ChainLinkC(ctypes.Structure):
    _fields_ = [("w", PackedW), ("block", ctypes.c_int32), ("flags", ctypes.c_int32), ("in_link", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("in_offset", ctypes.c_int64), ("out", ctypes.c_void_p),
                ("acc_out", ctypes.c_void_p)]


class ChainC(ctypes.Structure):
    _fields_ = [("fmt", ctypes.c_int32), ("n_links", ctypes.c_int32), ("M", ctypes.c_int32), ("K0", ctypes.c_int32),
                ("grid", ctypes.c_int32), ("kmax", ctypes.c_int32), ("region0", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("table", ctypes.c_void_p), ("counters", ctypes.c_void_p)]


_lib = None


def lib():
    """The loaded library; raises if it has not been built (no fallback exists)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_02823_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    pw = ctypes.POINTER(PackedW)
    sig = {
        "qift_packed_bytes": (sz, [i32, i64, i64]),
        "qift_pack_w2": (ctypes.c_int, [vp, vp, i64, i64, i32, vp, pw, vp]),
        "qift_pack_w4": (ctypes.c_int, [vp, vp, i64, i64, vp, pw, vp]),
        "qift_quantize_weights": (ctypes.c_int, [vp, i64, HadamardSpec, i32, vp, vp, vp]),
        "qift_quantize_weights_mirror": (ctypes.c_int, [vp, i64, HadamardSpec, ctypes.c_double, vp, vp, vp]),
        "qift_ratio_scan": (ctypes.c_int, [vp, i64, vp, i32, vp, i32, vp, vp, vp, vp, vp]),
        "qift_kv4_quant": (ctypes.c_int, [vp, i64, i32, vp, vp, vp, vp]),
        "qift_kv4_attention_workspace_bytes": (sz, [i64, i32, i32, i32, i64]),
        "qift_kv4_attention_decode": (ctypes.c_int, [vp, i64, i32, i32, i32, i64, i32, vp, vp, vp, vp, vp, vp, vp, vp, sz,
                                                     vp]),
        "qift_kv4_attention_decode_noalloc": (ctypes.c_int, [vp, i64, i32, i32, i32, i64, i32, vp, vp, vp, vp, vp, vp,
                                                             vp, vp]),
        "qift_rotate_quant_act": (ctypes.c_int, [vp, i64, HadamardSpec, vp, vp, vp, vp]),
        "qift_rotate_quant_act_bf16": (ctypes.c_int, [vp, i64, HadamardSpec, vp, vp, vp, vp]),
        "qift_w2a4_linear": (ctypes.c_int, [pw, vp, vp, i64, vp, vp]),
        "qift_w2a4_lut_linear": (ctypes.c_int, [pw, vp, vp, vp, i64, vp, vp]),
        "qift_w2a4_linear_ex": (ctypes.c_int, [pw, vp, vp, vp, i64, vp, vp, vp, sz, vp]),
        "qift_w4a4_linear": (ctypes.c_int, [pw, vp, vp, i64, vp, vp]),
        "qift_w4a4_linear_ex": (ctypes.c_int, [pw, vp, vp, vp, i64, vp, vp, vp, sz, vp]),
        "qift_rotate_quant_linear": (ctypes.c_int, [pw, vp, i64, HadamardSpec, vp, vp, vp, vp, vp, vp]),
        "qift_hbm_read_probe": (ctypes.c_int, [vp, sz, vp, vp]),
        "qift_workspace_bytes": (sz, [pw, i64]),
        "qift_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "qift_last_hip_error": (ctypes.c_int, []),
        "qift_device_error": (ctypes.c_int, [ctypes.POINTER(ctypes.c_uint32), i32, vp]),
        "qift_set_wait_limit": (ctypes.c_int, [i32]),
        "qift_chain_workspace_bytes": (sz, [ctypes.POINTER(ChainLinkC), i32, i64]),
        "qift_chain_prepare": (ctypes.c_int, [ctypes.POINTER(ChainLinkC), i32, i64, i64, vp, sz, ctypes.POINTER(ChainC),
                                              vp]),
        "qift_decode_chain": (ctypes.c_int, [ctypes.POINTER(ChainC), vp, vp]),
        "qift_version": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype, f.argtypes = res, args
    _lib = L
    return L


def _check(fn: str, status: int):
    if status != 0:
        raise QiftError(fn, status, lib())


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _dev(t: torch.Tensor, dtype, shape, name):
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _fp16_bits(t: torch.Tensor) -> torch.Tensor:
    return t.view(torch.int16) if t.dtype == torch.float16 else t


@dataclass
class Packed:
    """A packed weight matrix: the C view plus the tensors that own its memory."""
    fmt: int
    N: int
    K: int
    words: torch.Tensor   # uint32 words as int32 [N, K/16] or [N, K/8]
    scales: torch.Tensor  # fp16 [N]

    def cview(self) -> PackedW:
        return PackedW(self.fmt, LAYOUT_V1, self.N, self.K, self.words.data_ptr(), self.scales.data_ptr())

    @property
    def nbytes(self) -> int:
        return self.words.numel() * 4


def packed_bytes(fmt: int, N: int, K: int) -> int:
    return int(lib().qift_packed_bytes(fmt, N, K))


def workspace_bytes(w: Packed, M: int) -> int:
    v = w.cview()
    return int(lib().qift_workspace_bytes(ctypes.byref(v), M))


def pack_w2(levels: torch.Tensor, scales: torch.Tensor, fmt: int = W2_MNZ, out: torch.Tensor | None = None,
            stream=None) -> Packed:
    """Pack int8 levels [N, K] ({-3,-1,1,3} MNZ or {-4,-1,1,4} PoT; for W2_LUT the codes 0..3) into
    QW2v1 words.  The call validates every level and synchronizes the stream; a level outside the
    set raises QiftError with status QIFT_ERR_CODE."""
    N, K = levels.shape
    _dev(levels, torch.int8, (N, K), "levels")
    _dev(scales, torch.float16, (N,), "scales")
    if out is None:
        out = torch.empty((N, K // 16), dtype=torch.int32, device=levels.device)
    _dev(out, torch.int32, (N, K // 16), "out")
    st = lib().qift_pack_w2(levels.data_ptr(), scales.data_ptr(), N, K, fmt, out.data_ptr(), None, _stream(stream))
    _check("qift_pack_w2", st)
    return Packed(fmt, N, K, out, scales)


def pack_w4(levels: torch.Tensor, scales: torch.Tensor, out: torch.Tensor | None = None, stream=None) -> Packed:
    """Pack int8 W4 levels [N, K] in -7..7 into QW4v1 words (validated like pack_w2)."""
    N, K = levels.shape
    _dev(levels, torch.int8, (N, K), "levels")
    _dev(scales, torch.float16, (N,), "scales")
    if out is None:
        out = torch.empty((N, K // 8), dtype=torch.int32, device=levels.device)
    _dev(out, torch.int32, (N, K // 8), "out")
    st = lib().qift_pack_w4(levels.data_ptr(), scales.data_ptr(), N, K, out.data_ptr(), None, _stream(stream))
    _check("qift_pack_w4", st)
    return Packed(W4_SYM, N, K, out, scales)


@dataclass
class QAct:
    """Quantized activations of M tokens: the codes and scales every linear consumes, and the per-token
    code sums (written by rotate_quant_act when present; the linears compute their own)."""
    q: torch.Tensor                 # int8 [M, K]
    scale: torch.Tensor             # fp32 [M]
    sum: torch.Tensor | None = None  # int32 [M]

    @property
    def M(self):
        return self.q.shape[0]


def alloc_act(M: int, K: int, device="cuda") -> QAct:
    return QAct(torch.empty((M, K), dtype=torch.int8, device=device),
                torch.empty(M, dtype=torch.float32, device=device),
                torch.empty(M, dtype=torch.int32, device=device))


def quantize_weights(W: torch.Tensor, block: int, fmt: int, levels: torch.Tensor | None = None,
                     scales: torch.Tensor | None = None, stream=None):
    """Rotate the rows of fp32 W [N, K] by the block Hadamard, take the format's per-row scale and the
    nearest levels (the input of pack_w2 / pack_w4).  Returns (levels int8 [N, K], scales fp16 [N])."""
    N, K = W.shape
    _dev(W, torch.float32, (N, K), "W")
    if levels is None:
        levels = torch.empty((N, K), dtype=torch.int8, device=W.device)
    if scales is None:
        scales = torch.empty(N, dtype=torch.float16, device=W.device)
    _dev(levels, torch.int8, (N, K), "levels")
    _dev(scales, torch.float16, (N,), "scales")
    st = lib().qift_quantize_weights(W.data_ptr(), N, spec(K, block), int(fmt), levels.data_ptr(),
                                     scales.data_ptr(), _stream(stream))
    _check("qift_quantize_weights", st)
    return levels, scales


def quantize_weights_mirror(W: torch.Tensor, block: int, r: float, codes: torch.Tensor | None = None,
                            scales: torch.Tensor | None = None, stream=None):
    """Rotate the rows of fp32 W [N, K], take the 64-candidate MSE scale of the set {-1, -r, +r, +1} and
    the nearest codes 0..3 (ascending levels; the input of pack_w2 with FMT_LUT).  Returns (codes int8
    [N, K], scales fp16 [N])."""
    N, K = W.shape
    _dev(W, torch.float32, (N, K), "W")
    if codes is None:
        codes = torch.empty((N, K), dtype=torch.int8, device=W.device)
    if scales is None:
        scales = torch.empty(N, dtype=torch.float16, device=W.device)
    _dev(codes, torch.int8, (N, K), "codes")
    _dev(scales, torch.float16, (N,), "scales")
    st = lib().qift_quantize_weights_mirror(W.data_ptr(), N, spec(K, block), float(r), codes.data_ptr(),
                                            scales.data_ptr(), _stream(stream))
    _check("qift_quantize_weights_mirror", st)
    return codes, scales


def ratio_scan(x: torch.Tensor, ratios, cands, stream=None):
    """Squared error of the set {-1, -r, +r, +1} on the fp64 samples x at every scale c * max|x| of the
    candidate clip ratios, for each ratio r.  Returns (sse fp64 [R, C], nmse fp64 [R], best int32 [R],
    stats fp64 [2] = (max|x|, sum x^2)), all on x's device."""
    x = x.reshape(-1)
    _dev(x, torch.float64, (x.numel(),), "x")
    r = (ctypes.c_double * len(ratios))(*[float(v) for v in ratios])
    c = (ctypes.c_double * len(cands))(*[float(v) for v in cands])
    R, C = len(ratios), len(cands)
    sse = torch.empty((R, C), dtype=torch.float64, device=x.device)
    nmse = torch.empty(R, dtype=torch.float64, device=x.device)
    best = torch.empty(R, dtype=torch.int32, device=x.device)
    stats = torch.empty(2, dtype=torch.float64, device=x.device)
    st = lib().qift_ratio_scan(x.data_ptr(), x.numel(), r, R, c, C, sse.data_ptr(), nmse.data_ptr(),
                               best.data_ptr(), stats.data_ptr(), _stream(stream))
    _check("qift_ratio_scan", st)
    return sse, nmse, best, stats


class KV4:
    """A KV4 cache tensor: codes uint8 [..., 64], scales fp32 [...], zeros uint8 [...]."""

    def __init__(self, codes: torch.Tensor, scales: torch.Tensor, zeros: torch.Tensor):
        self.codes, self.scales, self.zeros = codes, scales, zeros


def kv4_quant(x: torch.Tensor, out: KV4 | None = None, stream=None) -> KV4:
    """Asymmetric 4-bit quantization of fp16 x [..., 128], one group per trailing vector."""
    lead = tuple(x.shape[:-1])
    _dev(x, torch.float16, lead + (128,), "x")
    if out is None:
        out = KV4(torch.empty(lead + (64,), dtype=torch.uint8, device=x.device),
                  torch.empty(lead, dtype=torch.float32, device=x.device),
                  torch.empty(lead, dtype=torch.uint8, device=x.device))
    _dev(out.codes, torch.uint8, lead + (64,), "codes")
    _dev(out.scales, torch.float32, lead, "scales")
    _dev(out.zeros, torch.uint8, lead, "zeros")
    groups = x.numel() // 128
    st = lib().qift_kv4_quant(x.data_ptr(), groups, 128, out.codes.data_ptr(), out.scales.data_ptr(),
                              out.zeros.data_ptr(), _stream(stream))
    _check("qift_kv4_quant", st)
    return out


KV4_TOKEN_MAJOR, KV4_HEAD_MAJOR = 0, 1


def kv4_attention_decode(q: torch.Tensor, k: KV4, v: KV4, out=None, workspace=None, head_major=False,
                         stream=None) -> torch.Tensor:
    """One decode step of grouped-query attention: q fp16 [B, Hq, 128] over the KV4 cache k, v of
    groups [B, T, Hkv] (token-major) or, head_major, [B, Hkv, T]; returns fp16 [B, Hq, 128]."""
    B, Hq, d = q.shape
    _dev(q, torch.float16, (B, Hq, 128), "q")
    if head_major:
        Hkv, T = k.codes.shape[1], k.codes.shape[2]
        rows = (B, Hkv, T)
    else:
        T, Hkv = k.codes.shape[1], k.codes.shape[2]
        rows = (B, T, Hkv)
    for name, c in (("k", k), ("v", v)):
        _dev(c.codes, torch.uint8, rows + (64,), name + ".codes")
        _dev(c.scales, torch.float32, rows, name + ".scales")
        _dev(c.zeros, torch.uint8, rows, name + ".zeros")
    if out is None:
        out = torch.empty((B, Hq, 128), dtype=torch.float16, device=q.device)
    _dev(out, torch.float16, (B, Hq, 128), "out")
    need = int(lib().qift_kv4_attention_workspace_bytes(B, Hq, Hkv, 128, T))
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
    st = lib().qift_kv4_attention_decode(q.data_ptr(), B, Hq, Hkv, 128, T,
                                         KV4_HEAD_MAJOR if head_major else KV4_TOKEN_MAJOR,
                                         k.codes.data_ptr(), k.scales.data_ptr(),
                                         k.zeros.data_ptr(), v.codes.data_ptr(), v.scales.data_ptr(),
                                         v.zeros.data_ptr(), out.data_ptr(), workspace.data_ptr(),
                                         workspace.numel() * workspace.element_size(), _stream(stream))
    _check("qift_kv4_attention_decode", st)
    return out


KV4_SCRATCH_BYTES = 8 << 20   # QIFT_KV4_SCRATCH_BYTES


def kv4_attention_decode_noalloc(q: torch.Tensor, k: KV4, v: KV4, out: torch.Tensor, head_major=False,
                                 stream=None) -> torch.Tensor:
    """kv4_attention_decode through the entry point that allocates nothing (its partial records in the
    library's per-GPU array): out must be given, and calls that overlap on one GPU race."""
    B, Hq, d = q.shape
    _dev(q, torch.float16, (B, Hq, 128), "q")
    if head_major:
        Hkv, T = k.codes.shape[1], k.codes.shape[2]
        rows = (B, Hkv, T)
    else:
        T, Hkv = k.codes.shape[1], k.codes.shape[2]
        rows = (B, T, Hkv)
    for name, c in (("k", k), ("v", v)):
        _dev(c.codes, torch.uint8, rows + (64,), name + ".codes")
        _dev(c.scales, torch.float32, rows, name + ".scales")
        _dev(c.zeros, torch.uint8, rows, name + ".zeros")
    _dev(out, torch.float16, (B, Hq, 128), "out")
    st = lib().qift_kv4_attention_decode_noalloc(q.data_ptr(), B, Hq, Hkv, 128, T,
                                                 KV4_HEAD_MAJOR if head_major else KV4_TOKEN_MAJOR,
                                                 k.codes.data_ptr(), k.scales.data_ptr(), k.zeros.data_ptr(),
                                                 v.codes.data_ptr(), v.scales.data_ptr(), v.zeros.data_ptr(),
                                                 out.data_ptr(), _stream(stream))
    _check("qift_kv4_attention_decode_noalloc", st)
    return out


def rotate_quant_act(x: torch.Tensor, block: int, clip=(1, 1), out: QAct | None = None, stream=None) -> QAct:
    """Exact block-Hadamard rotation + per-token INT4 quantization of fp16 or bf16 x [M, K]."""
    M, K = x.shape
    bf16 = x.dtype == torch.bfloat16
    _dev(x, torch.bfloat16 if bf16 else torch.float16, (M, K), "x")
    if out is None:
        out = alloc_act(M, K, x.device)
    _dev(out.q, torch.int8, (M, K), "act_q")
    _dev(out.scale, torch.float32, (M,), "act_scale")
    if out.sum is not None:
        _dev(out.sum, torch.int32, (M,), "act_sum")
    name = "qift_rotate_quant_act_bf16" if bf16 else "qift_rotate_quant_act"
    st = getattr(lib(), name)(x.data_ptr(), M, spec(K, block, clip), out.q.data_ptr(), out.scale.data_ptr(),
                              _ptr(out.sum), _stream(stream))
    _check(name, st)
    return out


def _linear(name: str, w: Packed, act: QAct, out, acc_out, workspace, use_sum, stream):
    M, K = act.q.shape
    if K != w.K:
        raise ValueError(f"activation width {K} != weight K {w.K}")
    _dev(act.scale, torch.float32, (M,), "act_scale")
    act_sum = act.sum if use_sum else None
    if use_sum:
        _dev(act_sum, torch.int32, (M,), "act_sum")
    if out is None:
        out = torch.empty((M, w.N), dtype=torch.float16, device=act.q.device)
    _dev(out, torch.float16, (M, w.N), "out")
    if acc_out is not None:
        _dev(acc_out, torch.int32, (M, w.N), "acc_out")
    v = w.cview()
    L = lib()
    if workspace is not None:
        _dev(workspace, torch.uint8, (workspace.numel(),), "workspace")
    if acc_out is None and workspace is None and act_sum is None:
        st = getattr(L, name)(ctypes.byref(v), act.q.data_ptr(), act.scale.data_ptr(), M, out.data_ptr(),
                              _stream(stream))
    else:
        ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
        st = getattr(L, name + "_ex")(ctypes.byref(v), act.q.data_ptr(), act.scale.data_ptr(),
                                      _ptr(act_sum), M, out.data_ptr(), _ptr(acc_out),
                                      _ptr(workspace), ws_bytes, _stream(stream))
    _check(name, st)
    return out


def w2a4_linear(w: Packed, act: QAct, out=None, acc_out=None, workspace=None, use_sum=False,
                stream=None) -> torch.Tensor:
    """fp16 y [M, N] of the 2-bit quantized linear (MNZ or PoT weights).  With acc_out, workspace or
    use_sum (pass act.sum as the precomputed code sums) the call goes through qift_w2a4_linear_ex."""
    return _linear("qift_w2a4_linear", w, act, out, acc_out, workspace, use_sum, stream)


def w2a4_lut_linear(w: Packed, lut, act: QAct, out=None, stream=None) -> torch.Tensor:
    """fp16 y [M, N] of the linear over a four-level table (W2_LUT code words); ``lut`` is the four
    levels (any sequence of numbers, rounded once to fp16, or an fp16 tensor)."""
    M, K = act.q.shape
    if K != w.K:
        raise ValueError(f"activation width {K} != weight K {w.K}")
    _dev(act.scale, torch.float32, (M,), "act_scale")
    if out is None:
        out = torch.empty((M, w.N), dtype=torch.float16, device=act.q.device)
    _dev(out, torch.float16, (M, w.N), "out")
    bits = torch.as_tensor(lut, dtype=torch.float64).to(torch.float16).cpu().contiguous().view(torch.int16)
    if bits.shape != (4,):
        raise ValueError("lut must hold four levels")
    table = (ctypes.c_uint16 * 4)(*[int(b) & 0xFFFF for b in bits.tolist()])
    v = w.cview()
    st = lib().qift_w2a4_lut_linear(ctypes.byref(v), table, act.q.data_ptr(), act.scale.data_ptr(), M,
                                    out.data_ptr(), _stream(stream))
    _check("qift_w2a4_lut_linear", st)
    return out


def w4a4_linear(w: Packed, act: QAct, out=None, acc_out=None, workspace=None, use_sum=False,
                stream=None) -> torch.Tensor:
    """fp16 y [M, N] of the W4 sibling."""
    return _linear("qift_w4a4_linear", w, act, out, acc_out, workspace, use_sum, stream)


def linear(w: Packed, act: QAct, out=None, acc_out=None, workspace=None, use_sum=False, stream=None) -> torch.Tensor:
    """Dispatch on the weight format."""
    f = w4a4_linear if w.fmt == W4_SYM else w2a4_linear
    return f(w, act, out=out, acc_out=acc_out, workspace=workspace, use_sum=use_sum, stream=stream)


def rotate_quant_linear(w: Packed, x: torch.Tensor, block: int, clip=(1, 1), out=None, acc_out=None,
                        act_out: QAct | None = None, stream=None) -> torch.Tensor:
    """Fused rotate_quant_act + linear for M <= 4 fp16 or bf16 tokens [M, K]; optional act_out receives the
    act triple."""
    M, K = x.shape
    bf16 = x.dtype == torch.bfloat16
    _dev(x, torch.bfloat16 if bf16 else torch.float16, (M, K), "x")
    if K != w.K:
        raise ValueError(f"activation width {K} != weight K {w.K}")
    if out is None:
        out = torch.empty((M, w.N), dtype=torch.float16, device=x.device)
    _dev(out, torch.float16, (M, w.N), "out")
    if acc_out is not None:
        _dev(acc_out, torch.int32, (M, w.N), "acc_out")
    if act_out is not None:
        _dev(act_out.q, torch.int8, (M, K), "act_q")
        _dev(act_out.scale, torch.float32, (M,), "act_scale")
        _dev(act_out.sum, torch.int32, (M,), "act_sum")
    v = w.cview()
    st = lib().qift_rotate_quant_linear(
        ctypes.byref(v), x.data_ptr(), M, spec(K, block, clip, bf16), out.data_ptr(), _ptr(acc_out),
        None if act_out is None else act_out.q.data_ptr(), None if act_out is None else act_out.scale.data_ptr(),
        None if act_out is None else act_out.sum.data_ptr(), _stream(stream))
    _check("qift_rotate_quant_linear", st)
    return out


@dataclass
class ChainLink:
    """One linear of a decode chain: weights, the Hadamard block (and clip) of its input, and where the
    input comes from (in_link = -1: the chain input; else elements [in_offset, in_offset + K) of that
    link's output rows)."""
    w: Packed
    block: int
    in_link: int = -1
    in_offset: int = 0
    clip: tuple = (1, 1)


class Chain:
    """A prepared decode chain (qift_chain_prepare): its workspace, the output buffer of every link and,
    with acc=True, the int32 accumulators.  run(x) performs one decode step (one kernel launch)."""

    def __init__(self, links, M: int, acc: bool = False, device="cuda", stream=None):
        self.links = list(links)
        self.M = M
        self.K0 = self.links[0].w.K
        self.outs = [torch.empty((M, l.w.N), dtype=torch.float16, device=device) for l in self.links]
        self.accs = [torch.empty((M, l.w.N), dtype=torch.int32, device=device) for l in self.links] if acc else None
        n = len(self.links)
        arr = (ChainLinkC * n)()
        for i, l in enumerate(self.links):
            arr[i] = ChainLinkC(l.w.cview(), l.block, clip_flags(*l.clip), l.in_link, 0, l.in_offset,
                                self.outs[i].data_ptr(), None if acc is False else self.accs[i].data_ptr())
        nbytes = int(lib().qift_chain_workspace_bytes(arr, n, M))
        self.workspace = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=device)
        self.c = ChainC()
        _check("qift_chain_prepare", lib().qift_chain_prepare(arr, n, M, self.K0, self.workspace.data_ptr(), nbytes,
                                                               ctypes.byref(self.c), _stream(stream)))

    def run(self, x: torch.Tensor, stream=None):
        _dev(x, torch.float16, (self.M, self.K0), "x")
        _check("qift_decode_chain", lib().qift_decode_chain(ctypes.byref(self.c), x.data_ptr(), _stream(stream)))
        return self.outs


READ_PROBE_SEGMENT = 65536   # bytes read by one workgroup of the read probe


def read_probe_slots(nbytes: int) -> int:
    return -(-nbytes // READ_PROBE_SEGMENT)


def hbm_read_probe(buf: torch.Tensor, partials: torch.Tensor, stream=None) -> torch.Tensor:
    """Read buf once on the GPU; partials[b] (int32, read_probe_slots(buf bytes) entries) receives the XOR
    of the 32-bit words of the b-th 64 KiB segment.  A measurement helper (achievable HBM read bandwidth),
    not part of the method."""
    if not isinstance(buf, torch.Tensor) or buf.device.type != "cuda" or not buf.is_contiguous():
        raise TypeError("buf must be a contiguous CUDA (HIP) tensor")
    nbytes = buf.numel() * buf.element_size()
    _dev(partials, torch.int32, (read_probe_slots(nbytes),), "partials")
    _check("qift_hbm_read_probe", lib().qift_hbm_read_probe(buf.data_ptr(), nbytes, partials.data_ptr(),
                                                            _stream(stream)))
    return partials


def device_error(clear: bool = True, stream=None) -> int:
    """Synchronize the stream and return the device error word (DEVERR_* bits; 0 when every bounded
    wait of the kernels since the last clear ended normally); clear it by default."""
    bits = ctypes.c_uint32(0)
    _check("qift_device_error", lib().qift_device_error(ctypes.byref(bits), 1 if clear else 0, _stream(stream)))
    return int(bits.value)


def set_wait_limit(spins: int) -> None:
    """Test hook: spin limit of the in-workgroup wave barriers for later launches (0: the default)."""
    _check("qift_set_wait_limit", lib().qift_set_wait_limit(int(spins)))


def version() -> str:
    return lib().qift_version().decode()
