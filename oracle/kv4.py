"""KV4: asymmetric 4-bit key/value cache quantization and decode attention over that cache.

Test infrastructure: a plain CPU statement of what the GPU path computes (only tests and the
benchmark's CPU leg use it).

The paper's pipeline quantizes the KV cache to four bits, asymmetrically, with clipping ratio 0.95
for keys and for values (Sec. 4.1 "Quantization configuration"), using the conventional
asymmetric quantizer q = clip(round(w / s) + z, 0, 2^b - 1) with reconstruction w_hat = s (q - z)
(Sec. 3.3 Eq. (15)); decode throughput is bounded by moving weights and this cache (Sec. 1).
Readings, where the paper fixes nothing:

* one quantization group per token and KV head: the head_dim values of one key or value vector;
* the range contains zero and is clipped: x_max = c * max(max_i x_i, 0), x_min = c * min(min_i x_i,
  0) with c = fp32(0.95); s = (x_max - x_min) / 15; z = round(-x_min / s); a group of zeros takes
  s = 1, z = 0 (all codes 0, reconstruction 0);
* every step in IEEE fp32 in the order written, rounding half to even: the codes are integers
  decided by floating point, so the GPU and this oracle decide them in the same precision;
* decode attention for query head h uses KV head h // (Hq / Hkv) (grouped queries): softmax over
  the cached tokens of q . k_hat / sqrt(d), applied to v_hat; reference arithmetic in fp64 on the
  fp32 reconstructions.
"""
from __future__ import annotations

import numpy as np

from . import quant

CLIP = np.float32(0.95)
LEVELS = 15   # 2^4 - 1


def kv4_quant(x: np.ndarray):
    """Quantize fp16 groups x [..., d].  Returns (codes uint8 [..., d] in 0..15, s fp32 [...], z uint8 [...])."""
    x = np.asarray(x, dtype=np.float16).astype(np.float32)
    f32 = np.float32
    x_max = np.maximum(x.max(axis=-1), f32(0.0)) * CLIP
    x_min = np.minimum(x.min(axis=-1), f32(0.0)) * CLIP
    s = (x_max - x_min) / f32(LEVELS)
    s = np.where(s == 0.0, f32(1.0), s).astype(np.float32)
    z = np.clip(quant.rne(-x_min / s), 0, LEVELS)
    q = np.clip(quant.rne(x / s[..., None]) + z[..., None], 0, LEVELS)
    assert s.dtype == np.float32 and (x / s[..., None]).dtype == np.float32
    return q.astype(np.uint8), s, z.astype(np.uint8)


def kv4_dequant(codes: np.ndarray, s: np.ndarray, z: np.ndarray) -> np.ndarray:
    """fp32 reconstruction s (q - z) of every value (Eq. (15))."""
    d = np.asarray(codes, dtype=np.float32) - np.asarray(z, dtype=np.float32)[..., None]
    return (np.asarray(s, dtype=np.float32)[..., None] * d).astype(np.float32)


def pack_nibbles(codes: np.ndarray) -> np.ndarray:
    """Codes [..., d] -> bytes [..., d / 2]: value 2i in the low nibble of byte i, 2i + 1 in the high."""
    c = np.asarray(codes, dtype=np.uint8)
    return (c[..., 0::2] | (c[..., 1::2] << 4)).astype(np.uint8)


def attention_decode(q: np.ndarray, k_hat: np.ndarray, v_hat: np.ndarray) -> np.ndarray:
    """One decode step of attention over a cache.

    q [B, Hq, d] (query of the new token), k_hat, v_hat [B, T, Hkv, d] (the reconstructed cache).
    Returns fp64 [B, Hq, d]: for head h, softmax_t(q_h . k_hat[t, h // (Hq / Hkv)] / sqrt(d)) applied
    to v_hat[:, h // (Hq / Hkv)].
    """
    q = np.asarray(q, dtype=np.float64)
    K = np.asarray(k_hat, dtype=np.float64)
    V = np.asarray(v_hat, dtype=np.float64)
    B, Hq, d = q.shape
    Hkv = K.shape[2]
    G = Hq // Hkv
    out = np.empty((B, Hq, d))
    for b in range(B):
        for h in range(Hq):
            kv = h // G
            scores = K[b, :, kv, :] @ q[b, h] / np.sqrt(float(d))
            p = np.exp(scores - scores.max())
            out[b, h] = (p / p.sum()) @ V[b, :, kv, :]
    return out
