"""Pins of the KV4 oracle (asymmetric 4-bit cache quantizer, Sec. 3.3 Eq. (15) with the Sec. 4.1
setting, and decode attention over the reconstructed cache) against hand cases, brute force and
closed forms."""
import numpy as np

from oracle import kv4


def test_hand_case():
    # x in [-1, 2]: range [-0.95, 1.9], s = 2.85 / 15 = 0.19, z = round(0.95 / 0.19) = 5
    x = np.zeros(8, dtype=np.float16)
    x[0], x[3], x[7] = -1.0, 0.5, 2.0
    q, s, z = kv4.kv4_quant(x)
    assert int(z) == 5
    assert abs(float(s) - 0.19) < 1e-7
    # -1 -> -5.26 -> -5 + 5 = 0; 0 -> 5; 0.5 -> 2.63 -> 3 + 5 = 8; 2 -> 10.5 -> 11 + 5 = 16 -> 15
    assert q.tolist() == [0, 5, 5, 8, 5, 5, 5, 15]


def test_zero_group_and_exact_zero():
    q, s, z = kv4.kv4_quant(np.zeros((3, 128), dtype=np.float16))
    assert (q == 0).all() and (s == 1.0).all() and (z == 0).all()
    assert (kv4.kv4_dequant(q, s, z) == 0).all()
    rng = np.random.default_rng(1)
    x = rng.normal(0, 1, (64, 128)).astype(np.float16)
    x[:, ::7] = 0
    q, s, z = kv4.kv4_quant(x)
    assert (q[:, ::7] == z[:, None]).all()
    assert (kv4.kv4_dequant(q, s, z)[:, ::7] == 0).all()


def test_codes_are_nearest_grid_points_off_ties():
    rng = np.random.default_rng(2)
    x = (rng.standard_t(4, (256, 128)) * rng.uniform(0.01, 5, (256, 1))).astype(np.float16)
    q, s, z = kv4.kv4_quant(x)
    xf = x.astype(np.float64)
    grid = s.astype(np.float64)[:, None] * (np.arange(16)[None, :] - z.astype(np.float64)[:, None])   # [G, 16]
    dist = np.abs(xf[:, :, None] - grid[:, None, :])
    best = dist.argmin(axis=-1)
    srt = np.sort(dist, axis=-1)
    clear = (srt[..., 1] - srt[..., 0]) > 1e-5 * s.astype(np.float64)[:, None]   # not within rounding of a tie
    assert clear.mean() > 0.99
    assert np.array_equal(q[clear], best[clear])


def test_saturation_and_monotone():
    x = np.linspace(-3, 5, 128).astype(np.float16)
    q, s, z = kv4.kv4_quant(x)
    assert (np.diff(q.astype(int)) >= 0).all()
    assert q[0] == 0 and q[-1] == 15          # the clipped ends saturate
    assert 0 <= int(z) <= 15
    # the step: 0.95 of the range (which contains 0) over 15 levels
    assert abs(float(s) - 0.95 * 8.0 / 15) < 1e-6


def test_pack_nibbles():
    c = np.arange(16, dtype=np.uint8).reshape(1, 16)
    assert kv4.pack_nibbles(c).tolist() == [[0x10, 0x32, 0x54, 0x76, 0x98, 0xBA, 0xDC, 0xFE]]


def test_attention_closed_forms():
    rng = np.random.default_rng(3)
    B, T, Hkv, G, d = 2, 5, 2, 4, 16
    K = rng.normal(0, 1, (B, T, Hkv, d))
    V = rng.normal(0, 1, (B, T, Hkv, d))
    # one cached token: every head returns it
    q = rng.normal(0, 1, (B, Hkv * G, d))
    out = kv4.attention_decode(q, K[:, :1], V[:, :1])
    for h in range(Hkv * G):
        assert np.allclose(out[:, h], V[:, 0, h // G], atol=0, rtol=1e-15)
    # zero query: uniform weights, the mean of the values
    out = kv4.attention_decode(np.zeros((B, Hkv * G, d)), K, V)
    for h in range(Hkv * G):
        assert np.allclose(out[:, h], V[:, :, h // G].mean(axis=1), rtol=1e-13, atol=1e-15)
    # equal queries in one group give equal outputs; the group's KV head decides
    q = np.repeat(rng.normal(0, 1, (B, Hkv, 1, d)), G, axis=2).reshape(B, Hkv * G, d)
    out = kv4.attention_decode(q, K, V)
    assert np.array_equal(out[:, 0], out[:, G - 1])
    # a query far along one cached key selects that token's value
    q = np.zeros((B, Hkv * G, d))
    q[:, :G] = 200.0 * K[:, 3, 0][:, None, :] / np.linalg.norm(K[:, 3, 0], axis=-1)[:, None, None]
    out = kv4.attention_decode(q, K, V)
    assert np.allclose(out[:, :G], V[:, 3, 0][:, None, :], atol=1e-9)
