"""GPU KV4 cache (qift_kv4_quant) and decode attention over it (qift_kv4_attention_decode) against
the oracle, through the C ABI.

The quantizer's codes, fp32 scales and zero-points must equal the oracle's bit for bit (both decide
in fp32, in the same order).  The attention output is fp16 from fp32 arithmetic; it is compared
with the oracle's fp64 softmax over the reconstructed cache, per query head, relative to the head's
largest output, against a tolerance derived from the arithmetic: the fp16 rounding of the output
(at most 2^-11 of |y| <= max |ref|), plus the fp32 scores and sums (exact operands: code - z and
the fp16 queries; p s split into two fp16 parts, 2^-21 relative) and the value sums of the f16
MFMA over subnormal code operands (about 1e-6 of sum |p s code|, which is at most 15 max s / max
|ref| ~ 100 times the output on these inputs): 2^-11 + 1.1e-4.
"""
import numpy as np
import pytest
import torch

from oracle import kv4 as okv4

pytestmark = pytest.mark.gpu

TOL = 2.0 ** -11 + 1.1e-4


@pytest.fixture(scope="module")
def Q():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_02823_amd import qift
    qift.lib()
    return qift


def groups_fp16(rng, n):
    x = rng.normal(0, 1, (n, 128))
    x[::5] *= rng.uniform(0.001, 30, (x[::5].shape[0], 1))
    x[1::7] = np.abs(x[1::7])            # all non-negative
    x[2::7] = -np.abs(x[2::7])           # all non-positive
    x[3::11] = 0.0                        # groups of zeros
    x[4::13] *= 1e-6                      # tiny (fp16 subnormals)
    x[5::17, 3] = 900.0                   # one outlier
    return x.astype(np.float16)


def unpack(codes):
    c = codes.astype(np.uint8)
    out = np.empty(c.shape[:-1] + (2 * c.shape[-1],), dtype=np.uint8)
    out[..., 0::2] = c & 15
    out[..., 1::2] = c >> 4
    return out


def test_kv4_quant_bitexact(Q):
    rng = np.random.default_rng(11)
    x = groups_fp16(rng, 3001)
    c = Q.kv4_quant(torch.from_numpy(x).cuda())
    torch.cuda.synchronize()
    q_ref, s_ref, z_ref = okv4.kv4_quant(x)
    assert np.array_equal(c.scales.cpu().numpy().view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(c.zeros.cpu().numpy(), z_ref)
    assert np.array_equal(unpack(c.codes.cpu().numpy()), q_ref)
    assert np.array_equal(c.codes.cpu().numpy(), okv4.pack_nibbles(q_ref))


def test_kv4_quant_one_token_into_a_cache_view(Q):
    # one decode step appends token t of a token-major [B, T, Hkv] cache: its zero-points start at
    # byte (b T + t) Hkv, 8-byte but not 16-byte aligned for odd t with Hkv = 8
    B, T, Hkv = 2, 5, 8
    rng = np.random.default_rng(5)
    cache = Q.KV4(torch.zeros((B, T, Hkv, 64), dtype=torch.uint8, device="cuda"),
                  torch.zeros((B, T, Hkv), dtype=torch.float32, device="cuda"),
                  torch.zeros((B, T, Hkv), dtype=torch.uint8, device="cuda"))
    misaligned = 0
    for b, t in ((0, 3), (1, 1), (1, 4)):
        x = groups_fp16(rng, Hkv)
        view = Q.KV4(cache.codes[b, t], cache.scales[b, t], cache.zeros[b, t])
        misaligned += view.zeros.data_ptr() % 16 != 0
        Q.kv4_quant(torch.from_numpy(x).cuda(), out=view)
        torch.cuda.synchronize()
        q_ref, s_ref, z_ref = okv4.kv4_quant(x)
        assert np.array_equal(cache.scales[b, t].cpu().numpy().view(np.uint32), s_ref.view(np.uint32))
        assert np.array_equal(cache.zeros[b, t].cpu().numpy(), z_ref)
        assert np.array_equal(cache.codes[b, t].cpu().numpy(), okv4.pack_nibbles(q_ref))
    assert misaligned >= 1   # (b T + t) Hkv = 24 and 72 bytes: not 16-byte aligned
    # the other rows are untouched
    assert int(cache.zeros[0, 0].sum().item()) == 0 and float(cache.scales[1, 0].abs().sum().item()) == 0.0


@pytest.mark.parametrize("head_major", [False, True], ids=["token_major", "head_major"])
@pytest.mark.parametrize("B,T,Hq,Hkv", [(1, 1, 32, 8), (2, 255, 32, 8), (1, 256, 32, 8), (2, 257, 16, 8),
                                        (1, 1000, 8, 8), (1, 4100, 64, 8), (3, 700, 32, 8), (2, 513, 4, 2),
                                        (4, 2100, 32, 8), (2, 4500, 16, 8), (1, 10000, 32, 8),
                                        (1, 8300, 32, 8), (2, 33000, 8, 2), (1, 140000, 8, 1),
                                        (1, 9000, 8, 8), (2, 9000, 16, 8)])
def test_kv4_attention_decode(Q, B, T, Hq, Hkv, head_major):
    rng = np.random.default_rng(B * 100003 + T)
    K = groups_fp16(rng, B * T * Hkv).reshape(B, T, Hkv, 128)
    V = rng.normal(0, 1, (B, T, Hkv, 128)).astype(np.float16)
    q = (rng.normal(0, 1, (B, Hq, 128)) * rng.uniform(0.2, 3, (B, Hq, 1))).astype(np.float16)
    # the cache rows in the chosen order: [B, T, Hkv] or [B, Hkv, T]
    rows = (lambda a: np.ascontiguousarray(a.transpose(0, 2, 1, 3))) if head_major else (lambda a: a)
    k = Q.kv4_quant(torch.from_numpy(rows(K)).cuda())
    v = Q.kv4_quant(torch.from_numpy(rows(V)).cuda())
    y = Q.kv4_attention_decode(torch.from_numpy(q).cuda(), k, v, head_major=head_major)
    torch.cuda.synchronize()
    kq, ks, kz = okv4.kv4_quant(K)
    vq, vs, vz = okv4.kv4_quant(V)
    assert np.array_equal(unpack(k.codes.cpu().numpy()), rows(kq))
    assert np.array_equal(unpack(v.codes.cpu().numpy()), rows(vq))
    ref = okv4.attention_decode(q, okv4.kv4_dequant(kq, ks, kz), okv4.kv4_dequant(vq, vs, vz))
    got = y.cpu().numpy().astype(np.float64)
    err = np.abs(got - ref).max(axis=-1) / np.abs(ref).max(axis=-1)
    print(f"B={B} T={T} Hq={Hq} Hkv={Hkv} head_major={head_major}: max rel err {err.max():.2e}")
    assert err.max() <= TOL, err.max()


@pytest.mark.parametrize("head_major", [False, True], ids=["token_major", "head_major"])
def test_kv4_attention_sharp_softmax(Q, head_major):
    """Large queries over keys with outliers: scores in the hundreds, a few near-tied tokens share the
    softmax, so any loss of precision in the scores shows in the output."""
    rng = np.random.default_rng(77)
    B, T, Hq, Hkv = 2, 900, 32, 8
    K = groups_fp16(rng, B * T * Hkv).reshape(B, T, Hkv, 128)
    V = rng.normal(0, 1, (B, T, Hkv, 128)).astype(np.float16)
    q = (rng.normal(0, 1, (B, Hq, 128)) * rng.uniform(5, 20, (B, Hq, 1))).astype(np.float16)
    rows = (lambda a: np.ascontiguousarray(a.transpose(0, 2, 1, 3))) if head_major else (lambda a: a)
    k = Q.kv4_quant(torch.from_numpy(rows(K)).cuda())
    v = Q.kv4_quant(torch.from_numpy(rows(V)).cuda())
    y = Q.kv4_attention_decode(torch.from_numpy(q).cuda(), k, v, head_major=head_major)
    torch.cuda.synchronize()
    kq, ks, kz = okv4.kv4_quant(K)
    vq, vs, vz = okv4.kv4_quant(V)
    Kh = okv4.kv4_dequant(kq, ks, kz)
    ref = okv4.attention_decode(q, Kh, okv4.kv4_dequant(vq, vs, vz))
    # the case is sharp: the largest scores reach the hundreds
    scores = np.einsum("bhd,bthd->bht", q.astype(np.float64).reshape(B, Hkv, Hq // Hkv, 128).mean(2),
                       Kh.astype(np.float64)) / np.sqrt(128.0)
    assert np.abs(scores).max() > 100
    err = np.abs(y.cpu().numpy().astype(np.float64) - ref).max(axis=-1) / np.abs(ref).max(axis=-1)
    print(f"sharp softmax head_major={head_major}: max rel err {err.max():.2e}")
    assert err.max() <= TOL, err.max()


@pytest.mark.parametrize("B,T,sample", [(16, 4096, (0, 9, 15)), (1, 32768, (0,))], ids=["B16-T4096", "B1-T32768"])
def test_kv4_attention_bench_sizes(Q, B, T, sample):
    """The benchmarked configurations (Hq 32, Hkv 8, head-major cache, the launch the bench times): the
    whole batch runs on the GPU, the oracle checks the sampled sequences, every query head."""
    Hq, Hkv = 32, 8
    rng = np.random.default_rng(B * 7 + T)
    K = rng.normal(0, 1, (B, Hkv, T, 128)).astype(np.float16)      # head-major rows
    V = rng.normal(0, 1, (B, Hkv, T, 128)).astype(np.float16)
    q = (rng.normal(0, 1, (B, Hq, 128)) * rng.uniform(0.2, 3, (B, Hq, 1))).astype(np.float16)
    k = Q.kv4_quant(torch.from_numpy(K).cuda())
    v = Q.kv4_quant(torch.from_numpy(V).cuda())
    y = Q.kv4_attention_decode(torch.from_numpy(q).cuda(), k, v, head_major=True).cpu().numpy().astype(np.float64)
    for b in sample:
        Kt = K[b:b + 1].transpose(0, 2, 1, 3)                     # [1, T, Hkv, 128]
        Vt = V[b:b + 1].transpose(0, 2, 1, 3)
        kq, ks, kz = okv4.kv4_quant(Kt)
        vq, vs, vz = okv4.kv4_quant(Vt)
        ref = okv4.attention_decode(q[b:b + 1], okv4.kv4_dequant(kq, ks, kz), okv4.kv4_dequant(vq, vs, vz))
        err = np.abs(y[b:b + 1] - ref).max(axis=-1) / np.abs(ref).max(axis=-1)
        print(f"B={B} T={T} b={b}: max rel err {err.max():.2e}")
        assert err.max() <= TOL, (b, err.max())


def test_kv4_quant_exact_half_quotients(Q):
    """Groups whose values sit exactly on x = (k + 1/2) s (found by searching fp16 ranges whose fp32
    step s makes those products fp16 values): every code is decided at a tie, where the GPU's
    fast path must hand over to the division."""
    c32 = np.float32(0.95)
    groups = []
    for bits in range(0x3C00, 0x5000):                 # x_max in [1, 32)
        x_max = np.uint16(bits).view(np.float16)
        s = np.float32(np.float32(np.float32(x_max) * c32) / np.float32(15))
        ties = [np.float32((k + 0.5) * np.float64(s)) for k in range(0, 15)]
        exact = [t for t in ties if float(np.float16(t)) == float(t) and 0 < t < float(x_max)]
        if len(exact) >= 3:
            g = np.zeros(128, dtype=np.float16)
            g[0] = x_max
            vals = np.array(exact, dtype=np.float16)
            g[1:] = np.resize(vals, 127)
            groups.append(g)
        if len(groups) >= 64:
            break
    assert len(groups) >= 8, len(groups)
    x = np.stack(groups)
    c = Q.kv4_quant(torch.from_numpy(x).cuda())
    torch.cuda.synchronize()
    q_ref, s_ref, z_ref = okv4.kv4_quant(x)
    t = x.astype(np.float32) / s_ref[:, None]
    assert np.mean(t[:, 1:] == np.round(t[:, 1:] - 0.5) + 0.5) > 0.9      # the quotients are half-integers
    assert np.array_equal(c.scales.cpu().numpy().view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(unpack(c.codes.cpu().numpy()), q_ref)


def test_kv4_attention_workspace_reuse(Q):
    """One workspace serves consecutive calls of different T and B (the partials of one call never
    leak into the next): every call, repeated, matches the oracle."""
    Hq, Hkv = 32, 8
    cases = [(2, 3000), (1, 300), (2, 5000), (1, 1), (2, 256), (1, 4097)]
    need = max(int(Q.lib().qift_kv4_attention_workspace_bytes(B, Hq, Hkv, 128, T)) for B, T in cases)
    ws = torch.full((need,), 0xFF, dtype=torch.uint8, device="cuda")   # stale contents
    for B, T in cases:
        rng = np.random.default_rng(B * 31 + T)
        K = groups_fp16(rng, B * T * Hkv).reshape(B, T, Hkv, 128)
        V = rng.normal(0, 1, (B, T, Hkv, 128)).astype(np.float16)
        q = (rng.normal(0, 1, (B, Hq, 128)) * rng.uniform(0.2, 3, (B, Hq, 1))).astype(np.float16)
        k = Q.kv4_quant(torch.from_numpy(K).cuda())
        v = Q.kv4_quant(torch.from_numpy(V).cuda())
        kq, ks, kz = okv4.kv4_quant(K)
        vq, vs, vz = okv4.kv4_quant(V)
        ref = okv4.attention_decode(q, okv4.kv4_dequant(kq, ks, kz), okv4.kv4_dequant(vq, vs, vz))
        for rep in range(2):
            y = Q.kv4_attention_decode(torch.from_numpy(q).cuda(), k, v, workspace=ws)
            err = np.abs(y.cpu().numpy().astype(np.float64) - ref).max(axis=-1) / np.abs(ref).max(axis=-1)
            print(f"reused workspace B={B} T={T} call {rep}: max rel err {err.max():.2e}")
            assert err.max() <= TOL, (B, T, rep, err.max())
