"""The KV4 decode attention entry point that allocates nothing (qift_kv4_attention_decode_noalloc, its
partial records in the library's per-GPU array) against the entry point with a caller workspace: the
same fp16 outputs bit for bit, on two calls in a row, the second with a smaller input (the array
keeps the first call's records, and the second call must not read any of them)."""
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def Q():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_02823_amd import qift
    qift.lib()
    return qift


def _case(Q, gen, B, Hq, Hkv, T, head_major):
    shape = (B, Hkv, T, 128) if head_major else (B, T, Hkv, 128)
    K = torch.randn(shape, generator=gen, device="cuda").half()
    V = torch.randn(shape, generator=gen, device="cuda").half()
    q = torch.randn((B, Hq, 128), generator=gen, device="cuda").half()
    return q, Q.kv4_quant(K), Q.kv4_quant(V)


def test_noalloc_matches_workspace_entry(Q):
    gen = torch.Generator(device="cuda")
    gen.manual_seed(57)
    # (B, Hq, Hkv, T, head-major): 2 x 20 chunks of 256 tokens with 4 query heads per KV head, then a
    # smaller call (one sequence, 4 chunks, the last one partial, 8 query heads per KV head)
    for B, Hq, Hkv, T, hm in ((2, 32, 8, 5000, True), (1, 32, 4, 777, False)):
        print(f"noalloc kv4 attention B={B} Hq={Hq} Hkv={Hkv} T={T} head_major={hm}", flush=True)
        q, k, v = _case(Q, gen, B, Hq, Hkv, T, hm)
        ref = Q.kv4_attention_decode(q, k, v, head_major=hm)
        out = torch.full((B, Hq, 128), float("nan"), dtype=torch.float16, device="cuda")
        Q.kv4_attention_decode_noalloc(q, k, v, out, head_major=hm)
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), (B, Hq, Hkv, T, hm)
    assert Q.device_error() == 0
