"""ssm_attention_static, the entry point that allocates nothing, against
ssm_attention with a caller workspace: bit-identical outputs (the same
kernels and split choice), over two calls in a row on the shared static
scratch, the second smaller than the first, with the key range split so that
the partial results pass through the scratch, then a launch that does not
split."""
import pytest
import torch

from synthetic.generate import seeded_normal

pytestmark = pytest.mark.gpu


def _inputs(B, H, Hkv, n_q, cap, seed, dtype):
    q = seeded_normal((B, H, n_q, 128), seed, "static.q", device="cuda", dtype=dtype)
    k = seeded_normal((B, Hkv, cap, 128), seed, "static.k", device="cuda", dtype=dtype)
    v = seeded_normal((B, Hkv, cap, 128), seed, "static.v", device="cuda", dtype=dtype)
    return q, k, v


def _both(B, H, Hkv, n_q, n_keys, cap, seed, dtype):
    from paper_2608_23167_amd.api import (ssm_attention, ssm_attention_static,
                                          ssm_attention_workspace_size)
    q, k, v = _inputs(B, H, Hkv, n_q, cap, seed, dtype)
    ref = torch.empty((B, n_q, H * 128), device="cuda", dtype=torch.float32)
    ws = torch.empty(ssm_attention_workspace_size(B, H, n_q), device="cuda", dtype=torch.uint8)
    ssm_attention(q, k, v, n_keys, ref, ws)
    got = torch.full((B, n_q, H * 128), float("nan"), device="cuda", dtype=torch.float32)
    ssm_attention_static(q, k, v, n_keys, got)
    torch.cuda.synchronize()
    return got, ref


@pytest.mark.parametrize("dtype", [torch.float16, torch.bfloat16])
def test_static_scratch_matches_workspace_call(gpu, dtype):
    cases = [
        # 16 heads over 4 KV heads, 100 rows, 3000 keys: 16 key splits, 25600 partial rows
        (2, 8, 2, 100, 3000, 3072, 1),
        # smaller, right after: 12 splits over 1500 keys, fewer rows than the scratch holds
        (1, 4, 4, 70, 1500, 1536, 2),
        # 600 keys: no split, the scratch is not used
        (1, 4, 2, 33, 600, 640, 3),
    ]
    for B, H, Hkv, n_q, n_keys, cap, seed in cases:
        print(f"[static] {dtype} B {B} H {H}/{Hkv} rows {n_q} keys {n_keys}", flush=True)
        got, ref = _both(B, H, Hkv, n_q, n_keys, cap, seed, dtype)
        assert torch.equal(got, ref), (B, H, n_q, n_keys)
        assert torch.isfinite(got).all()
