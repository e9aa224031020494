"""Attention and row gather on their own (ssm_attention, ssm_gather_rows)
against the oracle: the attention-and-gather microbenchmark shape (LLaDA-8B
heads, batch 8, prefix KV of 4096, block 64, kept suffix 176 and the full
4096) and small ragged shapes.

Tolerance: the kernel rounds the softmax probabilities to the operand type
before the P V product (bfloat16 to nearest: relative rounding 2^-9 per
probability; float16 toward zero: below 2^-10), with scores, softmax and
accumulation in float32; the oracle is float64 on the same 16-bit inputs.
The relative L2 error of the output is then of order 2^-9; the bound 1e-2
leaves a factor of five.  Both operand types run: bfloat16 (the
microbenchmark's inputs) and float16 (what the step of a bfloat16 model
uses)."""
import numpy as np
import pytest
import torch

import oracle.model as OM
from synthetic.generate import seeded_normal, seeded_uniform_ints

pytestmark = pytest.mark.gpu

TOL = 1e-2


def _inputs(B, H, Hkv, n_q, cap, seed, dtype=torch.bfloat16):
    dev = "cuda"
    q = seeded_normal((B, H, n_q, 128), seed, "attn.q", device=dev, dtype=dtype)
    k = seeded_normal((B, Hkv, cap, 128), seed, "attn.k", device=dev, dtype=dtype)
    v = seeded_normal((B, Hkv, cap, 128), seed, "attn.v", device=dev, dtype=dtype)
    return q, k, v


def _run(q, k, v, n_keys):
    from paper_2608_23167_amd.api import ssm_attention, ssm_attention_workspace_size
    B, H, n_q, _ = q.shape
    out = torch.empty((B, n_q, H * 128), device="cuda", dtype=torch.float32)
    ws = torch.empty(ssm_attention_workspace_size(B, H, n_q), device="cuda", dtype=torch.uint8)
    ssm_attention(q, k, v, n_keys, out, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def _oracle_rows(q, k, v, n_keys, s, rows):
    """Oracle attention of query rows `rows` of sequence s: [len(rows), H*128]."""
    qs = q[s, :, rows, :].float().cpu().numpy().astype(np.float64).transpose(1, 0, 2)
    ks = k[s, :, :n_keys, :].float().cpu().numpy().astype(np.float64).transpose(1, 0, 2)
    vs = v[s, :, :n_keys, :].float().cpu().numpy().astype(np.float64).transpose(1, 0, 2)
    return OM.attention(qs, ks, vs)


def _rel(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float16])
@pytest.mark.parametrize("B,H,Hkv,n_q,n_keys,cap", [
    (2, 4, 2, 70, 200, 256),      # GQA, ragged query tile and key tile
    (1, 2, 2, 1, 1, 8),           # one query, one key
    (1, 4, 1, 64, 64, 64),        # exact tiles, 4 heads on one KV head
    (3, 2, 2, 129, 1000, 1030),   # several key tiles: split key ranges and merge
    (1, 32, 32, 120, 472, 512),   # decode step (LLaDA-8B heads): 16 query rows per workgroup
    (1, 28, 4, 119, 600, 640),    # decode, GQA (Dream-7B heads), two key tiles for some waves
    (1, 32, 32, 376, 472, 512),   # block start: two key groups per workgroup
])
def test_attention_matches_oracle(gpu, B, H, Hkv, n_q, n_keys, cap, dtype):
    q, k, v = _inputs(B, H, Hkv, n_q, cap, seed=B * 1000 + n_q, dtype=dtype)
    got = _run(q, k, v, n_keys)
    for s in range(B):
        ref = _oracle_rows(q, k, v, n_keys, s, list(range(n_q)))
        assert _rel(got[s], ref) < TOL, (s, _rel(got[s], ref))


@pytest.mark.parametrize("kept,dtype", [(0, torch.bfloat16), (48, torch.bfloat16),
                                        (176, torch.bfloat16), (512, torch.bfloat16),
                                        (4096, torch.bfloat16), (176, torch.float16)])
def test_attention_microbench_shape_every_row(gpu, kept, dtype):
    """Batch 8, 32 heads: prefix 4096 + block 64 + kept suffix rows attend to
    all prefix, block and kept keys, at points of the kept-suffix sweep (0:
    block only, 48: the first point with middle and tail, 176: the workload's
    budgets, 512, 4096: the whole suffix).  Every element of every row of two
    of the eight sequences is checked against the float64 oracle, within the
    bound that the bfloat16 rounding of the probabilities allows: each
    p_j moves by at most 2^-9 p_j and so does their sum, so an output element
    moves by at most 2^-8 sum_j p_j |v_j| (taken as 2^-7, plus 1e-6 for the
    float32 softmax and accumulation); sum_j p_j |v_j| is the oracle's
    attention over |v|."""
    B, H = 8, 32
    n_q = 64 + kept
    n_keys = 4096 + 64 + kept
    q, k, v = _inputs(B, H, H, n_q, n_keys, seed=kept, dtype=dtype)
    got = _run(q, k, v, n_keys)
    rows = list(range(n_q))
    for s in (0, 7):
        ref = _oracle_rows(q, k, v, n_keys, s, rows)
        bound = 2.0 ** -7 * _oracle_rows(q, k, v.abs(), n_keys, s, rows) + 1e-6
        err = np.abs(got[s].astype(np.float64) - ref)
        worst = float(np.max(err / bound))
        print(f"[attention] {dtype} kept {kept} sequence {s}: {n_q} rows x {n_keys} keys, rel "
              f"{_rel(got[s], ref):.2e}, worst error / bound {worst:.3f}", flush=True)
        assert worst <= 1.0, (s, worst)
        assert _rel(got[s], ref) < TOL


def test_gather_rows_bit_exact(gpu):
    from paper_2608_23167_amd.api import ssm_gather_rows
    B, rows, width = 3, 100, 4096
    src = seeded_normal((B, rows, width), 5, "gather.src", device="cuda", dtype=torch.bfloat16)
    pos = seeded_uniform_ints((37,), 0, rows, 5, "gather.pos", device="cuda")
    pos[3] = -1                      # outside the source: zeros
    pos[10] = rows
    pos[11] = pos[12]                # repeated position
    out = torch.empty((B, pos.numel(), width), device="cuda", dtype=torch.bfloat16)
    ssm_gather_rows(src, pos, out)
    torch.cuda.synchronize()
    s_np = src.view(torch.int16).cpu().numpy()
    p_np = pos.cpu().numpy()
    ref = np.zeros((B, p_np.size, width), np.int16)
    ok = (p_np >= 0) & (p_np < rows)
    ref[:, ok] = s_np[:, p_np[ok]]
    assert np.array_equal(out.view(torch.int16).cpu().numpy(), ref)


def test_gather_rows_microbench_shape(gpu):
    """The kept suffix rows (local 128, middle 32, tail 16 of 4096) of a
    [8, 4096, 4096] bf16 tensor."""
    from paper_2608_23167_amd.api import ssm_gather_rows
    import oracle.selection as OS
    B, rows, width = 8, 4096, 4096
    # prefix 4096, block [4096, 4160), suffix [4160, 8256): kept suffix rows
    # as indices into the suffix tensor
    kept = OS.retained_suffix(4096, 64 + rows, 64, 0, 128, 32, 0, 16).positions
    pos = torch.tensor(np.asarray(kept, np.int32) - 4160, device="cuda")
    src = seeded_normal((B, rows, width), 6, "gather.big", device="cuda", dtype=torch.bfloat16)
    out = torch.empty((B, pos.numel(), width), device="cuda", dtype=torch.bfloat16)
    ssm_gather_rows(src, pos, out)
    torch.cuda.synchronize()
    assert pos.numel() == 176
    assert torch.equal(out, src[:, pos.long()])
