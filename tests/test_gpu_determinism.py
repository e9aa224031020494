"""Run-to-run determinism: the library uses no atomics in its reductions and
fixed split orders, so the same step on the same inputs must give
bit-identical outputs every time.  Each case runs twice from the same state
(through the C ABI) and compares every output bit for bit: hidden states,
logits, row statistics, tokens and prediction state."""
import numpy as np
import pytest
import torch

from synthetic import WORKLOADS, initial_tokens, make_weights, mid_generation_state
from tests._parity import gpu_step

pytestmark = pytest.mark.gpu

KEYS = ("x", "hidden", "logits", "argmax", "conf", "topk_ids", "topk_w", "tokens", "selected")


def _decoder(wl, mw_dev):
    from paper_2608_23167_amd.decoder import Decoder
    from paper_2608_23167_amd.model import DeviceModel
    return Decoder(wl, DeviceModel(wl.model, mw_dev))


def _load(dec, state, step):
    """Puts a seeded decoding state (tokens, prediction ids, weights, stamps)
    into the decoder."""
    dev = dec.tokens.device
    t, pi, pw, ps = state
    dec.tokens.copy_(torch.from_numpy(np.asarray(t, np.int32)).to(dev))
    dec.pred_ids.copy_(torch.from_numpy(np.asarray(pi, np.int32)).to(dev))
    dec.pred_w.copy_(torch.from_numpy(np.asarray(pw, np.float32)).to(dev))
    dec.pred_step.copy_(torch.from_numpy(np.asarray(ps, np.int32)).to(dev))
    dec.step_idx = step


def _twice(dec, state, step, block_idx, first):
    outs = []
    for _ in range(2):
        _load(dec, state, step)
        out = gpu_step(dec, block_idx, first)
        out["pred"] = [a.cpu().numpy() for a in (dec.pred_ids, dec.pred_w, dec.pred_step)]
        outs.append(out)
    a, b = outs
    for key in KEYS:
        assert np.array_equal(a[key], b[key]), f"{key} differs between two identical runs"
    for x, y in zip(a["pred"], b["pred"]):
        assert np.array_equal(x, y), "prediction state differs between two identical runs"
    return a


@pytest.mark.parametrize("name,block,first", [
    ("llada_gen256", 0, True),        # 376 rows: one-pass tiles, split-K sums
    ("llada_gen256", 0, False),       # 120 rows: decode tiles, split-K 2-8
    ("llada_long1024", 8, True),      # 1776 rows: big tiles with split-K
    ("llada_long2048", 31, False),    # 64 rows over a 3008-key prefix: split-KV attention
])
def test_step_bit_identical(gpu, name, block, first):
    wl = WORKLOADS[name]
    wl = wl.replace(model=wl.model.with_layers(2))
    mw = make_weights(wl.model, seed=0, norm_jitter=0.1).to("cuda:0")
    dec = _decoder(wl, mw)
    step = 0 if first else 1
    state = mid_generation_state(wl, block, step, seed=1)
    if wl.cache and not first:
        # the prefix cache of this block, written by its block-start step
        _load(dec, state, step)
        dec.step(block, True, unmask=False)
        torch.cuda.synchronize()
    out = _twice(dec, state, step, block, first)
    print(f"[determinism] {name} block {block} first={first}: {out['info'].n_rows} rows identical",
          flush=True)


def test_generation_bit_identical(gpu):
    """Two free-running generations of the bench workload's first block (2
    layers) give the same tokens and prediction state."""
    wl = WORKLOADS["llada_gen256"]
    wl = wl.replace(model=wl.model.with_layers(2))
    mw = make_weights(wl.model, seed=0).to("cuda:0")
    dec = _decoder(wl, mw)
    tok0 = initial_tokens(wl).to("cuda:0")
    res = []
    for _ in range(2):
        dec.generate(tok0, max_steps=wl.steps_per_block() + 2)
        torch.cuda.synchronize()
        res.append([t.cpu().numpy().copy() for t in (dec.tokens, dec.pred_ids, dec.pred_w, dec.pred_step)])
    for a, b in zip(*res):
        assert np.array_equal(a, b)


def test_attention_split_bit_identical(gpu):
    """The split-KV attention and its merge (240 queries x 4336 keys, batch 2:
    the microbenchmark's kept-176 shape) twice on the same inputs."""
    from paper_2608_23167_amd.api import ssm_attention, ssm_attention_workspace_size
    torch.manual_seed(0)
    B, H, dh, nq, nk = 2, 32, 128, 240, 4336
    q = torch.randn(B, H, nq, dh, device="cuda:0").to(torch.float16)
    k = torch.randn(B, H, nk, dh, device="cuda:0").to(torch.float16)
    v = torch.randn(B, H, nk, dh, device="cuda:0").to(torch.float16)
    ws = torch.empty(ssm_attention_workspace_size(B, H, nq), dtype=torch.uint8, device="cuda:0")
    outs = []
    for _ in range(2):
        o = torch.empty(B, nq, H * dh, dtype=torch.float32, device="cuda:0")
        ssm_attention(q, k, v, nk, o, ws)
        torch.cuda.synchronize()
        outs.append(o.cpu().numpy())
    assert np.array_equal(outs[0], outs[1])
