"""Batches whose prompts differ in length, against the oracle run on each
sequence alone with its own prompt length.

The batch shares the row layout of its longest prompt; sequence s, pad[s]
tokens shorter, reads row r at its own position pos[r] - pad[s] (Section
3.2: every retained token keeps its original position; with a shared
generation length its suffix regions and retained set R_t are those of the
longest prompt shifted by pad[s]).  Its padding rows are never keys.  So
sequence s of the batch must reproduce, row for row, the oracle's step of
that sequence alone: positions bit-exact, hidden states and logits within
the float32 or bfloat16 tolerances, decisions under the rule of
tests/_parity.py, tokens and prediction state after the step identical.
"""
import numpy as np
import pytest
import torch

import oracle.generate as OG
from synthetic import WORKLOADS, initial_tokens, make_weights, mid_generation_state, spread
from tests._parity import (Counts, check_decisions, check_unmask, check_unmask_consistency,
                           gpu_step, logit_budget, max_abs, rel_err)

pytestmark = pytest.mark.gpu


def _decoder(wl, mw_dev, prompt_lens):
    from paper_2608_23167_amd import _lib as L
    from paper_2608_23167_amd.decoder import Decoder
    from paper_2608_23167_amd.model import DeviceModel
    return Decoder(wl, DeviceModel(wl.model, mw_dev), prompt_lens=prompt_lens)


def _own(wl, P0):
    """The workload of one sequence alone."""
    return wl.replace(prompt_len=P0, batch=1)


def _load_states(dec, states):
    """Puts each sequence's oracle state (batch 1, its own length) into the
    batched decoder, at the start of that sequence's row of every array."""
    wl = dec.wl
    L, k = wl.total_len, wl.topk
    tok = np.full((wl.batch, L), wl.model.mask_id, np.int32)
    ids = np.zeros((wl.batch, L, k), np.int32)
    w = np.zeros((wl.batch, L, k), np.float32)
    ps = np.full((wl.batch, L), -1, np.int32)
    for s, st in enumerate(states):
        n = st.tokens.shape[1]
        tok[s, :n], ids[s, :n], w[s, :n], ps[s, :n] = st.tokens[0], st.pred_ids[0], st.pred_w[0], st.pred_step[0]
    dev = dec.tokens.device
    dec.tokens.copy_(torch.from_numpy(tok).to(dev))
    dec.pred_ids.copy_(torch.from_numpy(ids).to(dev))
    dec.pred_w.copy_(torch.from_numpy(w).to(dev))
    dec.pred_step.copy_(torch.from_numpy(ps).to(dev))
    dec.step_idx = states[0].step


def _seq_view(out, s):
    """Sequence s of a batched GPU step as a batch-1 result."""
    one = {}
    for key in ("argmax", "conf", "topk_ids", "topk_w", "logits", "selected"):
        one[key] = out[key][s:s + 1]
    one["tokens"] = out["tokens"][s:s + 1]
    return one


def _compare(out, recs, wls, pads, fp32, dc, uc):
    """Sequence s of the batched step `out` against the oracle's step `recs[s]`."""
    first_batched = out["info"].first_out_row
    for s, (rec, wl_s, pad) in enumerate(zip(recs, wls, pads)):
        rows = rec.rows
        # a block-start step: the oracle's prefix is pad rows shorter
        off = pad if rec.include_prefix else 0
        n = len(rows.pos)
        assert first_batched - off == rows.first_out_row
        pos = out["pos"][off:off + n] - pad
        assert np.array_equal(pos, rows.pos), f"positions of sequence {s}"
        assert np.array_equal(out["region"][off:off + n], rows.region)
        if rec.include_prefix and pad:
            assert np.all(out["pos"][:off] - pad < 0)                 # the padding rows
        h = out["hidden"][s, off:off + n]
        if fp32:
            assert max_abs(out["x"][s, off:off + n], rec.x[0]) < 1e-6
            assert max_abs(h, rec.hidden[0]) < 1e-4, f"hidden of sequence {s}"
            assert max_abs(out["logits"][s], rec.stats[0].logits) < 1e-4
        else:
            assert max_abs(out["x"][s, off:off + n], rec.x[0]) < 1e-5
            assert rel_err(h, rec.hidden[0]) < 2e-2, f"hidden of sequence {s}: {rel_err(h, rec.hidden[0])}"
            assert rel_err(out["logits"][s], rec.stats[0].logits) < 2e-2
        one = _seq_view(out, s)
        one["tokens"] = one["tokens"][:, :wl_s.total_len]
        dc.add(check_decisions(one, rec, wl_s, fp32))
        uc.add(check_unmask(one, rec, wl_s, fp32))
        check_unmask_consistency(one, rec, wl_s)


PROMPTS = [32, 21, 9]
# prompt seeds of the free-running cases: per sequence, one whose trajectory clears the budget
FREE_SEEDS = [21, 20, 20]


@pytest.mark.parametrize("cache", [False, True])
def test_tiny_fp32_ragged_every_step(gpu, cache):
    """Every teacher-forced step of a whole generation of the tiny workload
    (wide-margin variant) for three prompts of 32, 21 and 9 tokens."""
    wl = spread(WORKLOADS["tiny"]).replace(batch=len(PROMPTS), cache=cache, prompt_len=max(PROMPTS))
    mw = make_weights(wl.model, seed=0, norm_jitter=0.1, logit_scale=wl.logit_scale)
    w = OG.NumpyWeights(mw)
    dec = _decoder(wl, mw.to("cuda"), PROMPTS)
    pads = dec.pad
    wls = [_own(wl, P0) for P0 in PROMPTS]
    states = [OG.OracleState.start(initial_tokens(wl_s, seed=10 + s).numpy(), wl.topk)
              for s, wl_s in enumerate(wls)]
    dc, uc = Counts(), Counts()
    for j in range(wl.n_blocks):
        for i in range(wl.steps_per_block()):
            _load_states(dec, states)
            recs = [OG.step(wl_s, w, st, j, i == 0) for wl_s, st in zip(wls, states)]
            out = gpu_step(dec, j, i == 0)
            _compare(out, recs, wls, pads, True, dc, uc)
            got_t = out["tokens"]
            for s, st in enumerate(states):
                n = st.tokens.shape[1]
                assert np.array_equal(got_t[s, :n], st.tokens[0]), f"tokens of sequence {s}"
            ps = dec.pred_step.cpu().numpy()
            for s, st in enumerate(states):
                n = st.tokens.shape[1]
                assert np.array_equal(ps[s, :n], st.pred_step[0])
    print(f"[ragged] tiny cache {cache}: argmax {dc}; unmask {uc}", flush=True)
    assert dc.checked > 0.95 * dc.total and uc.checked > 0.7 * uc.total


@pytest.mark.parametrize("cache", [False, True])
def test_tiny_fp32_ragged_free_running(gpu, cache):
    """Free-running top-n generation of three prompts of different lengths:
    each sequence's final tokens equal the oracle's generation of that
    sequence alone (whose decisions clear the float32 budget and whose
    trajectory does not depend on float32 rounding).  Top-n keeps the batch
    in lockstep with each sequence's own schedule; under the threshold rule a
    batch steps until its slowest sequence has finished the block, and the
    extra steps refresh the finished sequences' suffix predictions, which a
    sequence decoded alone never sees."""
    wl = spread(WORKLOADS["tiny"]).replace(batch=len(PROMPTS), cache=cache, prompt_len=max(PROMPTS))
    mw = make_weights(wl.model, seed=0, norm_jitter=0.1, logit_scale=wl.logit_scale)
    wls = [_own(wl, P0) for P0 in PROMPTS]
    tok = np.full((wl.batch, wl.total_len), wl.model.mask_id, np.int32)
    finals, n_steps = [], 0
    for s, wl_s in enumerate(wls):
        t0 = initial_tokens(wl_s, seed=FREE_SEEDS[s]).numpy()
        tok[s, :wl_s.total_len] = t0[0]
        st, recs = OG.generate(wl_s, OG.NumpyWeights(mw), t0, keep=True)
        st32, recs32 = OG.generate(wl_s, OG.NumpyWeights(mw, dtype=np.float32), t0, keep=True)
        assert np.array_equal(st32.tokens, st.tokens) and len(recs32) == len(recs)
        drift = max(float(np.max(np.abs(a.stats[0].logits - b.stats[0].logits)))
                    for a, b in zip(recs, recs32))
        eps = max(1e-4, 4.0 * drift)
        uc = Counts()
        for rec in recs:
            uc.add(check_unmask({"argmax": [x.argmax for x in rec.stats], "topk_ids": None,
                                 "selected": rec.selected, "tokens": rec.tokens_after},
                                rec, wl_s, True, eps=eps))
        assert uc.inside == 0, f"sequence {s}: {uc.inside} decisions inside the budget"
        finals.append(st.tokens[0])
        n_steps = max(n_steps, len(recs))
    dec = _decoder(wl, mw.to("cuda"), PROMPTS)
    out = dec.generate(torch.from_numpy(tok).cuda()).cpu().numpy()
    print(f"[ragged] free-running cache {cache}: GPU {dec.step_idx} steps, oracle {n_steps}", flush=True)
    for s, f in enumerate(finals):
        assert np.array_equal(out[s, :len(f)], f), f"sequence {s}"
    assert dec.step_idx == n_steps


def _ragged_cache(dec, states, prompt_lens, P_u, seed):
    """Seeded bf16/f16 values in cache slots [0, P_u) of every layer; sequence
    s's prefix of P_u - pad rows sits in slots [pad, P_u), which its oracle
    state receives."""
    from synthetic import seeded_normal
    shape = dec.wl.model
    B = dec.wl.batch
    caches = [[] for _ in range(B)]
    for l in range(shape.n_layers):
        kv = []
        for name, buf in (("k", dec.cache.k), ("v", dec.cache.v)):
            t = seeded_normal((B, shape.n_kv_heads, P_u, shape.head_dim), seed,
                              f"ragged.{name}.{l}", std=1.0, device=buf.device, dtype=buf.dtype)
            buf[l, :, :, :P_u, :].copy_(t)
            kv.append(t.float().cpu().numpy())
        for s in range(B):
            pad = dec.pad[s]
            caches[s].append((np.ascontiguousarray(kv[0][s, :, pad:].transpose(1, 0, 2)),
                              np.ascontiguousarray(kv[1][s, :, pad:].transpose(1, 0, 2))))
    for s, st in enumerate(states):
        st.cache = [caches[s]]


@pytest.mark.parametrize("first,j", [(True, 3), (False, 3), (False, 7)])
def test_llada_shape_2_layers_bf16_ragged(gpu, first, j):
    """LLaDA-8B shape (two layers, sharpened LM head), bfloat16, prompts of
    256, 200 and 131 tokens: at block 3 the block-start step (prefix rows with
    padding, 472 rows in all) and a cached step (padding slots in the cache);
    at the last block (no suffix left, 32 rows) a cached step, whose attention
    takes the decode kernel (16 query rows per workgroup) over padded caches."""
    from synthetic import sharpened
    prompts = [256, 200, 131]
    wl = sharpened(WORKLOADS["llada_gen256"], 30.0).replace(batch=3)
    wl = wl.replace(model=wl.model.with_layers(2))
    mw = make_weights(wl.model, seed=0, device="cuda", norm_jitter=0.1, logit_scale=wl.logit_scale)
    w = OG.NumpyWeights(mw, dtype=np.float32)
    dec = _decoder(wl, mw, prompts)
    wls = [_own(wl, P0) for P0 in prompts]
    states = []
    for s, wl_s in enumerate(wls):
        t, pi, pw, ps = mid_generation_state(wl_s, j, 7, 30 + s)
        st = OG.OracleState.start(t, wl.topk)
        st.pred_ids[:], st.pred_w[:], st.pred_step[:], st.step = pi, pw, ps, 7
        states.append(st)
    if not first:
        _ragged_cache(dec, states, prompts, wl.prompt_len + j * wl.block_size, 11)
    _load_states(dec, states)
    recs = [OG.step(wl_s, w, st, j, first) for wl_s, st in zip(wls, states)]
    out = gpu_step(dec, j, first)
    dc, uc = Counts(), Counts()
    _compare(out, recs, wls, dec.pad, False, dc, uc)
    print(f"[ragged] llada 2 layers {'start' if first else 'cached'} rows {out['info'].n_rows}: "
          f"argmax {dc}; unmask {uc}", flush=True)
    assert dc.checked > 0
