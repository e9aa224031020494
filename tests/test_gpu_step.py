"""GPU step parity against the oracle (teacher-forced: every GPU step starts
from the oracle's state before that step).

fp32 mode (tiny model): hidden states and logits within max-abs 1e-4.
bf16 mode (LLaDA / Dream shapes): relative error <= 2e-2 against the fp32
oracle run on the bf16-rounded weights.  Decisions (argmax, top-k ids,
unmasking) must agree wherever the oracle's probability margin exceeds 1e-3,
except inside the fixed logit error budget of tests/_parity.py; every test
prints how many decisions it checked and how many were exempt, and asserts
a floor on the checked count.
"""
import numpy as np
import pytest
import torch

import oracle.generate as OG
from synthetic import (WORKLOADS, initial_tokens, make_weights, mid_generation_state, sharpened,
                       spread)
from tests._parity import (Counts, check_decisions, check_unmask, check_unmask_consistency,
                           gpu_step, load_oracle_state, max_abs, rel_err)

pytestmark = pytest.mark.gpu

def _decoder(wl, mw_dev, act_mode=None, pair_layers=0):
    from paper_2608_23167_amd import _lib as L
    from paper_2608_23167_amd.decoder import Decoder
    from paper_2608_23167_amd.model import DeviceModel
    mode = L.SSM_ACT_BF16X2 if act_mode is None else act_mode
    return Decoder(wl, DeviceModel(wl.model, mw_dev, act_mode=mode, pair_layers=pair_layers))


def _compare_step(out, rec, wl, fp32: bool):
    B = wl.batch
    assert np.array_equal(out["pos"], rec.rows.pos)
    assert np.array_equal(out["region"], rec.rows.region)
    tol_x = 1e-6 if fp32 else 1e-5
    assert max_abs(out["x"], rec.x) < tol_x
    if fp32:
        assert max_abs(out["hidden"], rec.hidden) < 1e-4
        for s in range(B):
            assert max_abs(out["logits"][s], rec.stats[s].logits) < 1e-4
            assert max_abs(out["conf"][s], rec.stats[s].conf) < 1e-5
            assert max_abs(out["topk_w"][s], rec.stats[s].topk_w) < 1e-4
    else:
        assert rel_err(out["hidden"], rec.hidden) < 2e-2
        for s in range(B):
            assert rel_err(out["logits"][s], rec.stats[s].logits) < 2e-2
    return check_decisions(out, rec, wl, fp32)


def _compare_unmask(out, rec, wl, fp32: bool):
    check_unmask_consistency(out, rec, wl)
    return check_unmask(out, rec, wl, fp32)


def _report(name, dec: Counts, unm: Counts):
    print(f"[decisions] {name}: argmax {dec}; unmask {unm}", flush=True)


@pytest.mark.parametrize("wide", [False, True])
def test_tiny_fp32_every_step(gpu, wide):
    """Every teacher-forced step of the tiny workload; with `wide`, the test
    variant whose confidences and margins spread over (0, 1), so that nearly
    every decision lies outside the budget and is checked."""
    wl = WORKLOADS["tiny"]
    if wide:
        wl = spread(wl)
    mw = make_weights(wl.model, seed=0, norm_jitter=0.1, logit_scale=wl.logit_scale)
    w = OG.NumpyWeights(mw)
    dec = _decoder(wl, mw.to("cuda"))
    tok0 = initial_tokens(wl).numpy()
    st = OG.OracleState.start(tok0, wl.topk)
    dc, uc = Counts(), Counts()
    for j in range(wl.n_blocks):
        for i in range(wl.steps_per_block()):
            before = st.copy()
            rec = OG.step(wl, w, st, j, i == 0)
            load_oracle_state(dec, before)
            out = gpu_step(dec, j, i == 0)
            dc.add(_compare_step(out, rec, wl, fp32=True))
            uc.add(_compare_unmask(out, rec, wl, fp32=True))
    _report(wl.name, dc, uc)
    if wide:
        assert dc.checked > 0.95 * dc.total and uc.checked > 0.7 * uc.total


def test_tiny_fp32_cached_steps(gpu):
    """Prefix cache on: block-start steps write the cache, later steps read it."""
    wl = spread(WORKLOADS["tiny"]).replace(cache=True)
    mw = make_weights(wl.model, seed=1, norm_jitter=0.1, logit_scale=wl.logit_scale)
    w = OG.NumpyWeights(mw)
    dec = _decoder(wl, mw.to("cuda"))
    st = OG.OracleState.start(initial_tokens(wl, seed=2).numpy(), wl.topk)
    dc, uc = Counts(), Counts()
    for j in range(wl.n_blocks):
        for i in range(wl.steps_per_block()):
            before = st.copy()
            rec = OG.step(wl, w, st, j, i == 0)
            load_oracle_state(dec, before)
            out = gpu_step(dec, j, i == 0)
            assert out["info"].include_prefix == (i == 0)
            dc.add(_compare_step(out, rec, wl, fp32=True))
            uc.add(_compare_unmask(out, rec, wl, fp32=True))
    _report(wl.name + " cached", dc, uc)
    assert dc.checked > 0.95 * dc.total and uc.checked > 0.7 * uc.total


@pytest.mark.parametrize("local,mmode,T,tmode", [
    (64, 1, 2, 0),    # the paper's block rule (Eq. 2-4): w = 2 blocks, middle starts, tail ends
    (40, 3, 1, 1),    # Table 2 variants: middle start+end tokens, tail start token only
    (40, 2, 3, 0),    # middle end tokens, tail start+mid+end
])
def test_tiny_fp32_selection_variants(gpu, local, mmode, T, tmode):
    """Whole teacher-forced generations of the tiny model (cached) under the
    paper's block rule and the Table 2 retention variants; a local budget of 40
    cuts a block, so the middle starts inside one."""
    wl = spread(WORKLOADS["tiny"]).replace(
        cache=True, gen_len=192, local_budget=local, middle_mode=mmode, tail_budget=T,
        tail_mode=tmode)
    mw = make_weights(wl.model, seed=3, norm_jitter=0.1, logit_scale=wl.logit_scale)
    w = OG.NumpyWeights(mw)
    dec = _decoder(wl, mw.to("cuda"))
    st = OG.OracleState.start(initial_tokens(wl, seed=4).numpy(), wl.topk)
    dc, uc = Counts(), Counts()
    for j in range(wl.n_blocks):
        for i in range(2):
            before = st.copy()
            rec = OG.step(wl, w, st, j, i == 0)
            load_oracle_state(dec, before)
            out = gpu_step(dec, j, i == 0)
            dc.add(_compare_step(out, rec, wl, fp32=True))
            uc.add(_compare_unmask(out, rec, wl, fp32=True))
    _report(f"{wl.name} local {local} middle {mmode} tail {T}/{tmode}", dc, uc)
    assert dc.checked > 0.95 * dc.total and uc.checked > 0.7 * uc.total


def test_tiny_fp32_early_termination(gpu):
    """Teacher-forced generation of the tiny model (two sequences) with an end
    id the model decodes in the first block: the GPU's per-block early-stop
    fill and done flags match the oracle's, and the generation ends there."""
    from paper_2608_23167_amd.api import ssm_early_stop
    eos = 7
    wl = WORKLOADS["tiny"].replace(batch=2, cache=True, eos_id=eos)
    mw = make_weights(wl.model, seed=0, norm_jitter=0.1)
    mw.lm_head[eos] *= 40.0          # logits of the end id about 40x the others' scale
    w = OG.NumpyWeights(mw)
    dec = _decoder(wl, mw.to("cuda"))
    st = OG.OracleState.start(initial_tokens(wl).numpy(), wl.topk)
    ended_at = None
    for j in range(wl.n_blocks):
        for i in range(wl.steps_per_block()):
            before = st.copy()
            rec = OG.step(wl, w, st, j, i == 0)
            load_oracle_state(dec, before)
            out = gpu_step(dec, j, i == 0)
            _compare_step(out, rec, wl, fp32=True)
            _compare_unmask(out, rec, wl, fp32=True)
        # both sides apply the block-end check to the same (oracle) tokens
        dec.tokens.copy_(torch.from_numpy(st.tokens))
        dec.done.copy_(torch.from_numpy(st.done.astype(np.int32)))
        all_done = OG.early_stop(st.tokens, st.done, wl.prompt_len + j * wl.block_size,
                                 wl.block_size, eos)
        assert dec.early_stop(j) == all_done
        assert np.array_equal(dec.tokens.cpu().numpy(), st.tokens)
        assert np.array_equal(dec.done.cpu().numpy().astype(bool), st.done)
        if all_done:
            ended_at = j
            break
    assert ended_at == 0


def _state_from(wl, block_idx, step, seed):
    t, pi, pw, ps = mid_generation_state(wl, block_idx, step, seed)
    st = OG.OracleState.start(t, wl.topk)
    st.pred_ids[:] = pi
    st.pred_w[:] = pw
    st.pred_step[:] = ps
    st.step = step
    return st


def _bf16_case(wl, blocks, seed=0, act_mode=None, pair_layers=0):
    torch.manual_seed(0)
    mw_dev = make_weights(wl.model, seed=seed, device="cuda", norm_jitter=0.1,
                          logit_scale=wl.logit_scale)
    w = OG.NumpyWeights(mw_dev, dtype=np.float32)
    dec = _decoder(wl, mw_dev, act_mode, pair_layers)
    dc, uc = Counts(), Counts()
    for j, n_steps in blocks:
        st = _state_from(wl, j, 5 + 3 * j, seed)
        for i in range(n_steps):
            before = st.copy()
            rec = OG.step(wl, w, st, j, i == 0)
            load_oracle_state(dec, before)
            out = gpu_step(dec, j, i == 0)
            dc.add(_compare_step(out, rec, wl, fp32=False))
            uc.add(_compare_unmask(out, rec, wl, fp32=False))
    _report(f"{wl.name} {wl.model.n_layers} layers blocks {blocks}", dc, uc)
    # sharpened LM head: a fixed share of the argmax decisions lies outside the budget
    assert dc.checked >= 0.2 * dc.total
    return dc, uc


def test_llada_shape_2_layers_bf16(gpu):
    wl = sharpened(WORKLOADS["llada_gen256"], 30.0)
    wl = wl.replace(model=wl.model.with_layers(2))
    _bf16_case(wl, [(0, 2), (5, 2)])


def test_dream_shape_gqa_2_layers_bf16(gpu):
    wl = sharpened(WORKLOADS["dream_gen512"], 30.0)
    wl = wl.replace(model=wl.model.with_layers(2))
    _bf16_case(wl, [(0, 1), (14, 1)])


def test_llada_long_shape_2_layers_bf16(gpu):
    wl = sharpened(WORKLOADS["llada_long2048"], 30.0)
    wl = wl.replace(model=wl.model.with_layers(2))
    _bf16_case(wl, [(0, 2), (31, 2)])


def test_llada_long_shape_2_layers_single_bf16_activations(gpu):
    """SSM_ACT_BF16 (projection inputs rounded once to bfloat16, one MFMA pass):
    the 1264-row block-start step runs the big-tile GEMM without the lo part,
    the 240-row cached step the 128-row kernel without it.  Two layers keep the
    single rounding well inside the bound."""
    from paper_2608_23167_amd import _lib as L
    wl = sharpened(WORKLOADS["llada_long2048"], 30.0)
    wl = wl.replace(model=wl.model.with_layers(2))
    _bf16_case(wl, [(0, 2)], act_mode=L.SSM_ACT_BF16)


@pytest.mark.parametrize("batch", [1, 2])
def test_llada_shape_one_pass_512_and_1024_rows(gpu, batch):
    """One-pass (SSM_ACT_BF16) block-start step of block 5 of the gen-256
    workload: 512 rows per sequence.  At batch 1 gate/up runs the 3-stage
    256 x 128 tiles and QKV, O, down the 128-row kernel; at batch 2 (1024
    rows) QKV the 256 x 128 tiles, gate/up the 256 x 256 tiles, O and down
    the 256 x 256 tiles with split-K."""
    from paper_2608_23167_amd import _lib as L
    wl = sharpened(WORKLOADS["llada_gen256"], 30.0)
    wl = wl.replace(model=wl.model.with_layers(2), batch=batch)
    _bf16_case(wl, [(5, 1)], act_mode=L.SSM_ACT_BF16)


def test_llada_long_shape_pair_in_first_layer_only(gpu):
    """SSM_ACT_BF16X2_FIRST with one pair layer: layer 0 multiplies the hi and
    lo parts, layer 1 and the LM head round once, on both the block-start
    (1264 rows, big tiles) and the cached (240 rows) launch paths."""
    from paper_2608_23167_amd import _lib as L
    wl = sharpened(WORKLOADS["llada_long2048"], 30.0)
    wl = wl.replace(model=wl.model.with_layers(2))
    _bf16_case(wl, [(0, 2)], act_mode=L.SSM_ACT_BF16X2_FIRST, pair_layers=1)


def test_llada_long1024_block_start_1776_rows_2_layers_bf16(gpu):
    """Block-start step of block 8 of the gen-1024 long workload: 1776 rows, a
    ragged last tile for both the 256-row (gate/up: 256 x 256, 3-stage ring)
    and the 128-row (O/down: 128 x 256, 3-stage ring) big-tile GEMMs."""
    wl = sharpened(WORKLOADS["llada_long1024"], 30.0)
    wl = wl.replace(model=wl.model.with_layers(2))
    _bf16_case(wl, [(8, 1)])
