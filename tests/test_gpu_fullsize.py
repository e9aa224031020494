"""Full-size GPU step parity: every layer of the LLaDA-8B and Dream-7B shapes
in bf16 against the float32 oracle on the same bf16-rounded weights, in the
launch configuration the benchmark uses (teacher-forced steps).

Cached steps read a seeded synthetic prefix cache that both sides share, so
a cached step is checked without an oracle block-start step first.

The LM head is sharpened (logit scale 30, both sides) so that argmax
decisions have probability margins above 1e-3: each test asserts that some
are checked under the fixed error budget of tests/_parity.py.  At random
initialisation the masked rows of a block are near-identical, so their
confidences nearly tie and no unmasking comparison lies outside the budget;
the unmasking stage is then checked for consistency instead: the rule applied
to the GPU's own confidences must pick exactly the GPU's positions.
"""
import time

import numpy as np
import pytest
import torch

import oracle.generate as OG
from synthetic import WORKLOADS, make_weights, mid_generation_state
from tests._parity import (check_decisions, check_unmask, check_unmask_consistency, gpu_step,
                           load_oracle_state, put_synthetic_cache, rel_err)

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

TOL = 2e-2
LOGIT_SCALE = 30.0


def _state(wl, block_idx, step, seed):
    t, pi, pw, ps = mid_generation_state(wl, block_idx, step, seed)
    st = OG.OracleState.start(t, wl.topk)
    st.pred_ids[:] = pi
    st.pred_w[:] = pw
    st.pred_step[:] = ps
    st.step = step
    return st


class _Model:
    def __init__(self, wl):
        from paper_2608_23167_amd.model import DeviceModel
        t0 = time.time()
        self.mw = make_weights(wl.model, seed=wl.seed, device="cuda", logit_scale=LOGIT_SCALE)
        self.dm = DeviceModel(wl.model, self.mw)
        self.w = OG.NumpyWeights(self.mw, dtype=np.float32)
        print(f"[fullsize] weights of {wl.model.name} ready in {time.time() - t0:.1f} s", flush=True)


@pytest.fixture(scope="module")
def llada():
    m = _Model(WORKLOADS["llada_gen256"])
    yield m
    del m


def _run(wl, model, block_idx, first, seed, synthetic_cache):
    from paper_2608_23167_amd.decoder import Decoder
    dec = Decoder(wl, model.dm)
    st = _state(wl, block_idx, 4 + block_idx, seed)
    if synthetic_cache:
        put_synthetic_cache(dec, st, wl.prompt_len + block_idx * wl.block_size, seed)
    before = st.copy()
    t0 = time.time()
    rec = OG.step(wl, model.w, st, block_idx, first)
    t_or = time.time() - t0
    load_oracle_state(dec, before)
    out = gpu_step(dec, block_idx, first)
    e_h = rel_err(out["hidden"], rec.hidden)
    e_l = max(rel_err(out["logits"][s], rec.stats[s].logits) for s in range(wl.batch))
    dc = check_decisions(out, rec, wl, fp32=False)
    uc = check_unmask(out, rec, wl, fp32=False)
    n_cons = check_unmask_consistency(out, rec, wl)
    print(f"[fullsize] {wl.name} block {block_idx} {'start' if first else 'cached'} rows "
          f"{out['info'].n_rows}: hidden rel {e_h:.2e} logits rel {e_l:.2e}; argmax {dc}; "
          f"unmask {uc}; unmask consistency {n_cons} (oracle {t_or:.1f} s)", flush=True)
    assert np.array_equal(out["pos"], rec.rows.pos)
    assert e_h < TOL and e_l < TOL
    assert dc.checked > 0
    del dec
    torch.cuda.empty_cache()


def test_llada_gen256_block_start(gpu, llada):
    _run(WORKLOADS["llada_gen256"], llada, 0, True, 1, False)


def test_llada_gen256_cached(gpu, llada):
    _run(WORKLOADS["llada_gen256"], llada, 3, False, 2, True)


def test_llada_long_cached(gpu, llada):
    _run(WORKLOADS["llada_long2048"], llada, 0, False, 3, True)


def test_llada_long_block_start(gpu, llada):
    _run(WORKLOADS["llada_long2048"], llada, 0, True, 4, False)


def test_llada_long_late_block_cached(gpu, llada):
    """Block 20 of the gen-2048 long workload: 1280 cached prefix keys plus the
    block and its retained suffix."""
    _run(WORKLOADS["llada_long2048"], llada, 20, False, 6, True)


def test_llada_long_last_block_cached(gpu, llada):
    """The last block of the gen-2048 long workload: prefix 3008 (cached), no
    suffix left, 64 query rows over 3072 keys."""
    _run(WORKLOADS["llada_long2048"], llada, 31, False, 7, True)


def test_llada_long1024_block_start_1776_rows(gpu, llada):
    """The block-start step on which the MFMA fraction is reported: block 8 of
    the gen-1024 long workload, prefix 1536 + block 64 + 176 retained suffix
    rows = 1776 rows through all 32 layers (big-tile GEMMs with ragged last
    tiles, long-key attention)."""
    _run(WORKLOADS["llada_long1024"], llada, 8, True, 8, False)


def test_llada_gen256_cached_pair_in_every_layer(gpu, llada):
    """SSM_ACT_BF16X2: the bfloat16 pair at the projections of all 32 layers
    and the LM head (the default keeps it in the first layers only)."""
    from paper_2608_23167_amd import _lib as L
    from paper_2608_23167_amd.model import DeviceModel
    wl = WORKLOADS["llada_gen256"]
    paired = type(llada).__new__(type(llada))
    paired.mw, paired.w = llada.mw, llada.w
    paired.dm = DeviceModel(wl.model, llada.mw, act_mode=L.SSM_ACT_BF16X2)
    _run(wl, paired, 3, False, 2, True)


@pytest.fixture(scope="module")
def dream():
    m = _Model(WORKLOADS["dream_gen512"])
    yield m
    del m


def test_dream_uncached(gpu, dream):
    _run(WORKLOADS["dream_gen512"], dream, 0, True, 5, False)


def test_dream_last_block_uncached(gpu, dream):
    """The last block of the Dream-7B workload (no cache): prefix 992 + block
    32 = 1024 rows, no suffix left."""
    _run(WORKLOADS["dream_gen512"], dream, 15, True, 9, False)


@pytest.mark.parametrize("gen,block,first,seed", [(256, 1, True, 10), (512, 3, False, 11)])
def test_llada_gen_sweep_lengths(gpu, llada, gen, block, first, seed):
    """The generation-length sweep's workloads (prompt 1024, block 64, top-8,
    budgets 128/32/16, prefix cache) at the lengths no other full-depth test
    covers: gen 256 (block-start step of block 1: prefix 1088, the two
    remaining suffix blocks all local) and gen 512 (cached step of block 3,
    prefix 1216 cached).  Gen 1024 and 2048 are the long workloads above."""
    wl = WORKLOADS["llada_long2048"].replace(gen_len=gen)
    _run(wl, llada, block, first, seed, not first)
