"""Full-size GPU step parity: every layer of the LLaDA-8B and Dream-7B shapes
in bf16 against the float32 oracle on the same bf16-rounded weights, in the
launch configuration the benchmark uses (teacher-forced steps).

Cached steps read a seeded synthetic prefix cache that both sides share, so
a cached step is checked without an oracle block-start step first.
"""
import time

import numpy as np
import pytest
import torch

import oracle.generate as OG
from synthetic import WORKLOADS, make_weights, mid_generation_state
from tests._parity import (check_decisions, check_unmask, gpu_step, load_oracle_state,
                           put_synthetic_cache, rel_err)

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

TOL = 2e-2


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
        self.mw = make_weights(wl.model, seed=wl.seed, device="cuda")
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
    pinned, total = check_decisions(out, rec, wl)
    n_unmask = check_unmask(out, rec, wl)
    print(f"[fullsize] {wl.name} block {block_idx} {'start' if first else 'cached'} rows "
          f"{out['info'].n_rows}: hidden rel {e_h:.2e} logits rel {e_l:.2e} pinned {pinned}/{total} "
          f"unmask-checked {n_unmask} (oracle {t_or:.1f} s)", flush=True)
    assert np.array_equal(out["pos"], rec.rows.pos)
    assert e_h < TOL and e_l < TOL
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


def test_dream_uncached(gpu):
    wl = WORKLOADS["dream_gen512"]
    m = _Model(wl)
    _run(wl, m, 0, True, 5, False)
