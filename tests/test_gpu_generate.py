"""Free-running generations on the GPU against the oracle's.

Decoder.generate() chains select, embed, denoise and unmask over every step
with nothing copied from the oracle in between: step t's unmasking and
prediction-state scatter feed step t+1's selection and soft suffix embedding
(Section 3.2, Eq. 6-8), the threshold and margin rules read the count of
masks left on the host, and early termination (Section 3.2) ends the
generation.  The oracle's generation (oracle.generate.generate) runs the same
workload from the same prompt.

A free-running comparison is only meaningful where no decision along the way
is left to rounding.  Within one step the float32 path keeps the logits
within 1e-4 (the per-step tests), but over a generation the carried
prediction state (Eq. 6 weights, in float32 on the GPU) lets small
differences grow.  So each case first measures, on the oracle alone, how far
the same generation run in float32 NumPy drifts from the float64 one (the
largest logit difference over all steps, `drift`); it requires the two to
take the same trajectory, and every unmasking choice and the argmax of every
decoded position to lie outside the budget eps = max(1e-4, 4 drift) of the
rule in tests/_parity.py.  The cases (the tiny float32 workload's
wide-margin test variant; generation length 64 under the threshold and
margin rules, which take about one step per token) are ones that clear it.
Then the final tokens, the step count, the done flags and the prediction
stamps must be bit-identical, the prediction ids identical wherever their
rank is decided, and the prediction weights within 1e-5.
"""
import numpy as np
import pytest
import torch

import oracle.generate as OG
from synthetic import WORKLOADS, initial_tokens, make_weights, spread
from tests._parity import Counts, check_unmask, logit_budget

pytestmark = pytest.mark.gpu


def _oracle_as_gpu(rec):
    return {"argmax": [s.argmax for s in rec.stats], "topk_ids": [s.topk_ids for s in rec.stats],
            "selected": rec.selected, "tokens": rec.tokens_after}


def _decided_ranks(logits_row, mask_id, eps, k):
    """Leading top-k ranks whose gap to the next logit exceeds 2 eps."""
    l = np.array(logits_row, np.float64)
    l[mask_id] = -np.inf
    top = np.sort(l)[::-1][:k + 1]
    n = 0
    while n < k and top[n] - top[n + 1] > 2 * eps:
        n += 1
    return n


# name: (workload changes, token seed, end-id boost, generation ends early)
CASES = {
    "topn": (dict(), 0, None, False),
    "topn_cached": (dict(cache=True), 0, None, False),
    "threshold_0.5": (dict(rule="threshold", threshold=0.5, gen_len=64), 0, None, False),
    "threshold_0.5_cached": (dict(rule="threshold", threshold=0.5, gen_len=64, cache=True), 0,
                             None, False),
    "margin_0.5": (dict(rule="margin", threshold=0.5, gen_len=64), 0, None, False),
    "margin_0.5_cached": (dict(rule="margin", threshold=0.5, gen_len=64, cache=True), 0, None,
                          False),
    "margin_0.3_cached": (dict(rule="margin", threshold=0.3, gen_len=64, cache=True), 0, None,
                          False),
    # the sequence ends in block 1: the generation stops after 16 of 32 steps
    "early_stop": (dict(eos_id=7, cache=True), 3, 3.0, True),
    # one of two sequences ends in block 0 and is filled; the other runs on
    "early_stop_one_sequence": (dict(batch=2, eos_id=7, cache=True), 0, 2.0, False),
}


@pytest.mark.parametrize("case", list(CASES))
def test_free_running_generation(gpu, case):
    from paper_2608_23167_amd.decoder import Decoder
    from paper_2608_23167_amd.model import DeviceModel
    kw, tok_seed, boost, ends_early = CASES[case]
    wl = spread(WORKLOADS["tiny"]).replace(**kw)
    mw = make_weights(wl.model, seed=0, norm_jitter=0.1, logit_scale=wl.logit_scale)
    if boost is not None:
        mw.lm_head[wl.eos_id] *= boost        # the end id wins where its logit is large
    w = OG.NumpyWeights(mw)
    tok0 = initial_tokens(wl, seed=tok_seed)
    st, recs = OG.generate(wl, w, tok0.numpy(), keep=True)
    st32, recs32 = OG.generate(wl, OG.NumpyWeights(mw, dtype=np.float32), tok0.numpy(), keep=True)
    assert len(recs32) == len(recs) and np.array_equal(st32.tokens, st.tokens), \
        "the oracle's trajectory itself depends on float32 rounding"
    drift = max(float(np.max(np.abs(a.stats[s].logits - b.stats[s].logits)))
                for a, b in zip(recs, recs32) for s in range(wl.batch))
    eps = max(1e-4, 4.0 * drift)

    # precondition, on the oracle alone: no decision of the trajectory is inside the budget
    uc = Counts()
    for rec in recs:
        uc.add(check_unmask(_oracle_as_gpu(rec), rec, wl, fp32=True, eps=eps))
        for s in range(wl.batch):
            sts = rec.stats[s]
            for i in np.nonzero(rec.selected[s])[0]:
                assert _decided_ranks(sts.logits[i], wl.model.mask_id, eps, 1) == 1, \
                    f"argmax of a decoded position inside the budget at step {rec.step}"
    assert uc.inside == 0, f"{uc.inside} unmasking choices inside the budget"
    if wl.eos_id >= 0:
        assert st.done.any()
        assert (len(recs) < wl.n_blocks * wl.steps_per_block()) == ends_early == bool(st.done.all())

    dec = Decoder(wl, DeviceModel(wl.model, mw.to("cuda")))
    out = dec.generate(tok0.to("cuda"))
    torch.cuda.synchronize()
    print(f"[generate] {case}: {len(recs)} steps, GPU {dec.step_idx} steps; float32 drift "
          f"{drift:.1e}, budget {eps:.1e}", flush=True)
    assert dec.step_idx == len(recs)
    assert np.array_equal(out.cpu().numpy(), st.tokens)
    assert not np.any(st.tokens == wl.model.mask_id)
    if wl.eos_id >= 0:
        assert np.array_equal(dec.done.cpu().numpy().astype(bool), st.done)
    ps = dec.pred_step.cpu().numpy()
    assert np.array_equal(ps, st.pred_step)
    g_ids, g_w = dec.pred_ids.cpu().numpy(), dec.pred_w.cpu().numpy()
    n_ids = 0
    for rec in recs:                      # the step that wrote each final prediction
        rows = rec.rows
        out_pos = rows.pos[rows.first_out_row:]
        for s in range(wl.batch):
            sts = rec.stats[s]
            eps_r = logit_budget(sts.logits, wl.model.mask_id, True, eps)
            for r in range(wl.block_size, len(out_pos)):
                p = int(out_pos[r])
                if st.pred_step[s, p] != rec.step:
                    continue
                n = _decided_ranks(sts.logits[r], wl.model.mask_id, eps_r[r], wl.topk)
                assert np.array_equal(g_ids[s, p, :n], st.pred_ids[s, p, :n])
                if n == wl.topk:
                    assert np.max(np.abs(g_w[s, p] - st.pred_w[s, p])) < 1e-5
                n_ids += n
    assert n_ids > 0
