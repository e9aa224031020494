"""Pins of the oracle's unmasking rules (Section 4.2) and generation loop (Section 3.2)."""
import itertools

import numpy as np
import pytest

from oracle import model as M
from oracle import selection as S
from oracle import unmask as U
from oracle import generate as G
from synthetic import WORKLOADS, TINY, make_weights, initial_tokens, sharpened, spread

rng = np.random.default_rng(11)


def test_topn_brute_force():
    for _ in range(200):
        b = 8
        conf = rng.random(b)
        masked = rng.random(b) < 0.7
        n = int(rng.integers(1, 9))
        sel = U.choose(conf, masked, U.TOPN, n)
        cands = [i for i in range(b) if masked[i]]
        m = min(n, len(cands))
        # brute force: the chosen subset has the largest total confidence among all m-subsets
        best = max(itertools.combinations(cands, m), key=lambda c: sum(conf[i] for i in c), default=())
        assert set(np.nonzero(sel)[0]) == set(best)
        assert not np.any(sel & ~masked)


def test_threshold_rules():
    conf = np.array([0.2, 0.95, 0.91, 0.5, 0.99])
    masked = np.array([True, True, True, True, False])
    assert list(U.choose(conf, masked, U.THRESHOLD, threshold=0.9)) == [False, True, True, False, False]
    # none above: only the most confident candidate
    assert list(U.choose(conf, masked, U.THRESHOLD, threshold=0.97)) == [False, True, False, False, False]
    # threshold 0: every candidate; threshold >= 1: exactly one
    assert U.choose(conf, masked, U.THRESHOLD, threshold=0.0).sum() == 4
    assert U.choose(conf, masked, U.THRESHOLD, threshold=1.0).sum() == 1
    # strict comparison
    assert not U.choose(np.array([0.9, 0.1]), np.array([True, True]), U.THRESHOLD, threshold=0.9)[1]


def test_ties_and_full_block():
    conf = np.array([0.5, 0.7, 0.7, 0.7])
    masked = np.ones(4, bool)
    assert list(U.choose(conf, masked, U.TOPN, 2)) == [False, True, True, False]
    assert U.choose(conf, masked, U.TOPN, 4).all()
    assert not U.choose(conf, np.zeros(4, bool), U.TOPN, 4).any()


def _tiny_wl(**kw):
    return WORKLOADS["tiny"].replace(**kw)


def test_tiny_trajectory_invariants():
    wl = _tiny_wl()
    w = G.NumpyWeights(make_weights(wl.model, seed=0))
    st, recs = G.generate(wl, w, initial_tokens(wl).numpy(), keep=False)
    assert len(recs) == wl.n_blocks * (wl.block_size // wl.n_per_step)
    assert not np.any(st.tokens == wl.model.mask_id)
    prompt = initial_tokens(wl).numpy()[:, :wl.prompt_len]
    assert np.array_equal(st.tokens[:, :wl.prompt_len], prompt)
    # every step decodes exactly n tokens of its own block
    for r in recs:
        assert r.selected.sum() == wl.n_per_step


def _unpruned_step_logits(wl, w, tokens, block_idx):
    """Standard block-wise decoding input [P; B_t; S_t] with plain [MASK]
    embeddings: every position of the sequence, no selection at all."""
    L = wl.total_len
    pos = np.arange(L)
    x = w.tok_emb[tokens]
    h = M.forward(x, pos, w, wl.model).hidden
    P = wl.prompt_len + block_idx * wl.block_size
    return M.output_stats(h[P:], w, wl.model, wl.topk)


def test_full_budgets_equal_unpruned_forward():
    wl = _tiny_wl(local_budget=10**6, middle_budget=10**6, tail_budget=10**6, alpha=0.0)
    w = G.NumpyWeights(make_weights(wl.model, seed=1, norm_jitter=0.1))
    tok0 = initial_tokens(wl, seed=5).numpy()
    st = G.OracleState.start(tok0, wl.topk)
    for j, first in [(0, True), (0, False), (1, True), (2, True)]:
        ref = _unpruned_step_logits(wl, w, st.tokens[0].copy(), j)
        rec = G.step(wl, w, st, j, first)
        assert np.max(np.abs(rec.stats[0].logits - ref.logits)) < 1e-12


def test_zero_budgets_equal_prefix_block_forward():
    wl = _tiny_wl(local_budget=0, middle_budget=0, tail_budget=0)
    w = G.NumpyWeights(make_weights(wl.model, seed=2, norm_jitter=0.1))
    tok0 = initial_tokens(wl, seed=6).numpy()
    st = G.OracleState.start(tok0, wl.topk)
    for j in range(3):
        P = wl.prompt_len + j * wl.block_size
        toks = st.tokens[0, :P + wl.block_size].copy()
        h = M.forward(w.tok_emb[toks], np.arange(P + wl.block_size), w, wl.model).hidden
        ref = M.output_stats(h[P:], w, wl.model, wl.topk)
        rec = G.step(wl, w, st, j, True)
        assert rec.rows.n_suffix == 0
        assert np.max(np.abs(rec.stats[0].logits - ref.logits)) < 1e-12


def test_cached_step_equals_uncached_when_nothing_changed():
    """Right after a block-start step, a cached step over unchanged inputs
    reproduces the block-start step's outputs."""
    wl = _tiny_wl(cache=True, alpha=0.0)
    w = G.NumpyWeights(make_weights(wl.model, seed=4, norm_jitter=0.1))
    tok0 = initial_tokens(wl, seed=7).numpy()
    st = G.OracleState.start(tok0, wl.topk)
    rec0 = G.step(wl, w, st.copy(), 1, True)       # block-start over the same tokens
    st1 = st.copy()
    G.step(wl, w, st1, 1, True)
    st1.tokens = st.tokens.copy()                  # undo the unmasking
    rec1 = G.step(wl, w, st1, 1, False)
    assert not rec1.include_prefix
    assert np.max(np.abs(rec1.stats[0].logits - rec0.stats[0].logits)) < 1e-12


def test_soft_embedding_used_on_next_step():
    wl = _tiny_wl()
    w = G.NumpyWeights(make_weights(wl.model, seed=0))
    st = G.OracleState.start(initial_tokens(wl).numpy(), wl.topk)
    rec0 = G.step(wl, w, st, 0, True)
    rec1 = G.step(wl, w, st, 0, False)
    rows = rec1.rows
    mask_e = w.tok_emb[wl.model.mask_id]
    suffix = rows.region >= S.REGION_LOCAL
    # every retained suffix row now differs from the plain mask embedding
    assert all(not np.allclose(rec1.x[0, r], mask_e) for r in np.nonzero(suffix)[0])
    # and equals Eq. 8 with the previous step's top-k
    r = int(np.nonzero(suffix)[0][0])
    o = r - rec0.rows.first_out_row
    ids, wts = rec0.stats[0].topk_ids[o], rec0.stats[0].topk_w[o]
    want = (1 - wl.alpha) * mask_e + wl.alpha * (wts[:, None] * w.tok_emb[ids]).sum(0)
    assert np.allclose(rec1.x[0, r], want, atol=1e-14)


def test_threshold_workload_terminates():
    wl = _tiny_wl(rule="threshold", threshold=0.9)
    w = G.NumpyWeights(make_weights(wl.model, seed=0))
    st, recs = G.generate(wl, w, initial_tokens(wl).numpy())
    assert not np.any(st.tokens == wl.model.mask_id)
    assert len(recs) >= wl.n_blocks


def test_early_stop_fill_rule():
    """Early termination after a block (Section 3.2; fill rule of Section 4.4):
    only sequences whose block holds the end id are filled from the block's end
    on; a sequence already done is left alone; all done -> True."""
    eos, b, L = 9, 4, 20
    tok = np.arange(3 * L, dtype=np.int32).reshape(3, L) % 7 + 100
    tok[0, 5] = eos                      # in block [4, 8) of sequence 0
    tok[2, 13] = eos                     # in a later block of sequence 2
    done = np.zeros(3, dtype=bool)
    before = tok.copy()
    assert not G.early_stop(tok, done, 4, b, eos)
    assert list(done) == [True, False, False]
    assert np.all(tok[0, 8:] == eos) and np.array_equal(tok[0, :8], before[0, :8])
    assert np.array_equal(tok[1:], before[1:])
    # block [12, 16): sequence 2 ends; sequence 0 is done already
    tok[0, 8:] = 3                       # a done sequence is not touched again
    assert not G.early_stop(tok, done, 12, b, eos)
    assert list(done) == [True, False, True]
    assert np.all(tok[0, 8:] == 3)
    assert np.all(tok[2, 16:] == eos) and tok[2, 13] == eos
    tok[1, 19] = eos                     # the last block: nothing after it to fill
    assert G.early_stop(tok, done, 16, b, eos)
    assert list(done) == [True, True, True]


def _eos_model(wl, eos, boost):
    mw = make_weights(wl.model, seed=0, norm_jitter=0.1)
    mw.lm_head[eos] *= boost             # the end id wins wherever h . w_eos > 0
    return mw


def test_early_termination_stops_generation():
    """With an end id that the model decodes in the first block, the generation
    ends after that block: later blocks are all end ids and are never run; the
    decoded first block equals that of the run without early termination."""
    eos = 7
    wl = WORKLOADS["tiny"].replace(batch=2)
    mw = _eos_model(wl, eos, 40.0)
    w = G.NumpyWeights(mw)
    tok0 = initial_tokens(wl).numpy()
    st_on, recs_on = G.generate(wl.replace(eos_id=eos), w, tok0)
    st_off, recs_off = G.generate(wl, w, tok0)
    spb = wl.steps_per_block()
    blk_end = wl.prompt_len + wl.block_size
    assert np.all(st_on.tokens[:, wl.prompt_len:blk_end] != wl.model.mask_id)
    assert np.all(np.any(st_on.tokens[:, wl.prompt_len:blk_end] == eos, axis=1))
    assert len(recs_on) == spb and len(recs_off) == wl.n_blocks * spb
    assert np.all(st_on.tokens[:, blk_end:] == eos) and np.all(st_on.done)
    assert np.array_equal(st_on.tokens[:, :blk_end], st_off.tokens[:, :blk_end])
    # an end id the model never decodes changes nothing
    st_none, recs_none = G.generate(wl.replace(eos_id=wl.model.mask_id), w, tok0)
    assert len(recs_none) == len(recs_off) and np.array_equal(st_none.tokens, st_off.tokens)


def _two_largest_scalar(logits, mask_id):
    """p1, p2 of one row from the softmax written out with math.exp ([MASK] excluded)."""
    import math
    vals = [float(v) for i, v in enumerate(logits) if i != mask_id]
    m = max(vals)
    z = sum(math.exp(v - m) for v in vals)
    p = sorted((math.exp(v - m) / z for v in vals), reverse=True)
    return p[0], p[1]


def _margin_brute(margin, masked, tau):
    """Margin rule (Section 4.6, Table 3) by enumeration: every candidate whose
    top-1/top-2 gap exceeds tau; if there is none, the single widest (lower
    position on ties)."""
    cand = [i for i in range(len(margin)) if masked[i]]
    chosen = {i for i in cand if margin[i] > tau}
    if not chosen and cand:
        best = cand[0]
        for i in cand[1:]:
            if margin[i] > margin[best]:
                best = i
        chosen = {best}
    return chosen


def test_margin_rule_brute_force():
    """choose(..., MARGIN) against enumeration, with margins p1 - p2 taken
    from the full softmax of random logit rows."""
    r = np.random.default_rng(21)
    for _ in range(300):
        b, V = 8, 12
        logits = r.normal(size=(b, V)) * r.uniform(0.5, 4.0)
        margin = np.array([np.subtract(*_two_largest_scalar(l, V - 1)) for l in logits])
        masked = r.random(b) < 0.7
        tau = float(r.choice([0.0, 0.05, 0.2, 0.5, 0.9, 1.0, 1.5]))
        sel = U.choose(np.zeros(b), masked, U.MARGIN, threshold=tau, margin=margin)
        assert set(np.nonzero(sel)[0]) == _margin_brute(margin, masked, tau)
        assert not np.any(sel & ~masked)


def test_margin_rule_special_cases():
    masked = np.array([True, True, False, True, True])
    margin = np.array([0.30, 0.05, 0.90, 0.30, 0.01])
    # tau = 0: every candidate with a positive margin
    assert list(U.choose(np.zeros(5), masked, U.MARGIN, threshold=0.0, margin=margin)) == \
        [True, True, False, True, True]
    # tau >= 1: no margin exceeds it (p1 - p2 <= 1): exactly one, the widest,
    # the lower position on ties (0.30 at positions 0 and 3)
    for tau in (1.0, 2.0):
        assert list(U.choose(np.zeros(5), masked, U.MARGIN, threshold=tau, margin=margin)) == \
            [True, False, False, False, False]
    # strict comparison; the confidence plays no part in the margin rule
    sel = U.choose(np.array([0.99, 0.0, 0.0, 0.0, 0.0]), masked, U.MARGIN, threshold=0.30,
                   margin=margin)
    assert list(sel) == [True, False, False, False, False]        # fallback: none > 0.30
    sel = U.choose(np.zeros(5), masked, U.MARGIN, threshold=0.2, margin=margin)
    assert list(sel) == [True, False, False, True, False]
    # no candidate left: nothing is decoded
    assert not U.choose(np.zeros(5), np.zeros(5, bool), U.MARGIN, threshold=0.0, margin=margin).any()


def test_margin_step_decodes_by_top_two_gap():
    """A whole step of the tiny model under the margin rule: the positions the
    oracle decodes are those the enumeration picks from p1 - p2 recomputed
    from the step's logits, and each gets its argmax."""
    wl = spread(_tiny_wl(rule="margin", threshold=0.5), init_std=0.2)
    w = G.NumpyWeights(make_weights(wl.model, seed=0, norm_jitter=0.1, logit_scale=wl.logit_scale))
    st = G.OracleState.start(initial_tokens(wl).numpy(), wl.topk)
    n_multi = 0
    for j, first in [(0, True), (0, False), (0, False), (1, True)]:
        P = wl.prompt_len + j * wl.block_size
        masked = st.tokens[0, P:P + wl.block_size] == wl.model.mask_id
        rec = G.step(wl, w, st, j, first)
        lg = rec.stats[0].logits[:wl.block_size]
        margin = np.array([np.subtract(*_two_largest_scalar(l, wl.model.mask_id)) for l in lg])
        want = _margin_brute(margin, masked, wl.threshold)
        assert set(np.nonzero(rec.selected[0])[0]) == want
        for i in want:
            assert st.tokens[0, P + i] == int(np.argmax(np.where(
                np.arange(wl.model.vocab) == wl.model.mask_id, -np.inf, lg[i])))
        n_multi += len(want) > 1
    assert n_multi > 0          # the threshold itself decided some step, not only the fallback
