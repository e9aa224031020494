"""Pins of the oracle's soft suffix embedding (Section 3.2, Eq. 6-8)."""
import numpy as np
import pytest

from oracle import embed as E
from oracle import selection as S

rng = np.random.default_rng(1234)


def test_alpha_zero_is_mask_embedding():
    Emb = rng.normal(size=(50, 16))
    ids = np.array([3, 7, 9])
    w = np.array([0.5, 0.3, 0.2])
    out = E.mix(Emb[49], E.soft_decoded_embedding(Emb, ids, w), 0.0)
    assert np.array_equal(out, Emb[49])


def test_k1_alpha1_is_argmax_embedding():
    Emb = rng.normal(size=(50, 16))
    logits = rng.normal(size=50)
    ids, w = E.topk_renormalised(logits, 1, mask_id=49)
    assert w[0] == 1.0
    assert ids[0] == int(np.argmax(logits[:49]))
    out = E.mix(Emb[49], E.soft_decoded_embedding(Emb, ids, w), 1.0)
    assert np.allclose(out, Emb[ids[0]], rtol=0, atol=0)


def test_mix_is_affine_in_alpha():
    Emb = rng.normal(size=(20, 8))
    a, s = Emb[19], Emb[:3].mean(0)
    for alpha in (0.2, 0.4, 0.7):
        assert np.allclose(E.mix(a, s, alpha), a + alpha * (s - a), atol=1e-15)


def test_renormalised_weights_sum_to_one_and_order():
    for _ in range(50):
        logits = rng.normal(size=300) * 3
        for k in (1, 3, 5, 7, 8):
            ids, w = E.topk_renormalised(logits, k, mask_id=299)
            assert abs(w.sum() - 1.0) < 1e-12
            assert np.all(np.diff(w) <= 0)
            assert 299 not in ids


def test_eq6_equals_softmax_over_topk_logits():
    """p(v)/sum_T p(u) = exp(l_v)/sum_T exp(l_u): the full-vocabulary
    normaliser cancels, so Eq. 6 needs only the k largest logits."""
    for _ in range(50):
        logits = rng.normal(size=1000) * 2
        mask = 999
        ids, w = E.topk_renormalised(logits, 5, mask)
        # independent: sort logits by brute force, softmax over the top 5
        cand = [(-logits[v], v) for v in range(1000) if v != mask]
        cand.sort()
        top = [v for _, v in cand[:5]]
        assert list(ids) == top
        l = np.array([logits[v] for v in top])
        ref = np.exp(l - l.max()) / np.exp(l - l.max()).sum()
        assert np.max(np.abs(w - ref)) < 1e-12


def test_topk_tie_break_lower_id():
    logits = np.zeros(10)
    logits[[2, 5, 7]] = 1.0
    ids, w = E.topk_renormalised(logits, 2, mask_id=9)
    assert list(ids) == [2, 5]
    assert np.allclose(w, [0.5, 0.5])


def test_mask_excluded_from_prediction():
    logits = np.zeros(10)
    logits[9] = 100.0   # the mask id has by far the largest logit
    ids, _ = E.topk_renormalised(logits, 3, mask_id=9)
    assert 9 not in ids


def test_embed_rows_rules():
    V, d, L, k = 40, 6, 20, 3
    Emb = rng.normal(size=(V, d))
    mask = V - 1
    tokens = np.array([1, 2, 3, 4] + [mask] * 16)
    pos = np.array([0, 1, 2, 3, 4, 5, 6, 7, 12, 19])
    region = np.array([S.REGION_PREFIX] * 4 + [S.REGION_BLOCK] * 4 + [S.REGION_MIDDLE, S.REGION_TAIL])
    pred_ids = np.zeros((L, k), np.int32)
    pred_w = np.zeros((L, k))
    pred_step = np.full(L, -1)
    pred_ids[12] = [5, 6, 7]
    pred_w[12] = [0.5, 0.3, 0.2]
    pred_step[12] = 4
    pred_ids[19] = [8, 9, 10]
    pred_w[19] = [0.6, 0.3, 0.1]
    pred_step[19] = 3        # stale: not the previous step
    pred_step[5] = 4         # block rows are never mixed
    pred_ids[5] = [1, 1, 1]
    pred_w[5] = [1, 0, 0]
    x = E.embed_rows(Emb, tokens, pos, region, pred_ids, pred_w, pred_step, 4, 0.4, mask)
    for r in range(4):
        assert np.array_equal(x[r], Emb[tokens[r]])
    for r in range(4, 8):
        assert np.array_equal(x[r], Emb[mask])
    want = 0.6 * Emb[mask] + 0.4 * (0.5 * Emb[5] + 0.3 * Emb[6] + 0.2 * Emb[7])
    assert np.allclose(x[8], want, atol=1e-14)
    assert np.array_equal(x[9], Emb[mask])
    # no previous step at all
    x0 = E.embed_rows(Emb, tokens, pos, region, pred_ids, pred_w, pred_step, -1, 0.4, mask)
    assert np.array_equal(x0[8], Emb[mask])
