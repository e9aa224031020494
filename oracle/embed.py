"""Soft suffix embedding mixing (Section 3.2, "Soft Suffix Embedding Mixing", Eq. 6-8).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Readings taken where the paper is silent:
  * p_{t+1}^i is the softmax, at temperature 1, of the final logits of
    position i at the previous step, with the [MASK] id excluded from the
    vocabulary (its logit is treated as -inf).
  * Top-k order: larger probability first, the lower token id on ties.
  * Only a prediction made at the immediately preceding step counts as
    p_{t+1}; a retained suffix position without one (the first step of a
    generation, or a position that was not an output row at the previous
    step) is embedded as the plain [MASK] embedding.
  * Masked positions of the current block are not mixed: Eq. 8 is stated for
    retained suffix positions only.
"""
from __future__ import annotations

from typing import Tuple

import numpy as np

from .selection import REGION_LOCAL


def full_softmax(logits: np.ndarray, exclude_id: int) -> np.ndarray:
    """p(v) over the vocabulary for one row, with `exclude_id` removed."""
    l = np.array(logits, dtype=np.float64)
    if 0 <= exclude_id < l.shape[-1]:
        l[..., exclude_id] = -np.inf
    m = np.max(l, axis=-1, keepdims=True)
    e = np.exp(l - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def top_k_set(p: np.ndarray, k: int) -> np.ndarray:
    """T_{t+1}^i: ids of the k most probable tokens (lower id first on ties)."""
    order = np.argsort(-p, kind="stable")
    return order[:k]


def renormalise(p: np.ndarray, ids: np.ndarray) -> np.ndarray:
    """Eq. 6: p~(v) = p(v) / sum_{u in T} p(u) for v in T."""
    sel = p[ids]
    return sel / np.sum(sel)


def topk_renormalised(logits_row: np.ndarray, k: int, mask_id: int) -> Tuple[np.ndarray, np.ndarray]:
    """T and p~ of Eq. 6 for one row of final logits."""
    p = full_softmax(logits_row, mask_id)
    ids = top_k_set(p, k)
    return ids.astype(np.int32), renormalise(p, ids)


def soft_decoded_embedding(E: np.ndarray, ids: np.ndarray, w: np.ndarray) -> np.ndarray:
    """Eq. 7: e~ = sum_{v in T} p~(v) e_v."""
    out = np.zeros(E.shape[1], dtype=E.dtype)
    for v, wv in zip(ids, w):
        out = out + wv * E[v]
    return out


def mix(e_mask: np.ndarray, e_soft: np.ndarray, alpha: float) -> np.ndarray:
    """Eq. 8: (1 - alpha) e_mask + alpha e~."""
    return (1.0 - alpha) * e_mask + alpha * e_soft


def embed_rows(E: np.ndarray, tokens: np.ndarray, pos: np.ndarray, region: np.ndarray,
               pred_ids: np.ndarray, pred_w: np.ndarray, pred_step: np.ndarray,
               prev_step: int, alpha: float, mask_id: int) -> np.ndarray:
    """Input embeddings of the compacted rows of one sequence.

    tokens: [L_tot] ids; pos/region: the compacted row list; pred_*: the
    per-position prediction state ([L_tot, k], [L_tot, k], [L_tot]).  Rows of
    the prefix and the block use E[x_p]; retained suffix rows use Eq. 7-8
    when a prediction from `prev_step` exists, E[mask] otherwise.
    """
    n = len(pos)
    x = np.zeros((n, E.shape[1]), dtype=E.dtype)
    for r in range(n):
        p = int(pos[r])
        if region[r] >= REGION_LOCAL and pred_step[p] == prev_step and prev_step >= 0:
            e_soft = soft_decoded_embedding(E, pred_ids[p], pred_w[p])
            x[r] = mix(E[mask_id], e_soft, alpha)
        else:
            x[r] = E[int(tokens[p])]
    return x
