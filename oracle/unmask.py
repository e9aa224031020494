"""Confidence-based unmasking inside the current block (Section 4.2 baselines;
Section 4.6 margin rule, Table 3).

TEST INFRASTRUCTURE ONLY (see the package docstring).

  * top-n:      decode the n most confident masked positions (n = 1 is the
                paper's "Vanilla" top-1 decoding).
  * threshold:  decode every masked position whose confidence exceeds the
                threshold ("Par."); if none does, decode the single most
                confident one so that every step makes progress.
  * margin:     decode every masked position whose gap between the two most
                probable tokens exceeds the threshold; at least one.

Confidence is the maximum softmax probability with [MASK] excluded; ties go
to the lower position.  The comparison with the threshold is strict.
"""
from __future__ import annotations

import numpy as np

TOPN = "topn"
THRESHOLD = "threshold"
MARGIN = "margin"


def choose(conf: np.ndarray, masked: np.ndarray, rule: str, n_per_step: int = 1,
           threshold: float = 0.9, margin: np.ndarray | None = None) -> np.ndarray:
    """Boolean [b] of the block positions to decode at this step."""
    b = len(conf)
    sel = np.zeros(b, dtype=bool)
    cand = [i for i in range(b) if masked[i]]
    if not cand:
        return sel
    score = conf if rule != MARGIN else margin
    ranked = sorted(cand, key=lambda i: (-float(score[i]), i))
    if rule == TOPN:
        for i in ranked[:min(n_per_step, len(ranked))]:
            sel[i] = True
        return sel
    for i in cand:
        if score[i] > threshold:
            sel[i] = True
    if not sel.any():
        sel[ranked[0]] = True
    return sel
