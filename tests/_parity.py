"""Shared helpers of the GPU parity tests (not collected by pytest)."""
from __future__ import annotations

import numpy as np
import torch

import oracle.generate as OG


def rel_err(gpu, ref) -> float:
    g = np.asarray(gpu, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-30))


def max_abs(gpu, ref) -> float:
    return float(np.max(np.abs(np.asarray(gpu, np.float64) - np.asarray(ref, np.float64))))


def load_oracle_state(dec, st: OG.OracleState) -> None:
    """Teacher forcing: put the oracle's state before a step into the decoder."""
    dev = dec.tokens.device
    dec.tokens.copy_(torch.from_numpy(st.tokens.astype(np.int32)).to(dev))
    dec.pred_ids.copy_(torch.from_numpy(st.pred_ids.astype(np.int32)).to(dev))
    dec.pred_w.copy_(torch.from_numpy(st.pred_w.astype(np.float32)).to(dev))
    dec.pred_step.copy_(torch.from_numpy(st.pred_step.astype(np.int32)).to(dev))
    dec.step_idx = st.step


def gpu_step(dec, block_idx, first, want_logits=True, want_hidden=True):
    """Runs one decoder step and returns host copies of everything it produced."""
    wl = dec.wl
    B, V, d, k = wl.batch, wl.model.vocab, wl.model.d_model, wl.topk
    logits = torch.empty(B * dec.max_rows * V, dtype=torch.float32, device=dec.tokens.device) if want_logits else None
    hidden = torch.empty(B * dec.max_rows * d, dtype=torch.float32, device=dec.tokens.device) if want_hidden else None
    info = dec.step(block_idx, first, logits=logits, hidden=hidden)
    torch.cuda.synchronize()
    n, no = info.n_rows, info.n_out
    out = {
        "info": info,
        "pos": dec.pos[:n].cpu().numpy(),
        "region": dec.region[:n].cpu().numpy(),
        "tok_c": dec.tok_c[:, :n].cpu().numpy(),
        "x": dec.x[:B * n * d].view(B, n, d).cpu().numpy(),
        "argmax": dec.argmax[:B * no].view(B, no).cpu().numpy(),
        "conf": dec.conf[:B * no].view(B, no).cpu().numpy(),
        "topk_ids": dec.topk_ids[:B * no * k].view(B, no, k).cpu().numpy(),
        "topk_w": dec.topk_w[:B * no * k].view(B, no, k).cpu().numpy(),
        "tokens": dec.tokens.cpu().numpy(),
        "selected": dec.selected[:B * wl.block_size].view(B, wl.block_size).cpu().numpy().astype(bool),
    }
    if want_logits:
        out["logits"] = logits[:B * no * V].view(B, no, V).cpu().numpy()
    if want_hidden:
        out["hidden"] = hidden[:B * n * d].view(B, n, d).cpu().numpy()
    return out


def decision_margins(stats):
    """Per output row: p1 - p2 (argmax margin)."""
    return stats.p_sorted2[:, 0] - stats.p_sorted2[:, 1]


def check_decisions(gpu, rec, wl, tol):
    """Argmax, top-k ids and unmasking decisions must agree wherever the
    oracle's margin exceeds `tol`; returns the fraction of decisions pinned."""
    pinned = total = 0
    b = wl.block_size
    for s, stats in enumerate(rec.stats):
        m = decision_margins(stats)
        wide = m > tol
        assert np.array_equal(gpu["argmax"][s][wide], stats.argmax[wide]), "argmax mismatch"
        # top-k ids: compare the prefix of the list whose consecutive gaps are wide
        p = np.exp(stats.logits - stats.logits.max(axis=1, keepdims=True))
        p[:, wl.model.mask_id] = 0
        p = p / p.sum(axis=1, keepdims=True)
        for r in range(len(m)):
            ids = stats.topk_ids[r]
            pv = p[r, ids]
            for i in range(wl.topk):
                nxt = np.sort(p[r])[::-1][i + 1] if i + 1 < p.shape[1] else 0.0
                if pv[i] - nxt <= tol:
                    break
                assert gpu["topk_ids"][s][r, i] == ids[i], f"top-k id mismatch row {r} rank {i}"
        pinned += int(wide.sum())
        total += len(m)
    return pinned / max(total, 1)
