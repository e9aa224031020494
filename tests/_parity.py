"""Shared helpers of the GPU parity tests (not collected by pytest)."""
from __future__ import annotations

import numpy as np
import torch

import oracle.generate as OG

# Decision rule of the parity tests.  A decision (argmax, a top-k rank, an
# unmasking choice) must be identical on both sides when
#   (a) the oracle's probability margin exceeds PROB_MARGIN, and
#   (b) the oracle's logit gap exceeds ERR_FACTOR times the largest logit
#       difference between the two sides on that row -- a gap smaller than
#       the measured error is not decided by the arithmetic of either side.
PROB_MARGIN = 1e-3
ERR_FACTOR = 2.0


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
    dev = dec.tokens.device
    logits = torch.empty(B * dec.max_rows * V, dtype=torch.float32, device=dev) if want_logits else None
    hidden = torch.empty(B * dec.max_rows * d, dtype=torch.float32, device=dev) if want_hidden else None
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


def check_decisions(gpu, rec, wl):
    """Argmax and top-k ids must agree wherever the decision rule above pins
    them.  Returns (pinned, total) over argmax decisions."""
    pinned = total = 0
    mask = wl.model.mask_id
    for s, stats in enumerate(rec.stats):
        L = np.array(stats.logits, dtype=np.float64)
        L[:, mask] = -np.inf
        err = np.max(np.abs(np.asarray(gpu["logits"][s], np.float64) - stats.logits), axis=1)
        order = np.argsort(-L, axis=1, kind="stable")[:, : wl.topk + 1]
        top = np.take_along_axis(L, order, axis=1)
        pm = stats.p_sorted2[:, 0] - stats.p_sorted2[:, 1]
        for r in range(L.shape[0]):
            total += 1
            ok_r = pm[r] > PROB_MARGIN and top[r, 0] - top[r, 1] > ERR_FACTOR * err[r]
            if ok_r:
                pinned += 1
                assert gpu["argmax"][s][r] == stats.argmax[r], (
                    f"argmax row {r}: gpu {gpu['argmax'][s][r]} oracle {stats.argmax[r]}, "
                    f"p-margin {pm[r]:.3g} logit gap {top[r, 0] - top[r, 1]:.3g} err {err[r]:.3g}")
            for i in range(wl.topk):
                if top[r, i] - top[r, i + 1] <= max(ERR_FACTOR * err[r], 0.0) or not np.isfinite(top[r, i + 1]):
                    break
                if i == 0 and not ok_r:
                    break
                assert gpu["topk_ids"][s][r, i] == stats.topk_ids[r, i], f"top-k id row {r} rank {i}"
    return pinned, total


def check_unmask(gpu, rec, wl):
    """Unmasking decisions must agree where the confidence ranking (or the
    distance to the threshold) is wider than PROB_MARGIN and than twice the
    largest confidence difference between the two sides."""
    b = wl.block_size
    P = wl.prompt_len + rec.block_idx * b
    n_checked = 0
    for s in range(wl.batch):
        st = rec.stats[s]
        conf = st.conf[:b]
        err = float(np.max(np.abs(gpu["conf"][s][:b] - conf)))
        tol = max(PROB_MARGIN, ERR_FACTOR * err)
        sel_o = rec.selected[s]
        sel_g = gpu["selected"][s]
        still = rec.tokens_after[s, P:P + b] == wl.model.mask_id
        if wl.rule == "topn":
            chosen, rest = conf[sel_o], conf[still]
            gap = (chosen.min() - rest.max()) if len(rest) and len(chosen) else np.inf
            decided = gap > tol
        else:
            cand = sel_o | still
            decided = bool(np.all(np.abs(conf[cand] - wl.threshold) > tol))
            if not np.any(conf[cand] > wl.threshold):   # fallback: the single best
                srt = np.sort(conf[cand])[::-1]
                decided = decided and (len(srt) < 2 or srt[0] - srt[1] > tol)
        if decided:
            n_checked += 1
            assert np.array_equal(sel_g, sel_o), "unmasking decision mismatch"
            exp = rec.tokens_after[s]
            assert np.array_equal(gpu["tokens"][s][P:P + b][sel_o], exp[P:P + b][sel_o])
    return n_checked


def put_synthetic_cache(dec, st: OG.OracleState, n_prefix: int, seed: int) -> None:
    """Fills the first n_prefix slots of every layer's KV cache with seeded
    values (bf16/fp32 as the model) on the device and hands the oracle the
    very same numbers, so a cached step can be checked on its own."""
    from synthetic import seeded_normal
    shape = dec.wl.model
    B = dec.wl.batch
    caches = [[] for _ in range(B)]
    for l in range(shape.n_layers):
        kv = []
        for name, buf in (("k", dec.cache.k), ("v", dec.cache.v)):
            t = seeded_normal((B, shape.n_kv_heads, n_prefix, shape.head_dim), seed,
                              f"cache.{name}.{l}", std=1.0, device=buf.device, dtype=buf.dtype)
            buf[l, :, :, :n_prefix, :].copy_(t)
            kv.append(t.float().cpu().numpy())
        for s in range(B):
            caches[s].append((np.ascontiguousarray(kv[0][s].transpose(1, 0, 2)),
                              np.ascontiguousarray(kv[1][s].transpose(1, 0, 2))))
    st.cache = caches
