"""Shared helpers of the GPU parity tests (not collected by pytest)."""
from __future__ import annotations

import numpy as np
import torch

import oracle.generate as OG

# Decision rule of the parity tests.  A decision (an argmax, a top-k rank, an
# unmasking choice) must be identical on both sides wherever the oracle's
# probability margin exceeds PROB_MARGIN (1e-3).  The only exemption comes
# from a fixed error budget of the logits, derived from the stated tolerances
# and the oracle's own logits -- never from the GPU output:
#   * float32 mode: every logit is within FP32_LOGIT_TOL (1e-4, asserted in the
#     same tests), so eps = 1e-4;
#   * bfloat16 mode: the relative L2 error of the logits is at most
#     BF16_REL_TOL (2e-2).  The error of one logit is an LM-head row applied to
#     the error of the normalised hidden row; over independent random head
#     rows each such error is close to N(0, s^2) with s = 2e-2 * rms(row
#     logits), and the largest of V of them is about s * sqrt(2 ln V).  So
#     eps = 2e-2 * rms(row) * sqrt(2 ln V).
# Two logits of a row further apart than 2 eps keep their order; a
# log-probability (a logit minus the row's log-sum-exp) moves by at most
# 2 eps, so two confidences whose logarithms are further apart than the sum of
# their budgets keep their order too.  A decision with a probability margin
# above 1e-3 that lies inside the budget is counted as exempt; every test
# reports its exempt count next to the count of decisions it checked.
PROB_MARGIN = 1e-3
FP32_LOGIT_TOL = 1e-4
BF16_REL_TOL = 2e-2


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


class Counts:
    """Decisions checked (required and compared), exempt (margin above 1e-3
    but inside the fixed error budget; compared and reported only) and the
    total considered, with the exempt ones the two sides decided differently.
    `inside` counts every decision inside the budget, whatever its margin: a
    decision outside it is fixed by the arithmetic of both sides."""

    def __init__(self):
        self.checked = self.exempt = self.total = self.exempt_differ = self.inside = 0

    def add(self, o: "Counts") -> "Counts":
        self.checked += o.checked
        self.exempt += o.exempt
        self.total += o.total
        self.exempt_differ += o.exempt_differ
        self.inside += o.inside
        return self

    def __repr__(self):
        return (f"checked {self.checked}/{self.total}, exempt {self.exempt} "
                f"({self.exempt_differ} decided differently)")


def logit_budget(logits: np.ndarray, mask_id: int, fp32: bool, eps=None) -> np.ndarray:
    """eps per row of the oracle's logits [n, V] (see the rule above); `eps`
    replaces the float32 bound where a test states a wider one."""
    n, V = logits.shape
    if fp32:
        return np.full(n, FP32_LOGIT_TOL if eps is None else eps)
    L = np.delete(np.asarray(logits, np.float64), mask_id, axis=1)
    rms = np.sqrt(np.mean(L * L, axis=1))
    return BF16_REL_TOL * rms * np.sqrt(2.0 * np.log(V))


def _log_probs(logits_row: np.ndarray, mask_id: int) -> np.ndarray:
    l = np.array(logits_row, dtype=np.float64)
    l[mask_id] = -np.inf
    m = np.max(l)
    return l - (m + np.log(np.sum(np.exp(l - m))))


def check_decisions(gpu, rec, wl, fp32: bool) -> Counts:
    """Argmax and top-k ids of every output row under the rule above."""
    c = Counts()
    mask = wl.model.mask_id
    for s, stats in enumerate(rec.stats):
        eps = logit_budget(stats.logits, mask, fp32)
        for r in range(stats.logits.shape[0]):
            lp = _log_probs(stats.logits[r], mask)
            order = np.argsort(-lp, kind="stable")[: wl.topk + 1]
            top = lp[order]
            p = np.exp(top)
            c.total += 1
            c.inside += int(not top[0] - top[1] > 2 * eps[r])
            if not p[0] - p[1] > PROB_MARGIN:
                continue                          # below the 1e-3 rule: not required
            if not top[0] - top[1] > 2 * eps[r]:
                c.exempt += 1
                c.exempt_differ += int(gpu["argmax"][s][r] != stats.argmax[r])
                continue
            c.checked += 1
            assert gpu["argmax"][s][r] == stats.argmax[r], (
                f"argmax seq {s} row {r}: gpu {gpu['argmax'][s][r]} oracle {stats.argmax[r]}, "
                f"p-margin {p[0] - p[1]:.3g} logit gap {top[0] - top[1]:.3g} budget {2 * eps[r]:.3g}")
            # top-k ranks, in order, while each is decided
            for i in range(1, wl.topk):
                if not (p[i] - p[i + 1] > PROB_MARGIN and top[i] - top[i + 1] > 2 * eps[r]):
                    break
                assert gpu["topk_ids"][s][r, i] == stats.topk_ids[r, i], \
                    f"top-k id seq {s} row {r} rank {i}"
    return c


def check_unmask(gpu, rec, wl, fp32: bool, eps=None) -> Counts:
    """The unmasking choice of each sequence under the rule above: top-n by the
    gap between the n-th chosen and the best unchosen confidence; threshold
    and margin by every candidate's distance to the threshold (and, for the
    at-least-one fallback, the gap between the two best).  A choice is checked
    when every comparison it rests on has a margin above 1e-3 outside the
    budget, exempt when one of them is inside the budget, and not required
    when one of them has a margin of 1e-3 or less."""
    b = wl.block_size
    P = wl.prompt_len + rec.block_idx * b
    mask = wl.model.mask_id
    c = Counts()
    for s in range(wl.batch):
        st = rec.stats[s]
        eps_r = logit_budget(st.logits[:b], mask, fp32, eps)
        conf = np.asarray(st.conf[:b], np.float64)
        logc = np.log(np.maximum(conf, 1e-300))
        p1, p2 = st.p_sorted2[:b, 0], st.p_sorted2[:b, 1]
        marg = p1 - p2
        rho = np.expm1(2 * eps_r)                   # relative bound of a probability
        sel_o = np.asarray(rec.selected[s], bool)
        still = rec.tokens_after[s, P:P + b] == mask
        cand = sel_o | still
        required, inside = True, False

        def pair(i, j, by_margin=False):
            nonlocal required, inside
            if by_margin:
                gap = abs(marg[i] - marg[j])
                ok = gap > rho[i] * (p1[i] + p2[i]) + rho[j] * (p1[j] + p2[j])
            else:
                gap = abs(conf[i] - conf[j])
                ok = abs(logc[i] - logc[j]) > 2 * eps_r[i] + 2 * eps_r[j]
            required &= gap > PROB_MARGIN
            inside |= not ok

        def vs_threshold(i):
            nonlocal required, inside
            if wl.rule == "margin":
                gap = abs(marg[i] - wl.threshold)
                ok = gap > rho[i] * (p1[i] + p2[i])
            else:
                gap = abs(conf[i] - wl.threshold)
                ok = abs(logc[i] - np.log(wl.threshold)) > 2 * eps_r[i] if wl.threshold > 0 else True
            required &= gap > PROB_MARGIN
            inside |= not ok

        idx = np.nonzero(cand)[0]
        if wl.rule == "topn":
            chosen, rest = np.nonzero(sel_o)[0], np.nonzero(still)[0]
            if len(chosen) and len(rest):
                pair(chosen[np.argmin(conf[chosen])], rest[np.argmax(conf[rest])])
        else:
            score = marg if wl.rule == "margin" else conf
            for i in idx:
                vs_threshold(i)
            if len(idx) >= 2 and not np.any(score[idx] > wl.threshold):
                o = idx[np.argsort(-score[idx], kind="stable")]
                pair(o[0], o[1], by_margin=wl.rule == "margin")
        c.total += 1
        c.inside += int(inside)
        if not required:
            continue
        differ = not np.array_equal(np.asarray(gpu["selected"][s], bool), sel_o)
        if inside:
            c.exempt += 1
            c.exempt_differ += int(differ)
            continue
        c.checked += 1
        assert not differ, f"unmasking decision mismatch, sequence {s}"
        exp = rec.tokens_after[s]
        assert np.array_equal(gpu["tokens"][s][P:P + b][sel_o], exp[P:P + b][sel_o])
    return c


def check_unmask_consistency(gpu, rec, wl) -> int:
    """The unmasking rule applied by the oracle's choose() to the GPU's own
    confidences (float32, with the margin formed as the kernel forms it:
    conf * (1 - w1 / w0) in float32) selects exactly the GPU's positions: the
    decision stage is bit-exact on the GPU's inputs, whatever the margins.
    Returns the number of sequences checked."""
    import oracle.unmask as OU
    b = wl.block_size
    P = wl.prompt_len + rec.block_idx * b
    f32 = np.float32
    for s in range(wl.batch):
        conf = np.asarray(gpu["conf"][s][:b], f32)
        w = np.asarray(gpu["topk_w"][s][:b], f32)
        margin = conf * (f32(1) - w[:, 1] / w[:, 0]) if wl.topk >= 2 else None
        # masked before the step: still masked after it, or decoded by it
        masked = (rec.tokens_after[s, P:P + b] == wl.model.mask_id) | np.asarray(rec.selected[s], bool)
        want = OU.choose(conf, masked, wl.rule, wl.n_per_step, f32(wl.threshold), margin)
        assert np.array_equal(np.asarray(gpu["selected"][s], bool), want), \
            f"unmask stage differs from the rule on the GPU's own confidences, sequence {s}"
        dec = np.asarray(gpu["tokens"][s][P:P + b])
        assert np.array_equal(dec[want], np.asarray(gpu["argmax"][s][:b])[want])
    return wl.batch


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
