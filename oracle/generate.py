"""Block-wise generation with SSM (Section 3.2; decoding settings of Section 4).

TEST INFRASTRUCTURE ONLY (see the package docstring).

One step, in the paper's order:
  1. partition the suffix of the current block and keep R_t        (Eq. 1-5)
  2. build the sparse input [P; B_t; R_t] at original positions    (Sparse Input Construction)
  3. embed it, mixing previous-step predictions into R_t            (Eq. 6-8)
  4. run the bidirectional transformer (prefix KV cache optional)
  5. decode the chosen masked positions of the block                (Section 4.2)
  6. remember the top-k prediction of every retained suffix row for the next step.

Steps are numbered 0, 1, 2, ... over the whole generation; the paper's
"previous timestep t+1" is step s-1 here.  With a fixed top-n rule a block
takes ceil(b/n) steps, with the threshold or margin rule it steps until the
block has no mask left.

Early termination (Section 3.2, "Early Termination"; the fill rule of
Section 4.4) is optional (workload eos_id >= 0): after the last step of a
block, a sequence whose block holds the end-of-sequence id has every later
position set to that id and is done; the generation stops once every
sequence is done.  Random-init models have no meaningful end token, so the
workloads leave it off.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, List, Optional

import numpy as np

from . import embed as E
from . import model as M
from . import selection as S
from . import unmask as U


def _to_np(t, dtype):
    if isinstance(t, np.ndarray):
        return t.astype(dtype, copy=False)
    return np.asarray(t.detach().float().cpu().numpy(), dtype=dtype)


class _Layer:
    __slots__ = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")

    def __init__(self, lw, dtype):
        for name in self.__slots__:
            setattr(self, name, _to_np(getattr(lw, name), dtype))


class _Layers:
    def __init__(self, layers, dtype, keep=True):
        self._src, self._dtype, self._keep = layers, dtype, keep
        self._cache = {}

    def __len__(self):
        return len(self._src)

    def __getitem__(self, i):
        if i in self._cache:
            return self._cache[i]
        lw = _Layer(self._src[i], self._dtype)
        if self._keep:
            self._cache[i] = lw
        return lw


class NumpyWeights:
    """The oracle's view of a model: NumPy arrays in the oracle's precision."""

    def __init__(self, mw, dtype=np.float64, keep_layers=True):
        self.tok_emb = _to_np(mw.tok_emb, dtype)
        self.final_norm = _to_np(mw.final_norm, dtype)
        self.lm_head = _to_np(mw.lm_head, dtype)
        self.layers = _Layers(mw.layers, dtype, keep_layers)
        self.dtype = dtype


@dataclass
class OracleState:
    tokens: np.ndarray                  # [B, L_tot] int32
    pred_ids: np.ndarray                # [B, L_tot, k] int32
    pred_w: np.ndarray                  # [B, L_tot, k]
    pred_step: np.ndarray               # [B, L_tot] int32, -1 = none
    step: int = 0
    cache: Optional[list] = None        # per sequence: per layer (k, v) of the prefix
    done: Optional[np.ndarray] = None   # [B] bool: ended by early termination

    @staticmethod
    def start(tokens: np.ndarray, k: int) -> "OracleState":
        B, L = tokens.shape
        return OracleState(np.array(tokens, dtype=np.int32).copy(),
                           np.zeros((B, L, k), np.int32), np.zeros((B, L, k), np.float64),
                           np.full((B, L), -1, np.int32), done=np.zeros(B, dtype=bool))

    def copy(self) -> "OracleState":
        return OracleState(self.tokens.copy(), self.pred_ids.copy(), self.pred_w.copy(),
                           self.pred_step.copy(), self.step,
                           None if self.cache is None else [list(c) for c in self.cache],
                           None if self.done is None else self.done.copy())


@dataclass
class StepRecord:
    block_idx: int
    step: int
    include_prefix: bool
    rows: S.Compacted
    x: np.ndarray = None          # [B, n, d] input embeddings
    hidden: np.ndarray = None     # [B, n, d] after the last layer
    stats: list = field(default_factory=list)   # per sequence OutputStats
    selected: np.ndarray = None   # [B, b] bool
    tokens_after: np.ndarray = None


def step(wl, w: NumpyWeights, st: OracleState, block_idx: int, first_in_block: bool,
         keep: bool = True) -> StepRecord:
    """One denoising step of every sequence of the batch; updates `st` in place."""
    shape = wl.model
    b = wl.block_size
    include_prefix = (not wl.cache) or first_in_block
    rows = S.compacted_rows(wl.prompt_len, wl.gen_len, b, block_idx, wl.local_budget,
                            wl.middle_budget, wl.middle_mode, wl.tail_budget, include_prefix,
                            wl.tail_mode)
    B = st.tokens.shape[0]
    P = wl.prompt_len + block_idx * b
    rec = StepRecord(block_idx, st.step, include_prefix, rows)
    xs, hs, sel_all = [], [], []
    new_cache = []
    for s in range(B):
        x = E.embed_rows(w.tok_emb, st.tokens[s], rows.pos, rows.region, st.pred_ids[s],
                         st.pred_w[s], st.pred_step[s], st.step - 1, wl.alpha, shape.mask_id)
        prefix_kv = None if include_prefix else st.cache[s]
        fo = M.forward(x, rows.pos, w, shape, prefix_kv)
        if wl.cache and include_prefix:
            new_cache.append([(k[:rows.n_prefix].copy(), v[:rows.n_prefix].copy())
                              for (k, v) in fo.kv])
        stats = M.output_stats(fo.hidden[rows.first_out_row:], w, shape, wl.topk)
        masked = st.tokens[s, P:P + b] == shape.mask_id
        margin = stats.p_sorted2[:b, 0] - stats.p_sorted2[:b, 1]
        sel = U.choose(stats.conf[:b], masked, wl.rule, wl.n_per_step, wl.threshold, margin)
        for i in np.nonzero(sel)[0]:
            st.tokens[s, P + i] = stats.argmax[i]
        out_pos = rows.pos[rows.first_out_row:]
        for r in range(b, len(out_pos)):
            p = int(out_pos[r])
            st.pred_ids[s, p] = stats.topk_ids[r]
            st.pred_w[s, p] = stats.topk_w[r]
            st.pred_step[s, p] = st.step
        if keep:
            xs.append(x)
            hs.append(fo.hidden)
            rec.stats.append(stats)
        sel_all.append(sel)
    if wl.cache and include_prefix:
        st.cache = new_cache
    if keep:
        rec.x = np.stack(xs)
        rec.hidden = np.stack(hs)
    rec.selected = np.stack(sel_all)
    rec.tokens_after = st.tokens.copy()
    st.step += 1
    return rec


def early_stop(tokens: np.ndarray, done: np.ndarray, block_start: int, block_size: int,
               eos_id: int) -> bool:
    """Early termination check after a block (Section 3.2; fill rule of Section
    4.4): every sequence not yet done whose block holds eos_id gets all later
    positions set to eos_id and becomes done.  Returns whether all are done."""
    for s in range(tokens.shape[0]):
        if done[s]:
            continue
        if np.any(tokens[s, block_start:block_start + block_size] == eos_id):
            tokens[s, block_start + block_size:] = eos_id
            done[s] = True
    return bool(np.all(done))


def block_done(wl, st: OracleState, block_idx: int) -> bool:
    P = wl.prompt_len + block_idx * wl.block_size
    return not np.any(st.tokens[:, P:P + wl.block_size] == wl.model.mask_id)


def generate(wl, w: NumpyWeights, tokens0: np.ndarray, keep: bool = False,
             on_step: Optional[Callable[[StepRecord, OracleState], None]] = None,
             max_steps: Optional[int] = None):
    """Whole generation.  Returns (final state, list of step records)."""
    st = OracleState.start(tokens0, wl.topk)
    recs: List[StepRecord] = []
    fixed = wl.steps_per_block()
    for j in range(wl.n_blocks):
        i = 0
        while True:
            if fixed is not None and i >= fixed:
                break
            if fixed is None and block_done(wl, st, j):
                break
            rec = step(wl, w, st, j, i == 0, keep)
            recs.append(rec)
            if on_step is not None:
                on_step(rec, st)
            i += 1
            if max_steps is not None and len(recs) >= max_steps:
                return st, recs
        if wl.eos_id >= 0 and early_stop(st.tokens, st.done, wl.prompt_len + j * wl.block_size,
                                         wl.block_size, wl.eos_id):
            break
    return st, recs
