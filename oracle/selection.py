"""Suffix region partition and token retention (Section 3.2, "Suffix Region
Partition", "Suffix Token Retention", Eq. 1-5; "Sparse Input Construction").

TEST INFRASTRUCTURE ONLY (see the package docstring).

Positions are absolute indices into the sequence [prompt; generated].  Block j
of the generated part covers [P0 + j*b, P0 + (j+1)*b); the suffix of block j
is everything after it.

The paper states budgets in blocks: the first w suffix blocks are kept whole
(Eq. 2), every middle block keeps its start token (Eq. 3), and the last block
keeps its start and end tokens (Eq. 4).  The workloads here state budgets in
tokens, so the oracle follows this generalisation (a reading, since the paper
gives only the block rule):

  * local region  = the first min(L, n) suffix tokens                 (Eq. 2 with L = w*b)
  * tail region   = the last block, minus anything already local      (Eq. 1)
  * middle region = whatever lies between them                        (Eq. 1)
  * middle, strided mode: M' = min(M, len) tokens at offsets floor(i*len/M')
  * middle, block-start mode: the start token of every middle block    (Eq. 3)
  * middle, block-end and block-start+end modes: the end token, or both end
    tokens, of every middle block (the middle-region variants of the ablation
    in Table 2)
  * tail, spread mode: T' = min(T, len) tokens at offsets
    floor(i*(len-1)/(T'-1)), so both ends are always kept (Eq. 4 is T = 2);
    T' = 1 keeps the end token only, T' = 3 adds the token at floor((len-1)/2)
    (the "end only" and "start+mid+end" variants of Table 2)
  * tail, start mode: the start token only, if T >= 1 (the "start only"
    variant of Table 2)
  * fewer suffix tokens than the local budget: everything is local (the
    paper's "fewer than w blocks" case); local wins any overlap with the tail.
"""
from __future__ import annotations

from typing import List, NamedTuple, Tuple

import numpy as np

REGION_PREFIX = 0
REGION_BLOCK = 1
REGION_LOCAL = 2
REGION_MIDDLE = 3
REGION_TAIL = 4

MIDDLE_STRIDED = 0
MIDDLE_BLOCK_START = 1
MIDDLE_BLOCK_END = 2
MIDDLE_BLOCK_START_END = 3

TAIL_SPREAD = 0
TAIL_START = 1

Range = Tuple[int, int]


def suffix_partition(prompt_len: int, gen_len: int, block_size: int, block_idx: int,
                     local_budget: int) -> Tuple[Range, Range, Range]:
    """Eq. 1: split the suffix of block `block_idx` into local, middle and tail ranges."""
    b = block_size
    s0 = prompt_len + (block_idx + 1) * b          # first suffix position
    s_end = prompt_len + gen_len                   # one past the last position
    n = s_end - s0
    n_local = min(local_budget, n)
    local = (s0, s0 + n_local)
    tail_start = max(s0 + n_local, s_end - b)      # last block, minus the local part
    middle = (s0 + n_local, tail_start)
    tail = (tail_start, s_end)
    return local, middle, tail


def retain_local(local: Range) -> List[int]:
    """Eq. 2: every local token is kept."""
    return list(range(local[0], local[1]))


def retain_middle(middle: Range, budget: int, mode: int, block_grid_origin: int,
                  block_size: int) -> List[int]:
    """Eq. 3 (block-start mode), the Table 2 variants that keep each middle
    block's end token instead or both end tokens, or the token-budget
    generalisation (strided mode)."""
    lo, hi = middle
    length = hi - lo
    if length <= 0:
        return []
    if mode in (MIDDLE_BLOCK_START, MIDDLE_BLOCK_END, MIDDLE_BLOCK_START_END):
        keep = {MIDDLE_BLOCK_START: (0,), MIDDLE_BLOCK_END: (block_size - 1,),
                MIDDLE_BLOCK_START_END: (0, block_size - 1)}[mode]
        return [p for p in range(lo, hi) if (p - block_grid_origin) % block_size in keep]
    m = min(budget, length)
    return [lo + (i * length) // m for i in range(m)]


def retain_tail(tail: Range, budget: int, mode: int = TAIL_SPREAD) -> List[int]:
    """Eq. 4: start and end token of the last block; generalised to T evenly
    spread tokens, or (start mode, Table 2) the start token alone."""
    lo, hi = tail
    length = hi - lo
    t = min(budget, length)
    if t <= 0:
        return []
    if mode == TAIL_START:
        return [lo]
    if t == 1:
        return [hi - 1]
    return [lo + (i * (length - 1)) // (t - 1) for i in range(t)]


class Retained(NamedTuple):
    positions: List[int]
    regions: List[int]


def retained_suffix(prompt_len: int, gen_len: int, block_size: int, block_idx: int,
                    local_budget: int, middle_budget: int, middle_mode: int,
                    tail_budget: int, tail_mode: int = TAIL_SPREAD) -> Retained:
    """Eq. 5: R_t = R_local U R_middle U R_tail, in ascending position order."""
    local, middle, tail = suffix_partition(prompt_len, gen_len, block_size, block_idx,
                                           local_budget)
    r_local = retain_local(local)
    r_middle = retain_middle(middle, middle_budget, middle_mode, prompt_len, block_size)
    r_tail = retain_tail(tail, tail_budget, tail_mode)
    pos = r_local + r_middle + r_tail
    reg = ([REGION_LOCAL] * len(r_local) + [REGION_MIDDLE] * len(r_middle)
           + [REGION_TAIL] * len(r_tail))
    return Retained(pos, reg)


class Compacted(NamedTuple):
    pos: np.ndarray            # int32 [n_rows] absolute position of every row
    region: np.ndarray         # int8  [n_rows]
    n_prefix: int              # rows of prefix included (0 on a cached step)
    first_out_row: int         # first row that needs logits (the current block)
    n_suffix: int              # |R_t|


def compacted_rows(prompt_len: int, gen_len: int, block_size: int, block_idx: int,
                   local_budget: int, middle_budget: int, middle_mode: int, tail_budget: int,
                   include_prefix: bool, tail_mode: int = TAIL_SPREAD) -> Compacted:
    """Sparse input [P; B_t; R_t] ("Sparse Input Construction").

    The prefix P is the prompt plus every block decoded so far (a reading: the
    paper writes it as the prompt).  On a cached step the prefix rows come from
    the KV cache and are not part of the input.  Every row keeps its original
    position, which is what RoPE is applied at.
    """
    b = block_size
    P = prompt_len + block_idx * b
    r = retained_suffix(prompt_len, gen_len, b, block_idx, local_budget, middle_budget,
                        middle_mode, tail_budget, tail_mode)
    pre = list(range(P)) if include_prefix else []
    blk = list(range(P, P + b))
    pos = np.array(pre + blk + r.positions, dtype=np.int32)
    region = np.array([REGION_PREFIX] * len(pre) + [REGION_BLOCK] * b + r.regions,
                      dtype=np.int8)
    return Compacted(pos, region, len(pre), len(pre), len(r.positions))
