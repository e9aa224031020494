"""Pins of the oracle's suffix partition and retention (Section 3.2, Eq. 1-5)."""
import itertools
import os

import numpy as np
import pytest

from oracle import selection as S

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "selection_fixtures.txt")


def _parse_positions(text):
    out = []
    for tok in text.split():
        if "-" in tok:
            a, b = tok.split("-")
            out.extend(range(int(a), int(b) + 1))
        else:
            out.append(int(tok))
    return out


def _golden_cases():
    cases = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            head, tail = line.split("|")
            cases.append((tuple(int(v) for v in head.split()), _parse_positions(tail)))
    return cases


@pytest.mark.parametrize("params,expected", _golden_cases())
def test_golden_retained_sets(params, expected):
    prompt, gen, b, j, L, M, mode, T = params[:8]
    tail_mode = params[8] if len(params) > 8 else S.TAIL_SPREAD
    r = S.retained_suffix(prompt, gen, b, j, L, M, mode, T, tail_mode)
    assert r.positions == expected


def paper_block_rule(prompt, gen, b, j, w):
    """Eq. 1-5 written over blocks: first w suffix blocks local, last block tail,
    the rest middle; fewer than (or exactly) w blocks: all local."""
    nb = gen // b
    suffix_blocks = list(range(j + 1, nb))
    start = lambda m: prompt + m * b
    if len(suffix_blocks) <= w:
        local, middle, tail = suffix_blocks, [], []
    else:
        local, middle, tail = suffix_blocks[:w], suffix_blocks[w:-1], suffix_blocks[-1:]
    r = set()
    for m in local:
        r.update(range(start(m), start(m) + b))
    for m in middle:
        r.add(start(m))
    for m in tail:
        r.add(start(m))
        r.add(start(m) + b - 1)
    return sorted(r)


@pytest.mark.parametrize("b", [1, 2, 4, 8, 32])
def test_block_budgets_reduce_to_paper_rule(b):
    for nb in range(1, 10):
        gen = nb * b
        for prompt in (0, 3):
            for w in range(0, 5):
                for j in range(nb):
                    r = S.retained_suffix(prompt, gen, b, j, w * b, 0, S.MIDDLE_BLOCK_START, 2)
                    want = paper_block_rule(prompt, gen, b, j, w)
                    if b == 1:
                        # a one-token block: its start and end coincide
                        want = sorted(set(want))
                    assert r.positions == want, (prompt, gen, b, j, w)


def paper_block_variant(prompt, gen, b, j, w, middle_keep, tail_keep):
    """Table 2 variants over blocks: middle blocks keep the in-block offsets
    `middle_keep`, the tail block keeps `tail_keep` (offsets from its start)."""
    nb = gen // b
    suffix_blocks = list(range(j + 1, nb))
    start = lambda m: prompt + m * b
    if len(suffix_blocks) <= w:
        return sorted(p for m in suffix_blocks for p in range(start(m), start(m) + b))
    r = set()
    for m in suffix_blocks[:w]:
        r.update(range(start(m), start(m) + b))
    for m in suffix_blocks[w:-1]:
        r.update(start(m) + o for o in middle_keep)
    r.update(start(suffix_blocks[-1]) + o for o in tail_keep)
    return sorted(r)


@pytest.mark.parametrize("b", [1, 2, 5, 8])
def test_table2_variants_reduce_to_block_rule(b):
    """Middle end / start+end tokens; tail start only, end only, start+mid+end."""
    variants = [
        (S.MIDDLE_BLOCK_END, 2, S.TAIL_SPREAD, (b - 1,), (0, b - 1)),
        (S.MIDDLE_BLOCK_START_END, 2, S.TAIL_SPREAD, (0, b - 1), (0, b - 1)),
        (S.MIDDLE_BLOCK_START, 1, S.TAIL_START, (0,), (0,)),
        (S.MIDDLE_BLOCK_START, 1, S.TAIL_SPREAD, (0,), (b - 1,)),
        (S.MIDDLE_BLOCK_START, 3, S.TAIL_SPREAD, (0,), (0, (b - 1) // 2, b - 1)),
    ]
    for nb in range(1, 9):
        gen = nb * b
        for prompt in (0, 3):
            for w in range(0, 4):
                for j in range(nb):
                    for mmode, T, tmode, mk, tk in variants:
                        r = S.retained_suffix(prompt, gen, b, j, w * b, 0, mmode, T, tmode)
                        want = paper_block_variant(prompt, gen, b, j, w, mk, tk)
                        assert r.positions == want, (prompt, gen, b, j, w, mmode, T, tmode)


def test_brute_force_block_modes():
    """Block modes with local budgets that cut a block: sorted, unique, the
    middle keeps exactly the in-range tokens at the mode's block offsets, the
    start-only tail keeps its first token."""
    prompt = 3
    for gen_blocks, b in itertools.product(range(1, 8), (1, 2, 3, 8)):
        gen = gen_blocks * b
        for j in range(gen_blocks):
            for L in (0, 1, b - 1, b + 1, 2 * b + 3, gen):
                for mmode, keep in ((S.MIDDLE_BLOCK_START, {0}), (S.MIDDLE_BLOCK_END, {b - 1}),
                                    (S.MIDDLE_BLOCK_START_END, {0, b - 1})):
                    for T, tmode in itertools.product((0, 1, 2, 3), (S.TAIL_SPREAD, S.TAIL_START)):
                        r = S.retained_suffix(prompt, gen, b, j, max(L, 0), 7, mmode, T, tmode)
                        pos, reg = r.positions, r.regions
                        s0, s_end = prompt + (j + 1) * b, prompt + gen
                        assert pos == sorted(set(pos))
                        l = min(max(L, 0), s_end - s0)
                        tail_lo = max(s0 + l, s_end - b)
                        mid = [p for p, g in zip(pos, reg) if g == S.REGION_MIDDLE]
                        assert mid == [p for p in range(s0 + l, tail_lo) if (p - prompt) % b in keep]
                        tail = [p for p, g in zip(pos, reg) if g == S.REGION_TAIL]
                        if tmode == S.TAIL_START:
                            assert tail == ([tail_lo] if T >= 1 and tail_lo < s_end else [])


def test_brute_force_properties():
    for gen_blocks, b in itertools.product(range(1, 9), (2, 4, 8)):
        gen = gen_blocks * b
        prompt = 5
        for j in range(gen_blocks):
            for L, M, T in itertools.product((0, 1, 3, b, 2 * b + 1, gen), (0, 1, 2, 5, gen),
                                              (0, 1, 2, 3, b)):
                r = S.retained_suffix(prompt, gen, b, j, L, M, S.MIDDLE_STRIDED, T)
                pos, reg = r.positions, r.regions
                s0, s_end = prompt + (j + 1) * b, prompt + gen
                n = s_end - s0
                # sorted, unique, inside the suffix
                assert pos == sorted(set(pos))
                assert all(s0 <= p < s_end for p in pos)
                l = min(L, n)
                tail_len = min(b, n - l)
                mid_len = n - l - tail_len
                # closed-form count
                assert len(pos) == l + min(M, mid_len) + min(T, tail_len)
                # region membership
                for p, g in zip(pos, reg):
                    if g == S.REGION_LOCAL:
                        assert p < s0 + l
                    elif g == S.REGION_MIDDLE:
                        assert s0 + l <= p < s_end - tail_len
                    else:
                        assert g == S.REGION_TAIL and p >= s_end - tail_len
                # the tail keeps its end token whenever it keeps anything
                tail = [p for p, g in zip(pos, reg) if g == S.REGION_TAIL]
                if tail:
                    assert tail[-1] == s_end - 1
                    if len(tail) >= 2:
                        assert tail[0] == s_end - tail_len
                # the middle keeps its first token whenever it keeps anything
                mid = [p for p, g in zip(pos, reg) if g == S.REGION_MIDDLE]
                if mid:
                    assert mid[0] == s0 + l


def test_full_and_zero_budgets():
    prompt, gen, b = 7, 96, 8
    for j in range(gen // b):
        s0, s_end = prompt + (j + 1) * b, prompt + gen
        full = S.retained_suffix(prompt, gen, b, j, gen, gen, S.MIDDLE_STRIDED, gen)
        assert full.positions == list(range(s0, s_end))
        zero = S.retained_suffix(prompt, gen, b, j, 0, 0, S.MIDDLE_STRIDED, 0)
        assert zero.positions == []


def test_compacted_rows_layout():
    c = S.compacted_rows(32, 128, 32, 1, 32, 8, 0, 4, include_prefix=True)
    P = 64
    assert list(c.pos[:P]) == list(range(P))
    assert list(c.pos[P:P + 32]) == list(range(P, P + 32))
    assert c.first_out_row == P and c.n_prefix == P and c.n_suffix == 36
    assert list(c.region[:P]) == [S.REGION_PREFIX] * P
    assert list(c.region[P:P + 32]) == [S.REGION_BLOCK] * 32
    c2 = S.compacted_rows(32, 128, 32, 1, 32, 8, 0, 4, include_prefix=False)
    assert c2.first_out_row == 0 and list(c2.pos) == list(c.pos[P:])
