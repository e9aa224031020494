"""Block-wise SSM generation driven through the C ABI (host loop only).

Per step: ssm_select_suffix -> ssm_embed_suffix -> ssm_denoise_step ->
ssm_unmask, all enqueued on the current stream.  The fixed top-n rule knows
its step count up front and never synchronises; the threshold and margin
rules read the number of masks left in the block once per step.

A batch whose prompts differ in length (`prompt_lens`) shares the row layout
of its longest prompt (the workload's prompt_len); every call gets each
sequence's left padding, the longest prompt length minus its own.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import torch

from . import _lib as L
from .api import (select_params, ssm_denoise_step, ssm_early_stop, ssm_embed_suffix, ssm_select_count,
                  ssm_select_suffix, ssm_unmask, ssm_workspace_size)
from .model import DeviceKVCache, DeviceModel

RULES = {"topn": L.SSM_UNMASK_TOPN, "threshold": L.SSM_UNMASK_THRESHOLD,
         "margin": L.SSM_UNMASK_MARGIN}


@dataclass
class StepInfo:
    block_idx: int
    step: int
    include_prefix: bool
    n_rows: int
    n_suffix: int
    first_out_row: int
    n_cached: int

    @property
    def n_out(self) -> int:
        return self.n_rows - self.first_out_row


class Decoder:
    def __init__(self, wl, model: DeviceModel, device="cuda", prompt_lens=None):
        self.wl, self.model, self.device = wl, model, device
        self.pad = None
        if prompt_lens is not None:
            if len(prompt_lens) != wl.batch or max(prompt_lens) != wl.prompt_len or min(prompt_lens) < 0:
                raise ValueError("prompt_lens: one per sequence, the longest equal to the workload's")
            self.pad = [wl.prompt_len - int(p) for p in prompt_lens]
        shape = wl.model
        B, Lt, k = wl.batch, wl.total_len, wl.topk
        self.max_rows, self.max_kv = 1, 1
        for j in range(wl.n_blocks):
            for incl in ((True,) if not wl.cache else (True, False)):
                n_rows, _, _ = ssm_select_count(self.params(j, incl))
                n_cached = 0 if incl else wl.prompt_len + j * wl.block_size
                self.max_rows = max(self.max_rows, n_rows)
                self.max_kv = max(self.max_kv, n_cached + n_rows)
        cap = self.max_rows
        i32, f32 = torch.int32, torch.float32
        self.tokens = torch.zeros((B, Lt), dtype=i32, device=device)
        self.pos = torch.zeros(cap, dtype=i32, device=device)
        self.tok_c = torch.zeros((B, cap), dtype=i32, device=device)
        self.region = torch.zeros(cap, dtype=torch.int8, device=device)
        self.x = torch.zeros(B * cap * shape.d_model, dtype=f32, device=device)
        self.argmax = torch.zeros(B * cap, dtype=i32, device=device)
        self.conf = torch.zeros(B * cap, dtype=f32, device=device)
        self.topk_ids = torch.zeros(B * cap * k, dtype=i32, device=device)
        self.topk_w = torch.zeros(B * cap * k, dtype=f32, device=device)
        self.pred_ids = torch.zeros((B, Lt, k), dtype=i32, device=device)
        self.pred_w = torch.zeros((B, Lt, k), dtype=f32, device=device)
        self.pred_step = torch.full((B, Lt), -1, dtype=i32, device=device)
        self.selected = torch.zeros(B * wl.block_size, dtype=torch.uint8, device=device)
        self.masked_left = torch.zeros(B, dtype=i32, device=device)
        self.done = torch.zeros(B, dtype=i32, device=device)
        self.ws = torch.zeros(ssm_workspace_size(model, B, cap), dtype=torch.uint8, device=device)
        self.cache = DeviceKVCache(shape, B, self.max_kv, device)
        self.step_idx = 0

    def params(self, block_idx: int, include_prefix: bool) -> L.SelectParams:
        wl = self.wl
        return select_params(wl.prompt_len, wl.gen_len, wl.block_size, block_idx,
                             wl.local_budget, wl.middle_budget, wl.middle_mode, wl.tail_budget,
                             include_prefix, wl.tail_mode)

    def reset(self, tokens0: torch.Tensor) -> None:
        self.tokens.copy_(tokens0)
        self.pred_step.fill_(-1)
        self.done.zero_()
        self.step_idx = 0

    def step(self, block_idx: int, first_in_block: bool, logits: Optional[torch.Tensor] = None,
             hidden: Optional[torch.Tensor] = None, unmask: bool = True) -> StepInfo:
        wl, m = self.wl, self.model
        include_prefix = (not wl.cache) or first_in_block
        n_rows, n_suffix, first_out = ssm_select_suffix(
            self.params(block_idx, include_prefix), self.tokens, self.pos, self.tok_c, self.region,
            pad=self.pad)
        ssm_embed_suffix(m, self.tok_c, self.pos, self.region, n_rows, self.pred_ids, self.pred_w,
                         self.pred_step, self.step_idx - 1, wl.topk, wl.alpha, self.x, pad=self.pad)
        P = wl.prompt_len + block_idx * wl.block_size
        if not wl.cache:
            mode, n_cached = L.SSM_CACHE_OFF, 0
        elif include_prefix:
            mode, n_cached = L.SSM_CACHE_WRITE, 0
        else:
            mode, n_cached = L.SSM_CACHE_READ, P
        ssm_denoise_step(m, self.cache, mode, n_cached, self.pos, n_rows, self.x.view(wl.batch, -1),
                         first_out, wl.topk, self.argmax, self.conf, self.topk_ids, self.topk_w,
                         self.ws, logits, hidden, pad=self.pad)
        n_out = n_rows - first_out
        if unmask:
            ssm_unmask(self.tokens, P, wl.block_size, wl.model.mask_id, RULES[wl.rule],
                       wl.n_per_step, wl.threshold, self.argmax, self.conf, self.topk_ids,
                       self.topk_w, wl.topk, n_out, self.pos[first_out:], self.step_idx,
                       self.pred_ids, self.pred_w, self.pred_step, self.selected, self.masked_left,
                       pad=self.pad)
        info = StepInfo(block_idx, self.step_idx, include_prefix, n_rows, n_suffix, first_out,
                        n_cached)
        self.step_idx += 1
        return info

    def schedule(self):
        """(block, first_in_block) pairs of a fixed-rule generation."""
        spb = self.wl.steps_per_block()
        assert spb is not None
        return [(j, i == 0) for j in range(self.wl.n_blocks) for i in range(spb)]

    def generate(self, tokens0: torch.Tensor, max_steps: Optional[int] = None,
                 pre_step=None, post_step=None) -> torch.Tensor:
        """Whole generation from tokens0.  pre_step / post_step (optional) are
        called with (block, first_in_block) around every step, e.g. to record
        the schedule of a confidence-driven rule or to place timing events."""
        self.reset(tokens0)
        wl = self.wl
        spb = wl.steps_per_block()
        n = 0
        for j in range(wl.n_blocks):
            i = 0
            while True:
                if spb is not None and i >= spb:
                    break
                if pre_step is not None:
                    pre_step(j, i == 0)
                self.step(j, i == 0)
                if post_step is not None:
                    post_step(j, i == 0)
                i += 1
                n += 1
                if max_steps is not None and n >= max_steps:
                    return self.tokens
                if spb is None and int(self.masked_left.max().item()) == 0:
                    break
            if wl.eos_id >= 0 and self.early_stop(j):
                break
        return self.tokens

    def early_stop(self, block_idx: int) -> bool:
        """Early termination after block `block_idx`: fills the later blocks of
        sequences that produced the end token; True once every sequence has."""
        wl = self.wl
        ssm_early_stop(self.tokens, wl.prompt_len + block_idx * wl.block_size, wl.block_size,
                       wl.eos_id, self.done, pad=self.pad)
        return bool(int(self.done.min().item()) == 1)
