"""Model shapes and decoding workloads.

The model shapes follow the diffusion LMs the paper evaluates (LLaDA-8B and
Dream-7B, Section 4.1) with random initialisation; the workloads follow the
paper's decoding settings (block 32, confidence threshold 0.9, top-k in
{3,5,7}, alpha in {0.2,0.3,0.4}; Section 4.1) and its long-sequence setting
(Section 4.8, Table 4).  Budgets are in tokens: a local budget of w*b with
block-start middle mode and a tail budget of 2 reproduces Eq. 2-4 exactly.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass


@dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    mask_id: int
    dtype: str = "bf16"          # storage/compute type of the GPU path: "f32" or "bf16"
    rope_base: float = 10000.0
    rms_eps: float = 1e-5
    init_std: float = 0.02

    def with_layers(self, n: int) -> "ModelShape":
        return dataclasses.replace(self, n_layers=n, name=f"{self.name}-L{n}")

    @property
    def qkv_dim(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    def params_per_layer(self) -> int:
        d, hd = self.d_model, self.head_dim
        return (d * self.n_heads * hd + 2 * d * self.n_kv_heads * hd
                + self.n_heads * hd * d + 3 * d * self.ffn_dim)

    def kv_bytes_per_token(self) -> int:
        el = 4 if self.dtype == "f32" else 2
        return 2 * self.n_layers * self.n_kv_heads * self.head_dim * el


TINY = ModelShape("tiny", n_layers=2, d_model=128, n_heads=4, n_kv_heads=4, head_dim=32,
                  ffn_dim=512, vocab=512, mask_id=511, dtype="f32")
LLADA_8B = ModelShape("llada8b", n_layers=32, d_model=4096, n_heads=32, n_kv_heads=32,
                      head_dim=128, ffn_dim=12288, vocab=126464, mask_id=126463)
DREAM_7B = ModelShape("dream7b", n_layers=28, d_model=3584, n_heads=28, n_kv_heads=4,
                      head_dim=128, ffn_dim=18944, vocab=152064, mask_id=152063)


# unmasking rules
TOPN = "topn"
THRESHOLD = "threshold"
MARGIN = "margin"

# middle-region modes
MIDDLE_STRIDED = 0        # evenly strided token budget
MIDDLE_BLOCK_START = 1    # start token of every middle block (Eq. 3)
MIDDLE_BLOCK_END = 2      # end token of every middle block (Table 2 variant)
MIDDLE_BLOCK_START_END = 3   # both (Table 2 variant)

# tail-region modes
TAIL_SPREAD = 0           # T evenly spread tokens, both ends first (Eq. 4 at T = 2)
TAIL_START = 1            # the start token only (Table 2 variant)


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    prompt_len: int
    gen_len: int
    block_size: int
    rule: str
    n_per_step: int = 1
    threshold: float = 0.9
    local_budget: int = 0
    middle_budget: int = 0
    tail_budget: int = 0
    middle_mode: int = MIDDLE_STRIDED
    tail_mode: int = TAIL_SPREAD
    cache: bool = False
    batch: int = 1
    seed: int = 0
    topk: int = 5
    alpha: float = 0.4
    logit_scale: float = 1.0   # test-only sharpening applied to the LM head weights
    eos_id: int = -1           # end-of-sequence id for early termination; -1: off

    @property
    def total_len(self) -> int:
        return self.prompt_len + self.gen_len

    @property
    def n_blocks(self) -> int:
        return self.gen_len // self.block_size

    def steps_per_block(self) -> int | None:
        if self.rule == TOPN:
            return -(-self.block_size // self.n_per_step)
        return None

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    "tiny": Workload("tiny", TINY, prompt_len=32, gen_len=128, block_size=32, rule=TOPN,
                     n_per_step=4, local_budget=32, middle_budget=8, tail_budget=4,
                     cache=False, batch=1),
    "llada_gen256": Workload("llada_gen256", LLADA_8B, prompt_len=256, gen_len=256,
                             block_size=32, rule=TOPN, n_per_step=1, local_budget=64,
                             middle_budget=16, tail_budget=8, cache=True, batch=1),
    "dream_gen512": Workload("dream_gen512", DREAM_7B, prompt_len=512, gen_len=512,
                             block_size=32, rule=THRESHOLD, threshold=0.9, local_budget=64,
                             middle_budget=32, tail_budget=8, cache=False, batch=1),
    "llada_long2048": Workload("llada_long2048", LLADA_8B, prompt_len=1024, gen_len=2048,
                               block_size=64, rule=TOPN, n_per_step=8, local_budget=128,
                               middle_budget=32, tail_budget=16, cache=True, batch=1),
    "llada_long1024": Workload("llada_long1024", LLADA_8B, prompt_len=1024, gen_len=1024,
                               block_size=64, rule=TOPN, n_per_step=8, local_budget=128,
                               middle_budget=32, tail_budget=16, cache=True, batch=1),
    # attention / gather microbenchmark at the LLaDA head shape: prefix KV 4096,
    # block 64, suffix 4096 pruned to 176 kept tokens, batch 8
    "attn_micro": Workload("attn_micro", LLADA_8B, prompt_len=4096, gen_len=4096 + 64,
                           block_size=64, rule=TOPN, n_per_step=8, local_budget=128,
                           middle_budget=32, tail_budget=16, cache=True, batch=8),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def sharpened(wl: Workload, scale: float = 60.0) -> Workload:
    """Test-only variant whose LM head is scaled so that decisions have wide margins."""
    return wl.replace(name=wl.name + "_sharp", logit_scale=scale)


def spread(wl: Workload, init_std: float = 0.1, scale: float = 3.0) -> Workload:
    """Test-only variant with five times the init scale of the matrices, so that
    attention is far from uniform and the rows of a block get distinct
    predictions: confidences and top-1/top-2 margins then spread over most of
    (0, 1) instead of clustering, and a free-running generation has decisions
    that are wide on both sides."""
    return wl.replace(name=wl.name + "_spread", logit_scale=scale,
                      model=dataclasses.replace(wl.model, init_std=init_std))
