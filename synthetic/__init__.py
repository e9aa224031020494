"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the benchmark.

This package holds shapes, budgets and random-number recipes only: none of the
method's arithmetic lives here.  Both the CPU oracle and the HIP path receive
their weights, prompts and random test tensors from these generators, so the
two sides see identical inputs while sharing no computation.
"""
from .configs import (ModelShape, Workload, TINY, LLADA_8B, DREAM_7B, WORKLOADS,
                      workload, sharpened, spread)
from .generate import (ModelWeights, LayerWeights, make_weights, make_layer,
                       prompt_tokens, initial_tokens, seeded_normal, seeded_uniform_ints,
                       mid_generation_state)

__all__ = [
    "ModelShape", "Workload", "TINY", "LLADA_8B", "DREAM_7B", "WORKLOADS", "workload",
    "sharpened", "spread", "ModelWeights", "LayerWeights", "make_weights", "make_layer",
    "prompt_tokens", "initial_tokens", "seeded_normal", "seeded_uniform_ints",
    "mid_generation_state",
]
