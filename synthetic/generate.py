"""Seeded tensor generators.

Every tensor is drawn from its own torch generator whose seed is derived from
(run seed, tensor tag), so any single tensor (for example one layer of an
8B-parameter model) can be regenerated independently and on any device.
Tensors generated on one device type are bit-identical across runs on that
device type; tests that compare two implementations hand both the very same
tensor (copied between host and device), never two independent draws.
"""
from __future__ import annotations

import zlib
from dataclasses import dataclass, field
from typing import Callable, List, Optional

import torch

from .configs import ModelShape, Workload


def _derive(seed: int, tag: str) -> int:
    return ((zlib.crc32(tag.encode()) << 20) ^ (int(seed) * 0x9E3779B1)) & 0x7FFF_FFFF_FFFF_FFFF


def seeded_normal(shape, seed: int, tag: str, std: float = 1.0, mean: float = 0.0,
                  device="cpu", dtype=torch.float32) -> torch.Tensor:
    g = torch.Generator(device=device)
    g.manual_seed(_derive(seed, tag))
    t = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    if mean != 0.0:
        t.add_(mean)
    return t.to(dtype)


def seeded_uniform_ints(shape, low: int, high: int, seed: int, tag: str,
                        device="cpu") -> torch.Tensor:
    g = torch.Generator(device=device)
    g.manual_seed(_derive(seed, tag))
    return torch.randint(low, high, tuple(shape), generator=g, device=device, dtype=torch.int32)


def _storage_dtype(shape: ModelShape):
    return torch.float32 if shape.dtype == "f32" else torch.bfloat16


@dataclass
class LayerWeights:
    attn_norm: torch.Tensor   # [d]
    wq: torch.Tensor          # [H*dh, d]
    wk: torch.Tensor          # [Hkv*dh, d]
    wv: torch.Tensor          # [Hkv*dh, d]
    wo: torch.Tensor          # [d, H*dh]
    ffn_norm: torch.Tensor    # [d]
    w_gate: torch.Tensor      # [F, d]
    w_up: torch.Tensor        # [F, d]
    w_down: torch.Tensor      # [d, F]

    def tensors(self):
        return [self.attn_norm, self.wq, self.wk, self.wv, self.wo, self.ffn_norm,
                self.w_gate, self.w_up, self.w_down]

    def to(self, device=None, dtype=None) -> "LayerWeights":
        return LayerWeights(*[t.to(device=device, dtype=dtype) for t in self.tensors()])


def make_layer(shape: ModelShape, layer: int, seed: int = 0, device="cpu",
               norm_jitter: float = 0.0) -> LayerWeights:
    d, hd, F = shape.d_model, shape.head_dim, shape.ffn_dim
    H, Hk = shape.n_heads, shape.n_kv_heads
    std = shape.init_std
    dt = _storage_dtype(shape)
    p = f"layer{layer}."

    def W(rows, cols, name):
        return seeded_normal((rows, cols), seed, p + name, std=std, device=device, dtype=dt)

    def norm(name):
        if norm_jitter == 0.0:
            return torch.ones(d, device=device, dtype=dt)
        return seeded_normal((d,), seed, p + name, std=norm_jitter, mean=1.0, device=device, dtype=dt)

    return LayerWeights(
        attn_norm=norm("attn_norm"), wq=W(H * hd, d, "wq"), wk=W(Hk * hd, d, "wk"),
        wv=W(Hk * hd, d, "wv"), wo=W(d, H * hd, "wo"), ffn_norm=norm("ffn_norm"),
        w_gate=W(F, d, "w_gate"), w_up=W(F, d, "w_up"), w_down=W(d, F, "w_down"))


@dataclass
class ModelWeights:
    shape: ModelShape
    tok_emb: torch.Tensor        # [V, d]
    final_norm: torch.Tensor     # [d]
    lm_head: torch.Tensor        # [V, d]
    layers: List[LayerWeights] = field(default_factory=list)

    def to(self, device=None, dtype=None) -> "ModelWeights":
        return ModelWeights(self.shape, self.tok_emb.to(device=device, dtype=dtype),
                            self.final_norm.to(device=device, dtype=dtype),
                            self.lm_head.to(device=device, dtype=dtype),
                            [lw.to(device, dtype) for lw in self.layers])


def make_weights(shape: ModelShape, seed: int = 0, device="cpu", norm_jitter: float = 0.0,
                 logit_scale: float = 1.0, with_layers: bool = True) -> ModelWeights:
    """Random-init model: N(0, init_std) matrices, unit (or jittered) norm weights."""
    d, V = shape.d_model, shape.vocab
    dt = _storage_dtype(shape)
    tok_emb = seeded_normal((V, d), seed, "tok_emb", std=shape.init_std, device=device, dtype=dt)
    lm_head = seeded_normal((V, d), seed, "lm_head", std=shape.init_std * logit_scale,
                            device=device, dtype=dt)
    if norm_jitter == 0.0:
        final_norm = torch.ones(d, device=device, dtype=dt)
    else:
        final_norm = seeded_normal((d,), seed, "final_norm", std=norm_jitter, mean=1.0,
                                   device=device, dtype=dt)
    layers = []
    if with_layers:
        layers = [make_layer(shape, l, seed, device, norm_jitter) for l in range(shape.n_layers)]
    return ModelWeights(shape, tok_emb, final_norm, lm_head, layers)


def prompt_tokens(wl: Workload, seed: Optional[int] = None, device="cpu") -> torch.Tensor:
    """Uniform random prompt ids in [0, V) with the mask id excluded; [B, prompt_len] int32."""
    s = wl.seed if seed is None else seed
    V, mask = wl.model.vocab, wl.model.mask_id
    ids = seeded_uniform_ints((wl.batch, wl.prompt_len), 0, V - 1, s, "prompt", device=device)
    return ids + (ids >= mask).to(torch.int32)


def initial_tokens(wl: Workload, seed: Optional[int] = None, device="cpu") -> torch.Tensor:
    """[B, prompt_len + gen_len] int32: the prompt followed by mask ids."""
    p = prompt_tokens(wl, seed, device)
    gen = torch.full((wl.batch, wl.gen_len), wl.model.mask_id, dtype=torch.int32, device=device)
    return torch.cat([p, gen], dim=1).contiguous()


def mid_generation_state(wl: Workload, block_idx: int, step: int, seed: int = 0,
                         decoded_frac: float = 0.5, predicted_frac: float = 0.8):
    """A seeded decoding state at the start of a step inside block `block_idx`:
    earlier blocks fully decoded with random ids, part of the current block
    decoded, and a previous-step prediction (random top-k ids with random
    descending weights summing to one) on part of the suffix.

    Returns numpy arrays (tokens [B, L], pred_ids [B, L, k], pred_w [B, L, k],
    pred_step [B, L]); predictions carry the stamp step - 1.
    """
    import numpy as np
    rng = np.random.default_rng(_derive(seed, f"state{block_idx}.{step}") & 0xFFFFFFFF)
    B, Lt, k = wl.batch, wl.total_len, wl.topk
    V, mask = wl.model.vocab, wl.model.mask_id
    tokens = initial_tokens(wl, seed).numpy().copy()
    P = wl.prompt_len + block_idx * wl.block_size
    dec = rng.integers(0, V - 1, size=(B, Lt)).astype(np.int32)
    dec = dec + (dec >= mask)
    tokens[:, wl.prompt_len:P] = dec[:, wl.prompt_len:P]
    blk = rng.random((B, wl.block_size)) < decoded_frac
    tokens[:, P:P + wl.block_size][blk] = dec[:, P:P + wl.block_size][blk]
    pred_ids = rng.integers(0, V - 1, size=(B, Lt, k)).astype(np.int32)
    pred_ids = pred_ids + (pred_ids >= mask)
    w = np.sort(rng.random((B, Lt, k)), axis=-1)[..., ::-1]
    pred_w = (w / w.sum(-1, keepdims=True)).astype(np.float32)
    pred_step = np.where(rng.random((B, Lt)) < predicted_frac, step - 1, -1).astype(np.int32)
    pred_step[:, :P + wl.block_size] = -1
    return tokens.astype(np.int32), pred_ids, pred_w, pred_step
