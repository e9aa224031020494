"""Device-side model description and prefix KV cache for the C ABI."""
from __future__ import annotations

import ctypes as C

import torch

from . import _lib as L


class DeviceModel:
    """Keeps the weight tensors alive and exposes them as an `ssm_model`.

    `weights` has the attributes tok_emb, final_norm, lm_head and layers[l]
    (attn_norm, wq, wk, wv, wo, ffn_norm, w_gate, w_up, w_down), each a
    contiguous device tensor of the model dtype; `shape` gives the sizes.
    """

    # Leading layers whose projection inputs keep the bfloat16 pair by default.
    # Rounding them once in layer 0 alone gives most of the error of rounding
    # them in every layer (the residual stream is smallest there).  With the
    # attention operands in float16, two pair layers keep the full-depth
    # relative error of the 8B shapes at or below 1.0e-2 (half the bound);
    # none gives up to 2.9e-2, one up to 1.3e-2.
    PAIR_LAYERS = 2

    def __init__(self, shape, weights, act_mode: int = L.SSM_ACT_BF16X2_FIRST,
                 pair_layers: int = PAIR_LAYERS):
        self.shape = shape
        self.weights = weights
        dt = torch.float32 if shape.dtype == "f32" else torch.bfloat16
        tensors = [weights.tok_emb, weights.final_norm, weights.lm_head]
        for lw in weights.layers:
            tensors += lw.tensors()
        for t in tensors:
            if not t.is_cuda or not t.is_contiguous() or t.dtype != dt:
                raise ValueError("model tensors must be contiguous device tensors of the model dtype")
        n = len(weights.layers)
        self._layers = (L.Layer * max(n, 1))()
        for i, lw in enumerate(weights.layers):
            self._layers[i] = L.Layer(*[t.data_ptr() for t in lw.tensors()])
        self.c_model = L.Model(
            n, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim, shape.ffn_dim,
            shape.vocab, shape.mask_id, L.SSM_DT_F32 if shape.dtype == "f32" else L.SSM_DT_BF16,
            float(shape.rope_base), float(shape.rms_eps), weights.tok_emb.data_ptr(),
            weights.final_norm.data_ptr(), weights.lm_head.data_ptr(),
            C.cast(self._layers, C.POINTER(L.Layer)), int(act_mode), min(int(pair_layers), n))

    @property
    def dtype(self):
        return torch.float32 if self.shape.dtype == "f32" else torch.bfloat16


class DeviceKVCache:
    """k, v: [n_layers, batch, n_kv_heads, capacity, head_dim], float32 for a
    float32 model and float16 for a bfloat16 one (its attention operands)."""

    def __init__(self, shape, batch: int, capacity: int, device="cuda"):
        dt = torch.float32 if shape.dtype == "f32" else torch.float16
        size = (shape.n_layers, batch, shape.n_kv_heads, capacity, shape.head_dim)
        self.k = torch.zeros(size, dtype=dt, device=device)
        self.v = torch.zeros(size, dtype=dt, device=device)
        self.capacity = capacity
        self.c_cache = L.KVCache(self.k.data_ptr(), self.v.data_ptr(), capacity)
