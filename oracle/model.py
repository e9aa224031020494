"""Bidirectional masked-diffusion transformer step over the sparse input
(Section 3.2, "Sparse Input Construction"; the models of Section 4.1).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper cites the architectures (LLaDA-8B, Dream-7B) rather than restating
them; the oracle uses the standard pre-norm decoder block of those models
without a causal mask:

    h  = x + W_o Attn(RoPE(W_q n1(x)), RoPE(W_k n1(x)), W_v n1(x))
    x' = h + W_down( silu(W_gate n2(h)) * W_up n2(h) )
    n(x) = x / sqrt(mean(x^2) + eps) * g                 (RMSNorm)

Attention is softmax(q k^T / sqrt(d_h)) v over every key (bidirectional);
with grouped-query attention, query head h reads key/value head
h // (H / H_kv).  RoPE is the rotate-half form, applied at each row's
original position, which is what lets the sparse input keep the retained
suffix tokens' relative positions (Section 3.2).

Prefix KV cache (the "PC." setting of Section 4.8, Table 4): on the first step of a
block the full sparse input is run and the post-RoPE keys and values of the
prefix rows are kept for every layer; on later steps of the block the input
is [B_t; R_t] only and attention reads the cached prefix keys and values
together with the rows' own.

Logits: the final RMSNorm and LM head are applied to the block and retained
suffix rows only; prefix rows need no prediction.
"""
from __future__ import annotations

from typing import List, NamedTuple, Optional, Sequence, Tuple

import numpy as np


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope_angles(pos: np.ndarray, head_dim: int, base: float) -> Tuple[np.ndarray, np.ndarray]:
    """cos/sin of pos * base^(-2i/d_h), i < d_h/2, in float64."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = 1.0 / (base ** (2.0 * i / head_dim))
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]
    return np.cos(ang), np.sin(ang)


def apply_rope(x: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """Rotate-half RoPE on x [n, heads, d_h] at absolute positions pos [n]."""
    dh = x.shape[-1]
    half = dh // 2
    cos, sin = rope_angles(pos, dh, base)
    cos = cos[:, None, :].astype(x.dtype)
    sin = sin[:, None, :].astype(x.dtype)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def softmax_rows(s: np.ndarray) -> np.ndarray:
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """Non-causal attention. q [n_q, H, d_h], k/v [n_k, H_kv, d_h] -> [n_q, H*d_h]."""
    n_q, H, dh = q.shape
    Hkv = k.shape[1]
    group = H // Hkv
    out = np.empty((n_q, H, dh), dtype=q.dtype)
    scale = 1.0 / np.sqrt(dh)
    for h in range(H):
        kh = k[:, h // group, :]
        vh = v[:, h // group, :]
        s = (q[:, h, :] @ kh.T) * q.dtype.type(scale)
        out[:, h, :] = softmax_rows(s) @ vh
    return out.reshape(n_q, H * dh)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


class LayerOut(NamedTuple):
    x: np.ndarray       # [n, d] residual stream after the layer
    k: np.ndarray       # [n, H_kv, d_h] post-RoPE keys of the input rows
    v: np.ndarray       # [n, H_kv, d_h] values of the input rows


def layer_forward(x: np.ndarray, pos: np.ndarray, lw, shape,
                  k_prefix: Optional[np.ndarray] = None,
                  v_prefix: Optional[np.ndarray] = None) -> LayerOut:
    """One pre-norm decoder layer over the rows x [n, d] at positions pos."""
    n = x.shape[0]
    H, Hkv, dh = shape.n_heads, shape.n_kv_heads, shape.head_dim
    xn = rms_norm(x, lw.attn_norm, shape.rms_eps)
    q = (xn @ lw.wq.T).reshape(n, H, dh)
    k = (xn @ lw.wk.T).reshape(n, Hkv, dh)
    v = (xn @ lw.wv.T).reshape(n, Hkv, dh)
    q = apply_rope(q, pos, shape.rope_base)
    k = apply_rope(k, pos, shape.rope_base)
    if k_prefix is not None and len(k_prefix):
        k_all = np.concatenate([k_prefix, k], axis=0)
        v_all = np.concatenate([v_prefix, v], axis=0)
    else:
        k_all, v_all = k, v
    o = attention(q, k_all, v_all)
    h = x + o @ lw.wo.T
    hn = rms_norm(h, lw.ffn_norm, shape.rms_eps)
    f = silu(hn @ lw.w_gate.T) * (hn @ lw.w_up.T)
    return LayerOut(h + f @ lw.w_down.T, k, v)


class ForwardOut(NamedTuple):
    hidden: np.ndarray                           # [n, d] after the last layer
    kv: List[Tuple[np.ndarray, np.ndarray]]      # per layer (k, v) of the input rows


def forward(x: np.ndarray, pos: np.ndarray, weights, shape,
            prefix_kv: Optional[Sequence[Tuple[np.ndarray, np.ndarray]]] = None) -> ForwardOut:
    """All layers.  prefix_kv[l] = cached (k, v) of the prefix for layer l, or None."""
    kv = []
    for l in range(shape.n_layers):
        lw = weights.layers[l]
        kp, vp = (prefix_kv[l] if prefix_kv is not None else (None, None))
        out = layer_forward(x, pos, lw, shape, kp, vp)
        x = out.x
        kv.append((out.k, out.v))
    return ForwardOut(x, kv)


class OutputStats(NamedTuple):
    logits: np.ndarray      # [n_out, V]
    argmax: np.ndarray      # [n_out] int32, [MASK] excluded
    conf: np.ndarray        # [n_out] max softmax probability, [MASK] excluded
    topk_ids: np.ndarray    # [n_out, k] int32
    topk_w: np.ndarray      # [n_out, k] Eq. 6 renormalised probabilities
    p_sorted2: np.ndarray   # [n_out, 2] the two largest probabilities (decision margins)


def output_stats(h_out: np.ndarray, weights, shape, k: int) -> OutputStats:
    """Final norm, LM head and the per-row quantities the decoding rule and Eq. 6 use."""
    from .embed import full_softmax, top_k_set, renormalise
    hn = rms_norm(h_out, weights.final_norm, shape.rms_eps)
    logits = hn @ weights.lm_head.T
    n = logits.shape[0]
    am = np.zeros(n, dtype=np.int32)
    conf = np.zeros(n, dtype=np.float64)
    ids = np.zeros((n, k), dtype=np.int32)
    w = np.zeros((n, k), dtype=np.float64)
    p2 = np.zeros((n, 2), dtype=np.float64)
    for r in range(n):
        p = full_softmax(logits[r], shape.mask_id)
        t = top_k_set(p, max(k, 2))
        am[r] = t[0]
        conf[r] = p[t[0]]
        p2[r] = p[t[:2]]
        ids[r] = t[:k]
        w[r] = renormalise(p, t[:k])
    return OutputStats(logits, am, conf, ids, w, p2)
