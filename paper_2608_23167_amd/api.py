"""Python binding of the C ABI: the same four calls (plus the size queries),
taking torch tensors for device memory and torch's current HIP stream.

Argument marshalling only: every step of the path runs in libssm.so.
"""
from __future__ import annotations

import ctypes as C
import numpy as np
from typing import Optional, Tuple

import torch

from . import _lib as L
from ._lib import check, lib


def _stream(stream) -> C.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def _ptr(t: Optional[torch.Tensor], dtype=None, name="tensor") -> C.c_void_p:
    if t is None:
        return C.c_void_p(None)
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    return C.c_void_p(t.data_ptr())


def _pad(pad, batch: int):
    """Host int32 array of per-sequence left padding (None: no padding)."""
    if pad is None:
        return None
    a = (C.c_int32 * batch)(*[int(v) for v in pad])
    if len(pad) != batch:
        raise ValueError(f"pad has {len(pad)} entries for a batch of {batch}")
    return a


def select_params(prompt_len, gen_len, block_size, block_idx, local_budget, middle_budget,
                  middle_mode, tail_budget, include_prefix, tail_mode=0) -> L.SelectParams:
    return L.SelectParams(prompt_len, gen_len, block_size, block_idx, local_budget, middle_budget,
                          middle_mode, tail_budget, int(bool(include_prefix)), tail_mode)


def ssm_select_count(p: L.SelectParams) -> Tuple[int, int, int]:
    n, s, f = C.c_int32(), C.c_int32(), C.c_int32()
    check(lib().ssm_select_count(C.byref(p), C.byref(n), C.byref(s), C.byref(f)), "ssm_select_count")
    return n.value, s.value, f.value


def ssm_select_positions_host(p: L.SelectParams) -> Tuple[np.ndarray, np.ndarray]:
    """(positions int32, regions int8) of the compacted rows, computed on the host."""
    n_rows, _, _ = ssm_select_count(p)
    pos = np.zeros(max(n_rows, 1), dtype=np.int32)
    reg = np.zeros(max(n_rows, 1), dtype=np.int8)
    n = C.c_int32()
    check(lib().ssm_select_positions_host(
        C.byref(p), pos.ctypes.data_as(C.POINTER(C.c_int32)),
        reg.ctypes.data_as(C.POINTER(C.c_int8)), pos.size, C.byref(n)), "ssm_select_positions_host")
    return pos[:n.value], reg[:n.value]


def ssm_select_suffix(p: L.SelectParams, tokens: torch.Tensor, pos: torch.Tensor,
                      tok_c: torch.Tensor, region: Optional[torch.Tensor], stream=None,
                      pad=None) -> Tuple[int, int, int]:
    B, seq_len = tokens.shape
    cap = pos.numel()
    if tok_c.shape != (B, cap):
        raise ValueError("tok_c must be [batch, cap]")
    n, s, f = C.c_int32(), C.c_int32(), C.c_int32()
    rc = lib().ssm_select_suffix(C.byref(p), B, seq_len, _pad(pad, B),
                                 _ptr(tokens, torch.int32, "tokens"),
                                 _ptr(pos, torch.int32, "pos"), _ptr(tok_c, torch.int32, "tok_c"),
                                 _ptr(region, torch.int8, "region"), cap, C.byref(n), C.byref(s),
                                 C.byref(f), _stream(stream))
    check(rc, "ssm_select_suffix")
    return n.value, s.value, f.value


def ssm_embed_suffix(model, tok_c: torch.Tensor, pos: torch.Tensor, region: torch.Tensor,
                     n_rows: int, pred_ids: torch.Tensor, pred_w: torch.Tensor,
                     pred_step: torch.Tensor, prev_step: int, k: int, alpha: float,
                     x: torch.Tensor, stream=None, pad=None) -> None:
    B, seq_len = pred_step.shape
    rc = lib().ssm_embed_suffix(C.byref(model.c_model), B, seq_len, _pad(pad, B),
                                _ptr(tok_c, torch.int32, "tok_c"), tok_c.shape[1],
                                _ptr(pos, torch.int32, "pos"), _ptr(region, torch.int8, "region"),
                                n_rows, _ptr(pred_ids, torch.int32, "pred_ids"),
                                _ptr(pred_w, torch.float32, "pred_w"),
                                _ptr(pred_step, torch.int32, "pred_step"), prev_step, k,
                                float(alpha), _ptr(x, torch.float32, "x"), _stream(stream))
    check(rc, "ssm_embed_suffix")


def ssm_workspace_size(model, batch: int, max_rows: int) -> int:
    n = C.c_size_t()
    check(lib().ssm_workspace_size(C.byref(model.c_model), batch, max_rows, C.byref(n)),
          "ssm_workspace_size")
    return n.value


def ssm_denoise_step(model, cache, cache_mode: int, n_cached: int, pos: torch.Tensor,
                     n_rows: int, x: torch.Tensor, first_out_row: int, k: int,
                     argmax: torch.Tensor, conf: torch.Tensor, topk_ids: torch.Tensor,
                     topk_w: torch.Tensor, ws: torch.Tensor,
                     logits: Optional[torch.Tensor] = None, hidden: Optional[torch.Tensor] = None,
                     stream=None, pad=None) -> None:
    B = x.shape[0]
    rc = lib().ssm_denoise_step(C.byref(model.c_model), C.byref(cache.c_cache), cache_mode,
                                n_cached, B, _pad(pad, B), _ptr(pos, torch.int32, "pos"), n_rows,
                                _ptr(x, torch.float32, "x"), first_out_row, k,
                                _ptr(argmax, torch.int32, "argmax"),
                                _ptr(conf, torch.float32, "conf"),
                                _ptr(topk_ids, torch.int32, "topk_ids"),
                                _ptr(topk_w, torch.float32, "topk_w"),
                                _ptr(logits, torch.float32, "logits"),
                                _ptr(hidden, torch.float32, "hidden"),
                                _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(stream))
    check(rc, "ssm_denoise_step")


def ssm_attention_workspace_size(batch: int, n_heads: int, n_q: int) -> int:
    n = C.c_size_t()
    check(lib().ssm_attention_workspace_size(batch, n_heads, n_q, C.byref(n)),
          "ssm_attention_workspace_size")
    return n.value


_ATTN_DT = {torch.bfloat16: L.SSM_DT_BF16, torch.float16: L.SSM_DT_F16}


def ssm_attention(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, n_keys: int,
                  out: torch.Tensor, ws: torch.Tensor, stream=None) -> None:
    """q [B, H, n_q, 128]; k, v [B, H_kv, capacity, 128], all bf16 or all
    float16; out float32 [B, n_q, H * 128]; ws uint8 of
    ssm_attention_workspace_size(B, H, n_q) bytes."""
    B, H, n_q, dh = q.shape
    if dh != 128 or k.shape != v.shape or k.shape[0] != B or k.shape[3] != 128:
        raise ValueError("shapes: q [B, H, n_q, 128], k = v [B, H_kv, capacity, 128]")
    if tuple(out.shape) != (B, n_q, H * 128):
        raise ValueError("out must be [B, n_q, H * 128]")
    if q.dtype not in _ATTN_DT:
        raise ValueError("q, k, v must be bfloat16 or float16")
    check(lib().ssm_attention(_ATTN_DT[q.dtype], B, H, k.shape[1], n_q, int(n_keys), k.shape[2],
                              _ptr(q, q.dtype, "q"), _ptr(k, q.dtype, "k"),
                              _ptr(v, q.dtype, "v"), _ptr(out, torch.float32, "out"),
                              _ptr(ws, None, "ws"), ws.numel() * ws.element_size(),
                              _stream(stream)), "ssm_attention")


def ssm_attention_static(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, n_keys: int,
                         out: torch.Tensor, stream=None) -> None:
    """ssm_attention without a workspace: the split-KV partials go to the
    library's static per-GPU scratch array (no allocation)."""
    B, H, n_q, dh = q.shape
    if dh != 128 or k.shape != v.shape or k.shape[0] != B or k.shape[3] != 128:
        raise ValueError("shapes: q [B, H, n_q, 128], k = v [B, H_kv, capacity, 128]")
    if tuple(out.shape) != (B, n_q, H * 128):
        raise ValueError("out must be [B, n_q, H * 128]")
    if q.dtype not in _ATTN_DT:
        raise ValueError("q, k, v must be bfloat16 or float16")
    check(lib().ssm_attention_static(_ATTN_DT[q.dtype], B, H, k.shape[1], n_q, int(n_keys),
                                     k.shape[2], _ptr(q, q.dtype, "q"), _ptr(k, q.dtype, "k"),
                                     _ptr(v, q.dtype, "v"), _ptr(out, torch.float32, "out"),
                                     _stream(stream)), "ssm_attention_static")


def ssm_gather_rows(src: torch.Tensor, pos: torch.Tensor, out: torch.Tensor, stream=None) -> None:
    """out[s, i, :] = src[s, pos[i], :]; src bf16 [B, src_rows, width], pos int32
    [n_rows], out bf16 [B, n_rows, width]; out-of-range positions give zeros."""
    B, rows, width = src.shape
    if tuple(out.shape) != (B, pos.numel(), width):
        raise ValueError("out must be [B, n_rows, width]")
    check(lib().ssm_gather_rows(B, rows, width, _ptr(src, torch.bfloat16, "src"),
                                _ptr(pos, torch.int32, "pos"), pos.numel(),
                                _ptr(out, torch.bfloat16, "out"), _stream(stream)),
          "ssm_gather_rows")


def ssm_unmask(tokens: torch.Tensor, block_start: int, block_size: int, mask_id: int, rule: int,
               n_per_step: int, threshold: float, argmax: torch.Tensor, conf: torch.Tensor,
               topk_ids: torch.Tensor, topk_w: torch.Tensor, k: int, n_out: int,
               pos_out: torch.Tensor, step: int, pred_ids: torch.Tensor, pred_w: torch.Tensor,
               pred_step: torch.Tensor, selected: Optional[torch.Tensor] = None,
               masked_left: Optional[torch.Tensor] = None, stream=None, pad=None) -> None:
    B, seq_len = tokens.shape
    rc = lib().ssm_unmask(_ptr(tokens, torch.int32, "tokens"), B, seq_len, _pad(pad, B), block_start,
                          block_size, mask_id, rule, n_per_step, float(threshold),
                          _ptr(argmax, torch.int32, "argmax"), _ptr(conf, torch.float32, "conf"),
                          _ptr(topk_ids, torch.int32, "topk_ids"),
                          _ptr(topk_w, torch.float32, "topk_w"), k, n_out,
                          _ptr(pos_out, torch.int32, "pos_out"), step,
                          _ptr(pred_ids, torch.int32, "pred_ids"),
                          _ptr(pred_w, torch.float32, "pred_w"),
                          _ptr(pred_step, torch.int32, "pred_step"),
                          _ptr(selected, torch.uint8, "selected"),
                          _ptr(masked_left, torch.int32, "masked_left"), _stream(stream))
    check(rc, "ssm_unmask")


def ssm_early_stop(tokens: torch.Tensor, block_start: int, block_size: int, eos_id: int,
                   done: torch.Tensor, stream=None, pad=None) -> None:
    B, seq_len = tokens.shape
    if done.numel() != B:
        raise ValueError("done must hold one int32 per sequence")
    rc = lib().ssm_early_stop(_ptr(tokens, torch.int32, "tokens"), B, seq_len, _pad(pad, B),
                              block_start, block_size, eos_id, _ptr(done, torch.int32, "done"),
                              _stream(stream))
    check(rc, "ssm_early_stop")


PROFILE_TAGS = ("select", "embed", "rope_table", "norm", "gemm_qkv", "attention", "gemm_o",
                "gemm_gate_up", "gemm_down", "gemm_lm_head", "rowstats", "unmask", "early_stop")


def ssm_profile_enable(on: bool) -> None:
    check(lib().ssm_profile_enable(int(bool(on))), "ssm_profile_enable")


def ssm_profile_query(tag: str, kernel: int = -1) -> Tuple[int, float]:
    """(kernels recorded, summed ms) under `tag`; kernel >= 0 selects one
    ordinal within each call (0 = the operation's main kernel)."""
    n, ms = C.c_int32(), C.c_double()
    check(lib().ssm_profile_query(tag.encode(), int(kernel), C.byref(n), C.byref(ms)),
          "ssm_profile_query")
    return n.value, ms.value
