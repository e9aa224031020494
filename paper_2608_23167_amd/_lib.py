"""ctypes view of libssm.so (the C ABI declared in include/ssm.h).

The library is loaded from this package directory; if it is missing the
import fails loudly: there is no CPU fallback.
"""
from __future__ import annotations

import ctypes as C
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libssm.so")

SSM_OK, SSM_E_INVAL, SSM_E_SHAPE, SSM_E_CAPACITY, SSM_E_HIP, SSM_E_UNSUPPORTED = 0, -1, -2, -3, -4, -5
SSM_MIDDLE_STRIDED, SSM_MIDDLE_BLOCK_START, SSM_MIDDLE_BLOCK_END, SSM_MIDDLE_BLOCK_START_END = 0, 1, 2, 3
SSM_TAIL_SPREAD, SSM_TAIL_START = 0, 1
SSM_UNMASK_TOPN, SSM_UNMASK_THRESHOLD, SSM_UNMASK_MARGIN = 0, 1, 2
SSM_DT_F32, SSM_DT_BF16, SSM_DT_F16 = 0, 1, 2
SSM_ACT_BF16, SSM_ACT_BF16X2, SSM_ACT_BF16X2_FIRST = 0, 1, 2
SSM_CACHE_OFF, SSM_CACHE_WRITE, SSM_CACHE_READ = 0, 1, 2

_ERR_NAMES = {SSM_E_INVAL: "SSM_E_INVAL", SSM_E_SHAPE: "SSM_E_SHAPE",
              SSM_E_CAPACITY: "SSM_E_CAPACITY", SSM_E_HIP: "SSM_E_HIP",
              SSM_E_UNSUPPORTED: "SSM_E_UNSUPPORTED"}


class SSMError(RuntimeError):
    def __init__(self, code: int, fn: str, msg: str):
        super().__init__(f"{fn} -> {_ERR_NAMES.get(code, code)}: {msg}")
        self.code = code


class SelectParams(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "prompt_len", "gen_len", "block_size", "block_idx", "local_budget", "middle_budget",
        "middle_mode", "tail_budget", "include_prefix", "tail_mode")]


class Layer(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in (
        "attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")]


class Model(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "n_layers", "d_model", "n_heads", "n_kv_heads", "head_dim", "ffn_dim", "vocab",
        "mask_id", "dtype")] + [
        ("rope_base", C.c_float), ("rms_eps", C.c_float),
        ("tok_emb", C.c_void_p), ("final_norm", C.c_void_p), ("lm_head", C.c_void_p),
        ("layers", C.POINTER(Layer)), ("act_mode", C.c_int32), ("pair_layers", C.c_int32)]


class KVCache(C.Structure):
    _fields_ = [("k", C.c_void_p), ("v", C.c_void_p), ("capacity", C.c_int32)]


P = C.c_void_p
I32 = C.c_int32
PI32 = C.POINTER(C.c_int32)

_SIGS = {
    "ssm_select_count": (I32, [C.POINTER(SelectParams), PI32, PI32, PI32]),
    "ssm_select_positions_host": (I32, [C.POINTER(SelectParams), PI32, C.POINTER(C.c_int8), I32, PI32]),
    "ssm_select_suffix": (I32, [C.POINTER(SelectParams), I32, I32, PI32, P, P, P, P, I32, PI32, PI32,
                                PI32, P]),
    "ssm_embed_suffix": (I32, [C.POINTER(Model), I32, I32, PI32, P, I32, P, P, I32, P, P, P, I32,
                               I32, C.c_float, P, P]),
    "ssm_workspace_size": (I32, [C.POINTER(Model), I32, I32, C.POINTER(C.c_size_t)]),
    "ssm_denoise_step": (I32, [C.POINTER(Model), C.POINTER(KVCache), I32, I32, I32, PI32, P, I32, P,
                               I32, I32, P, P, P, P, P, P, P, C.c_size_t, P]),
    "ssm_unmask": (I32, [P, I32, I32, PI32, I32, I32, I32, I32, I32, C.c_float, P, P, P, P, I32, I32,
                         P, I32, P, P, P, P, P, P]),
    "ssm_early_stop": (I32, [P, I32, I32, PI32, I32, I32, I32, P, P]),
    "ssm_attention_workspace_size": (I32, [I32, I32, I32, C.POINTER(C.c_size_t)]),
    "ssm_attention": (I32, [I32, I32, I32, I32, I32, I32, I32, P, P, P, P, P, C.c_size_t, P]),
    "ssm_attention_static": (I32, [I32, I32, I32, I32, I32, I32, I32, P, P, P, P, P]),
    "ssm_gather_rows": (I32, [I32, I32, I32, P, P, I32, P, P]),
    "ssm_profile_enable": (I32, [I32]),
    "ssm_profile_query": (I32, [C.c_char_p, I32, PI32, C.POINTER(C.c_double)]),
    "ssm_last_error": (C.c_char_p, []),
}

_lib = None
_path = LIB_PATH


def use_library(path: str) -> None:
    """Loads the C ABI from `path` instead of the package's libssm.so (e.g. a
    host-only build instrumented with sanitizers); only before the first call."""
    global _path
    if _lib is not None:
        raise RuntimeError("the library is already loaded")
    _path = path


def lib() -> C.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_path):
            raise ImportError(f"{_path} is missing: build it with "
                              "`python -m paper_2608_23167_amd.build` (no CPU fallback exists)")
        l = C.CDLL(_path)
        for name, (res, args) in _SIGS.items():
            f = getattr(l, name)
            f.restype = res
            f.argtypes = args
        _lib = l
    return _lib


def check(rc: int, fn: str) -> None:
    if rc != SSM_OK:
        raise SSMError(rc, fn, lib().ssm_last_error().decode())


def exported_symbols():
    return list(_SIGS)
