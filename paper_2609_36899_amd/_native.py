"""ctypes declarations of the C ABI in include/pdec.h.

Loads ``libpdec.so`` from this package directory.  There is no fallback: if
the library is missing, loading raises, naming the build command.
"""

from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_float, c_int32, c_int64, c_void_p

_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_DIR, "libpdec.so")

OK = 0
INVALID_ARG = -1
OUT_OF_PAGES = -2
BAD_SEQ = -3
SEQ_TOO_LONG = -4
HIP_ERROR = -5
UNSUPPORTED = -6
PAGE_TOKENS = 16
TIMER_ATTENTION, TIMER_GEMM, TIMER_LM_HEAD = 0, 1, 2
F32 = 0
BF16 = 1
FP8_E4M3 = 2

_CODE_NAMES = {INVALID_ARG: "INVALID_ARG", OUT_OF_PAGES: "OUT_OF_PAGES", BAD_SEQ: "BAD_SEQ",
               SEQ_TOO_LONG: "SEQ_TOO_LONG", HIP_ERROR: "HIP_ERROR",
               UNSUPPORTED: "UNSUPPORTED"}


class PdecError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{_CODE_NAMES.get(code, code)}: {msg}")
        self.code = code


class ModelCfg(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("d_model", c_int32), ("n_q_heads", c_int32),
                ("n_kv_heads", c_int32), ("head_dim", c_int32), ("ffn_dim", c_int32),
                ("vocab", c_int32), ("rms_eps", c_float), ("rope_base", c_float),
                ("dtype", c_int32), ("qk_norm", c_int32), ("kv_fp8", c_int32),
                ("kv_scale_k", c_float), ("kv_scale_v", c_float)]


class Weights(ctypes.Structure):
    _fields_ = [("embed", c_void_p), ("lm_head", c_void_p), ("final_norm", c_void_p),
                ("attn_norm", POINTER(c_void_p)), ("wq", POINTER(c_void_p)),
                ("wk", POINTER(c_void_p)), ("wv", POINTER(c_void_p)), ("wo", POINTER(c_void_p)),
                ("ffn_norm", POINTER(c_void_p)), ("w_gate", POINTER(c_void_p)),
                ("w_up", POINTER(c_void_p)), ("w_down", POINTER(c_void_p)),
                ("q_norm", POINTER(c_void_p)), ("k_norm", POINTER(c_void_p))]


# name -> (restype, argtypes)
SIGNATURES = {
    "last_error": (c_char_p, []),
    "kv_bytes_per_token": (c_int64, [POINTER(ModelCfg)]),
    "engine_workspace_bytes": (c_int64, [POINTER(ModelCfg), c_int32, c_int32, c_int32, c_int32,
                                         c_int64]),
    "engine_create": (c_int32, [POINTER(ModelCfg), POINTER(Weights), c_void_p, c_int64, c_int32,
                                c_int32, c_int32, c_int32, c_void_p, c_int64, c_void_p,
                                POINTER(c_void_p)]),
    "engine_destroy": (None, [c_void_p]),
    "engine_set_stream": (c_int32, [c_void_p, c_void_p]),
    "engine_profile": (c_int32, [c_void_p, c_int32]),
    "engine_profile_every": (c_int32, [c_void_p, c_int32]),
    "engine_profile_read": (c_int32, [c_void_p, c_int32, POINTER(ctypes.c_double),
                                      POINTER(c_int64)]),
    "kv_alloc": (c_int32, [c_void_p, c_int32, POINTER(c_int32)]),
    "kv_free": (c_int32, [c_void_p, c_int32]),
    "kv_len": (c_int32, [c_void_p, c_int32, POINTER(c_int32)]),
    "kv_headroom": (c_int32, [c_void_p, POINTER(c_int64)]),
    "kv_block_table": (c_int32, [c_void_p, c_int32, POINTER(c_int32), c_int32, POINTER(c_int32)]),
    "kv_extend_uninit": (c_int32, [c_void_p, c_int32, c_int32]),
    "kv_append_prefix": (c_int32, [c_void_p, c_int32, POINTER(c_int32), c_int32, c_int32,
                                   c_void_p]),
    "kv_append_prefix_batch": (c_int32, [c_void_p, c_int32, POINTER(c_int32), POINTER(c_int32),
                                         POINTER(c_int32), c_int32, c_void_p]),
    "decode_step": (c_int32, [c_void_p, c_int32, POINTER(c_int32), c_void_p, c_void_p]),
    "sample": (c_int32, [c_void_p, c_int32, c_void_p, c_void_p, c_int32]),
    "kv_export": (c_int32, [c_void_p, c_int32, c_void_p, c_int64, POINTER(c_int32)]),
    "kv_import": (c_int32, [c_void_p, c_int32, c_void_p, c_int64, c_int32]),
    "pacing_plan": (c_int32, [c_int64, c_int64, c_int64, c_int32, POINTER(c_int32),
                              POINTER(c_int32), POINTER(c_int64), c_int32, POINTER(c_int32),
                              POINTER(c_int32), POINTER(c_int32), POINTER(c_int32),
                              POINTER(c_int32), POINTER(c_int32)]),
    "sample_top_p_workspace_bytes": (c_int64, [c_int32]),
    "sample_top_p": (c_int32, [c_int32, c_int32, c_void_p, c_float, c_float, c_void_p, c_void_p,
                               c_void_p, c_int64, c_void_p]),
    "sample_top_p_noalloc": (c_int32, [c_int32, c_int32, c_void_p, c_float, c_float, c_void_p,
                                       c_void_p, c_void_p]),
    "packed_weight_bytes": (c_int64, [c_int32, c_int32, c_int32]),
    "pack_weight": (c_int32, [c_int32, c_int32, c_int32, c_void_p, c_void_p, c_void_p]),
    "weight_projection_workspace_bytes": (c_int64, [c_int32, c_int32, c_int32, c_int32]),
    "weight_projection": (c_int32, [c_int32, c_int32, c_int32, c_int32, c_void_p, c_void_p,
                                    c_void_p, c_void_p, c_int64, c_void_p]),
    "swiglu_projection_workspace_bytes": (c_int64, [c_int32, c_int32, c_int32, c_int32]),
    "swiglu_projection": (c_int32, [c_int32, c_int32, c_int32, c_int32, c_void_p, c_void_p,
                                    c_void_p, c_void_p, c_void_p, c_int64, c_void_p]),
    "paged_attention_workspace_bytes": (c_int64, [c_int32, c_int32, c_int32, c_int32, c_int64]),
    "paged_decode_attention": (c_int32, [c_int32, c_int32, c_int32, c_int32, c_int32, c_void_p,
                                         c_void_p, c_void_p, c_void_p, c_int32, POINTER(c_int32),
                                         c_void_p, c_void_p, c_int64, c_void_p]),
    "paged_decode_attention_fp8": (c_int32, [c_int32, c_int32, c_int32, c_int32, c_void_p, c_void_p,
                                             c_void_p, c_float, c_float, c_void_p, c_int32,
                                             POINTER(c_int32), c_void_p, c_void_p, c_int64,
                                             c_void_p]),
}

_lib = None


def load() -> ctypes.CDLL:
    """The device library, loaded once.  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing; build it with "
                               f"`python -m paper_2609_36899_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def check(rc: int) -> int:
    if rc < 0:
        raise PdecError(rc, load().last_error().decode())
    return rc
