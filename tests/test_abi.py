"""The device library loads on a machine without a GPU and exports every
function include/pdec.h declares; the ctypes binding declares the same set.
No compute call is made here."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pdec.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\**\s+\**([a-z_][a-z0-9_]*)\s*\(",
                       text, flags=re.M)
    return sorted(set(names))


def test_header_declares_the_core_calls():
    names = declared_functions()
    for core in ("kv_alloc", "kv_append_prefix", "decode_step", "sample", "kv_free",
                 "kv_headroom", "kv_len", "engine_create", "engine_destroy",
                 "paged_decode_attention", "last_error", "kv_bytes_per_token"):
        assert core in names


def test_library_exports_every_declared_symbol():
    from paper_2609_36899_amd import _native
    if not os.path.exists(_native.LIB_PATH):
        from paper_2609_36899_amd import build
        build.build_device()
    lib = ctypes.CDLL(_native.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing
    assert sorted(_native.SIGNATURES) == declared_functions()


def test_host_only_calls_without_gpu():
    """kv_bytes_per_token and the size queries run on the host only."""
    from ctypes import byref
    from paper_2609_36899_amd import _native as N
    from workload import EIGHT_B, TINY
    lib = N.load()
    cfg = N.ModelCfg(EIGHT_B.n_layers, EIGHT_B.d_model, EIGHT_B.n_q_heads, EIGHT_B.n_kv_heads,
                     EIGHT_B.head_dim, EIGHT_B.ffn_dim, EIGHT_B.vocab, 1e-6, 10000.0, N.BF16)
    assert lib.kv_bytes_per_token(byref(cfg)) == 131072
    tiny = N.ModelCfg(TINY.n_layers, TINY.d_model, TINY.n_q_heads, TINY.n_kv_heads,
                      TINY.head_dim, TINY.ffn_dim, TINY.vocab, 1e-6, 10000.0, N.F32)
    assert lib.kv_bytes_per_token(byref(tiny)) == 2048
    ws = lib.engine_workspace_bytes(byref(cfg), 512, 72 * 1024, 512, 2048, 250 << 30)
    assert 0 < ws < 4 << 30
    bad = N.ModelCfg(2, 256, 6, 4, 64, 688, 1024, 1e-6, 1e4, N.F32)  # 6 % 4 != 0
    assert lib.kv_bytes_per_token(byref(bad)) == N.INVALID_ARG
    assert b"multiple" in lib.last_error()
    odd = N.ModelCfg(2, 256, 4, 2, 96, 688, 1024, 1e-6, 1e4, N.F32)
    assert lib.kv_bytes_per_token(byref(odd)) == N.UNSUPPORTED
    # GQA groups of any size up to 16 query heads (a decode query's rows share
    # one 16-row tile): 5 and 16 are accepted, 17 is not.
    g5 = N.ModelCfg(2, 256, 10, 2, 128, 688, 1024, 1e-6, 1e4, N.F32)
    assert lib.kv_bytes_per_token(byref(g5)) == 2 * 2 * 2 * 128 * 4
    g16 = N.ModelCfg(2, 256, 16, 1, 64, 688, 1024, 1e-6, 1e4, N.F32)
    assert lib.kv_bytes_per_token(byref(g16)) == 2 * 2 * 1 * 64 * 4
    g17 = N.ModelCfg(2, 256, 17, 1, 64, 688, 1024, 1e-6, 1e4, N.F32)
    assert lib.kv_bytes_per_token(byref(g17)) == N.UNSUPPORTED
    assert b"at most 16" in lib.last_error()
    assert lib.paged_attention_workspace_bytes(64, 32, 8, 128, 0) > 0
    qk = N.ModelCfg(2, 256, 4, 2, 64, 688, 1024, 1e-6, 1e4, N.F32, 1)
    assert lib.kv_bytes_per_token(byref(qk)) == 2048
    qk.qk_norm = 2
    assert lib.kv_bytes_per_token(byref(qk)) == N.INVALID_ARG
    # packed weight sizes: bf16 pads N to whole 128-column groups, fp32 is row-major
    assert lib.packed_weight_bytes(N.BF16, 100, 128) == 128 * 128 * 2
    assert lib.packed_weight_bytes(N.BF16, 129, 64) == 256 * 64 * 2
    assert lib.packed_weight_bytes(N.BF16, 128256, 4096) == 128256 * 4096 * 2
    assert lib.packed_weight_bytes(N.F32, 100, 96) == 100 * 96 * 4
    assert lib.packed_weight_bytes(N.BF16, 100, 96) == N.UNSUPPORTED  # K % 64
    assert lib.packed_weight_bytes(N.BF16, 0, 64) == N.INVALID_ARG
    # SwiGLU projection scratch: none where the bf16 plan has no K split (the
    # fused epilogue), the split-K partials of gate|up otherwise
    assert lib.swiglu_projection_workspace_bytes(N.BF16, 256, 14336, 4096) == 0
    assert lib.swiglu_projection_workspace_bytes(N.BF16, 4, 256, 256) > 0
    assert lib.swiglu_projection_workspace_bytes(N.F32, 4, 688, 256) > 0
    assert lib.swiglu_projection_workspace_bytes(N.BF16, 0, 256, 256) == N.INVALID_ARG
    assert lib.sample_top_p_workspace_bytes(1) > 0
    assert lib.sample_top_p_workspace_bytes(32) > 0
    assert lib.sample_top_p_workspace_bytes(33) == 0
    assert lib.sample_top_p_workspace_bytes(0) == N.INVALID_ARG
