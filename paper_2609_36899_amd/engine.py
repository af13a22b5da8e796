"""Thin torch-facing binding of the C ABI (argument marshalling only).

Torch supplies device memory and the current stream; every step of the
decoder runs in the library's HIP kernels.  Function and method names follow
the C ABI: kv_alloc, kv_append_prefix, decode_step, sample, kv_free,
kv_len, kv_headroom, paged_decode_attention.
"""

from __future__ import annotations

import ctypes
from ctypes import POINTER, byref, c_int32, c_int64, c_void_p
from typing import Dict, Optional, Sequence

import numpy as np
import torch

from . import _native as N
from ._native import PAGE_TOKENS, PdecError

_TORCH_DTYPE = {N.F32: torch.float32, N.BF16: torch.bfloat16}


def _stream_handle(stream: Optional[torch.cuda.Stream]) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def model_cfg(shape, dtype: int, kv_fp8: Optional[Sequence[float]] = None) -> N.ModelCfg:
    """C struct for a shape object exposing the ModelCfg field names.

    ``kv_fp8=(k_scale, v_scale)`` stores the KV pages as E4M3 codes."""
    ks, vs = (float(kv_fp8[0]), float(kv_fp8[1])) if kv_fp8 is not None else (1.0, 1.0)
    return N.ModelCfg(shape.n_layers, shape.d_model, shape.n_q_heads, shape.n_kv_heads,
                      shape.head_dim, shape.ffn_dim, shape.vocab, float(shape.rms_eps),
                      float(shape.rope_base), dtype, int(bool(getattr(shape, "qk_norm", False))),
                      int(kv_fp8 is not None), ks, vs)


def kv_bytes_per_token(shape, dtype: int, kv_fp8: Optional[Sequence[float]] = None) -> int:
    cfg = model_cfg(shape, dtype, kv_fp8)
    return N.check(N.load().kv_bytes_per_token(byref(cfg)))


class PackedWeight:
    """A projection matrix [n][k] in the layout pack_weight produces."""

    def __init__(self, data: torch.Tensor, n: int, k: int, dtype: int):
        self.data, self.n, self.k, self.dtype = data, n, k, dtype

    @property
    def shape(self):
        return (self.n, self.k)

    def data_ptr(self) -> int:
        return self.data.data_ptr()


def pack_weight(w: torch.Tensor, stream: Optional[torch.cuda.Stream] = None) -> PackedWeight:
    """Pack a device row-major [n][k] matrix (bf16 or fp32) with pack_weight."""
    assert w.dim() == 2 and w.is_cuda and w.is_contiguous()
    assert w.dtype in (torch.bfloat16, torch.float32)
    dtype = N.BF16 if w.dtype == torch.bfloat16 else N.F32
    n, k = w.shape
    lib = N.load()
    nbytes = N.check(lib.packed_weight_bytes(dtype, n, k))
    data = torch.empty(nbytes // w.element_size(), dtype=w.dtype, device=w.device)
    N.check(lib.pack_weight(dtype, n, k, w.data_ptr(), data.data_ptr(), _stream_handle(stream)))
    return PackedWeight(data, n, k, dtype)


PROJECTIONS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")


def weights_to_device(arrays: Dict, dtype: int, device="cuda") -> Dict:
    """Copy a weight dict (numpy, nn.Linear layout) to the device.

    Matrices go to the storage dtype (bf16 inputs must already be
    bf16-representable, so the cast is exact) and the projections are packed
    with pack_weight; norm gains stay fp32.
    """
    td = _TORCH_DTYPE[dtype]
    mat = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(
        device=device).to(td).contiguous()
    vec = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)
    out = {"embed": mat(arrays["embed"]), "lm_head": pack_weight(mat(arrays["lm_head"])),
           "final_norm": vec(arrays["final_norm"]), "layers": []}
    for lay in arrays["layers"]:
        d = {k: pack_weight(mat(lay[k])) for k in PROJECTIONS}
        for k in ("attn_norm", "ffn_norm", "q_norm", "k_norm"):
            if k in lay:
                d[k] = vec(lay[k])
        out["layers"].append(d)
    return out


class Engine:
    """One rollout worker's decode backend over caller-owned device memory."""

    def __init__(self, shape, weights: Dict, dtype: int, kv_pool_bytes: int, max_seqs: int,
                 max_seq_len: int, max_batch: int, max_chunk: int, device="cuda",
                 stream: Optional[torch.cuda.Stream] = None,
                 kv_fp8: Optional[Sequence[float]] = None):
        self.lib = N.load()
        self.shape = shape
        self.dtype = dtype
        self.kv_fp8 = kv_fp8
        self.cfg = model_cfg(shape, dtype, kv_fp8)
        self.weights = weights  # keep the tensors alive
        self.kv_token_bytes = N.check(self.lib.kv_bytes_per_token(byref(self.cfg)))
        page_bytes = self.kv_token_bytes * PAGE_TOKENS
        self.n_pages = int(kv_pool_bytes // page_bytes)
        self.kv_pool = torch.empty(self.n_pages * page_bytes, dtype=torch.uint8, device=device)
        ws = N.check(self.lib.engine_workspace_bytes(byref(self.cfg), max_seqs, max_seq_len,
                                                     max_batch, max_chunk,
                                                     self.kv_pool.numel()))
        self.workspace = torch.empty(ws, dtype=torch.uint8, device=device)
        L = shape.n_layers

        def arr(key):
            a = (c_void_p * L)(*[weights["layers"][i][key].data_ptr() for i in range(L)])
            return ctypes.cast(a, POINTER(c_void_p)), a

        self._keep = []
        fields = {}
        keys = ["attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down"]
        if self.cfg.qk_norm:
            keys += ["q_norm", "k_norm"]
        for key in keys:
            p, a = arr(key)
            self._keep.append(a)
            fields[key] = p
        self.cw = N.Weights(embed=weights["embed"].data_ptr(),
                            lm_head=weights["lm_head"].data_ptr(),
                            final_norm=weights["final_norm"].data_ptr(), **fields)
        h = c_void_p()
        N.check(self.lib.engine_create(byref(self.cfg), byref(self.cw), self.kv_pool.data_ptr(),
                                       self.kv_pool.numel(), max_seqs, max_seq_len, max_batch,
                                       max_chunk, self.workspace.data_ptr(),
                                       self.workspace.numel(), _stream_handle(stream), byref(h)))
        self.handle = h
        self.max_batch, self.max_chunk = max_batch, max_chunk

    def close(self):
        if getattr(self, "handle", None):
            self.lib.engine_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---- pool views (layout [layer][K|V][page][Hkv][16 * Dh]) -------------
    def _pool_view(self):
        s = self.shape
        t = self.kv_pool if self.kv_fp8 is not None else self.kv_pool.view(_TORCH_DTYPE[self.dtype])
        return t.view(s.n_layers, 2, self.n_pages, s.n_kv_heads, PAGE_TOKENS * s.head_dim)

    def k_pages(self, layer: int) -> torch.Tensor:
        """[pages][Hkv][16][Dh] view of one layer's K pages."""
        s = self.shape
        return self._pool_view()[layer, 0].view(self.n_pages, s.n_kv_heads, PAGE_TOKENS,
                                                s.head_dim)

    def v_pages(self, layer: int) -> torch.Tensor:
        """[pages][Hkv][Dh][16] view of one layer's V pages (transposed per page)."""
        s = self.shape
        return self._pool_view()[layer, 1].view(self.n_pages, s.n_kv_heads, s.head_dim,
                                                PAGE_TOKENS)

    def profile(self, kinds: Sequence[int] = (), every: int = 1) -> None:
        """Time the launches of the given timer classes (N.TIMER_*), one in
        every `every` of each; an empty sequence turns timing off (see
        engine_profile, engine_profile_every)."""
        mask = 0
        for k in kinds:
            mask |= 1 << int(k)
        N.check(self.lib.engine_profile_every(self.handle, int(every)))
        N.check(self.lib.engine_profile(self.handle, mask))

    def profile_read(self, kind: int):
        """(total ms, launch count) of one timed class since the last read."""
        ms, n = ctypes.c_double(), c_int64()
        N.check(self.lib.engine_profile_read(self.handle, int(kind), byref(ms), byref(n)))
        return ms.value, n.value

    def set_stream(self, stream: Optional[torch.cuda.Stream] = None):
        N.check(self.lib.engine_set_stream(self.handle, _stream_handle(stream)))

    # ---- resident set --------------------------------------------------------
    def kv_alloc(self, reserve_tokens: int = 0) -> int:
        out = c_int32()
        N.check(self.lib.kv_alloc(self.handle, int(reserve_tokens), byref(out)))
        return out.value

    def kv_free(self, seq: int) -> None:
        N.check(self.lib.kv_free(self.handle, int(seq)))

    def kv_len(self, seq: int) -> int:
        out = c_int32()
        N.check(self.lib.kv_len(self.handle, int(seq), byref(out)))
        return out.value

    def kv_headroom(self) -> int:
        out = c_int64()
        N.check(self.lib.kv_headroom(self.handle, byref(out)))
        return out.value

    def kv_block_table(self, seq: int) -> np.ndarray:
        n = c_int32()
        cap = self.n_pages
        buf = (c_int32 * max(cap, 1))()
        N.check(self.lib.kv_block_table(self.handle, int(seq), buf, cap, byref(n)))
        return np.frombuffer(buf, dtype=np.int32, count=n.value).copy()

    def kv_extend_uninit(self, seq: int, n_tokens: int) -> None:
        N.check(self.lib.kv_extend_uninit(self.handle, int(seq), int(n_tokens)))

    # ---- compute -------------------------------------------------------------
    def kv_append_prefix(self, seq: int, tokens: Sequence[int], chunk_tokens: int,
                         last_logits: Optional[torch.Tensor] = None) -> None:
        tok = np.ascontiguousarray(np.asarray(tokens, dtype=np.int32))
        if last_logits is not None:
            assert last_logits.is_cuda and last_logits.dtype == torch.float32
            assert last_logits.numel() >= self.shape.vocab and last_logits.is_contiguous()
        N.check(self.lib.kv_append_prefix(self.handle, int(seq),
                                          tok.ctypes.data_as(POINTER(c_int32)), len(tok),
                                          int(chunk_tokens), _ptr(last_logits)))

    def kv_append_prefix_batch(self, seq_ids: Sequence[int], tokens: Sequence[Sequence[int]],
                               chunk_tokens: int,
                               last_logits: Optional[torch.Tensor] = None) -> None:
        """Append tokens[i] to seq_ids[i] for every i in one call (packed passes)."""
        ids = np.ascontiguousarray(np.asarray(seq_ids, dtype=np.int32))
        parts = [np.asarray(t, dtype=np.int32).ravel() for t in tokens]
        assert len(parts) == len(ids)
        counts = np.ascontiguousarray(np.array([len(t) for t in parts], dtype=np.int32))
        flat = np.ascontiguousarray(np.concatenate(parts) if parts else np.zeros(0, np.int32))
        if last_logits is not None:
            assert last_logits.is_cuda and last_logits.dtype == torch.float32
            assert last_logits.numel() >= len(ids) * self.shape.vocab
            assert last_logits.is_contiguous()
        N.check(self.lib.kv_append_prefix_batch(
            self.handle, len(ids), ids.ctypes.data_as(POINTER(c_int32)),
            counts.ctypes.data_as(POINTER(c_int32)), flat.ctypes.data_as(POINTER(c_int32)),
            int(chunk_tokens), _ptr(last_logits)))

    def decode_step(self, seq_ids: Sequence[int], tokens: torch.Tensor,
                    logits: torch.Tensor) -> None:
        ids = np.ascontiguousarray(np.asarray(seq_ids, dtype=np.int32))
        B = len(ids)
        assert tokens.is_cuda and tokens.dtype == torch.int32 and tokens.numel() >= B
        assert logits.is_cuda and logits.dtype == torch.float32 and logits.is_contiguous()
        assert logits.numel() >= B * self.shape.vocab and tokens.is_contiguous()
        N.check(self.lib.decode_step(self.handle, B, ids.ctypes.data_as(POINTER(c_int32)),
                                     tokens.data_ptr(), logits.data_ptr()))

    def kv_snapshot_bytes(self, n_tokens: int) -> int:
        """Host bytes kv_export needs for a sequence of n_tokens tokens."""
        return -(-int(n_tokens) // PAGE_TOKENS) * PAGE_TOKENS * self.kv_token_bytes

    def kv_export(self, seq: int, host_dst: torch.Tensor) -> int:
        """Snapshot a sequence's KV into a pinned host tensor; returns its length.

        The copy is asynchronous on the engine's stream: synchronise before
        reading host_dst."""
        assert host_dst.device.type == "cpu" and host_dst.is_pinned() and host_dst.is_contiguous()
        n = c_int32()
        N.check(self.lib.kv_export(self.handle, int(seq), host_dst.data_ptr(),
                                   host_dst.numel() * host_dst.element_size(), byref(n)))
        return n.value

    def kv_import(self, seq: int, host_src: torch.Tensor, n_tokens: int) -> None:
        """Restore a kv_export snapshot into an empty sequence."""
        assert host_src.device.type == "cpu" and host_src.is_pinned() and host_src.is_contiguous()
        N.check(self.lib.kv_import(self.handle, int(seq), host_src.data_ptr(),
                                   host_src.numel() * host_src.element_size(), int(n_tokens)))

    def sample(self, logits: torch.Tensor, tokens_out: torch.Tensor, mode: int = 0,
               batch: Optional[int] = None) -> None:
        B = batch if batch is not None else logits.shape[0]
        assert logits.is_cuda and logits.dtype == torch.float32 and logits.is_contiguous()
        assert tokens_out.is_cuda and tokens_out.dtype == torch.int32
        assert tokens_out.numel() >= B and logits.numel() >= B * self.shape.vocab
        N.check(self.lib.sample(self.handle, int(B), logits.data_ptr(), tokens_out.data_ptr(),
                                int(mode)))


def swiglu_projection_workspace_bytes(dtype: int, rows: int, ffn: int, k: int) -> int:
    """Scratch bytes swiglu_projection needs (0 when the SwiGLU is fused)."""
    return N.check(N.load().swiglu_projection_workspace_bytes(dtype, rows, ffn, k))


def swiglu_projection(x: torch.Tensor, w_gate: PackedWeight, w_up: PackedWeight,
                      u: torch.Tensor, workspace: Optional[torch.Tensor] = None,
                      stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """u = silu(x Wg^T) * (x Wu^T) through the library's kernels; see include/pdec.h."""
    rows, k = x.shape
    ffn = w_gate.n
    assert isinstance(w_gate, PackedWeight) and isinstance(w_up, PackedWeight)
    assert w_up.n == ffn and w_gate.k == k and w_up.k == k and x.is_contiguous()
    assert w_gate.dtype == w_up.dtype and x.dtype == _TORCH_DTYPE[w_gate.dtype]
    assert u.dtype == x.dtype and tuple(u.shape) == (rows, ffn) and u.is_contiguous()
    lib = N.load()
    need = N.check(lib.swiglu_projection_workspace_bytes(w_gate.dtype, rows, ffn, k))
    if need and (workspace is None or workspace.numel() < need):
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
    N.check(lib.swiglu_projection(w_gate.dtype, rows, ffn, k, x.data_ptr(), w_gate.data_ptr(),
                                  w_up.data_ptr(), u.data_ptr(),
                                  workspace.data_ptr() if need else None,
                                  workspace.numel() if need else 0, _stream_handle(stream)))
    return u


def weight_projection_workspace_bytes(dtype: int, rows: int, cols: int, k: int) -> int:
    """Scratch bytes weight_projection needs for split-K partials (0 if none)."""
    return N.check(N.load().weight_projection_workspace_bytes(dtype, rows, cols, k))


def weight_projection(x: torch.Tensor, w: PackedWeight, out: torch.Tensor,
                      workspace: Optional[torch.Tensor] = None,
                      stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """out = x W^T through the library's projection kernels; see include/pdec.h."""
    rows, k = x.shape
    cols = w.n
    assert isinstance(w, PackedWeight) and k == w.k and x.is_contiguous()
    assert out.dtype == torch.float32 and tuple(out.shape) == (rows, cols)
    assert out.is_contiguous()
    assert x.dtype == _TORCH_DTYPE[w.dtype]
    lib = N.load()
    need = N.check(lib.weight_projection_workspace_bytes(w.dtype, rows, cols, k))
    if need and (workspace is None or workspace.numel() < need):
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
    N.check(lib.weight_projection(w.dtype, rows, cols, k, x.data_ptr(), w.data_ptr(),
                                  out.data_ptr(), workspace.data_ptr() if need else None,
                                  workspace.numel() if need else 0, _stream_handle(stream)))
    return out


def sample_top_p_workspace_bytes(batch: int) -> int:
    """Scratch bytes for the split form of sample_top_p (0: one group per row)."""
    return N.check(N.load().sample_top_p_workspace_bytes(batch))


def sample_top_p(logits: torch.Tensor, tokens_out: torch.Tensor, temperature: float,
                 top_p: float, uniforms: torch.Tensor,
                 workspace: Optional[torch.Tensor] = None, split: bool = True,
                 stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """Temperature / top-p sampling of each row of logits [B, V] with the
    given uniforms [B] (see sample_top_p in include/pdec.h).  split=False
    passes no workspace (one work group per row)."""
    assert logits.dim() == 2 and logits.dtype == torch.float32 and logits.is_contiguous()
    B, V = logits.shape
    assert uniforms.dtype == torch.float32 and uniforms.numel() >= B and uniforms.is_cuda
    assert tokens_out.dtype == torch.int32 and tokens_out.numel() >= B
    lib = N.load()
    need = N.check(lib.sample_top_p_workspace_bytes(B)) if split else 0
    if need and (workspace is None or workspace.numel() < need):
        workspace = torch.empty(need, dtype=torch.uint8, device=logits.device)
    N.check(lib.sample_top_p(B, V, logits.data_ptr(), float(temperature), float(top_p),
                             uniforms.data_ptr(), tokens_out.data_ptr(),
                             workspace.data_ptr() if need else None,
                             workspace.numel() if need else 0, _stream_handle(stream)))
    return tokens_out


def paged_attention_workspace_bytes(batch: int, n_q_heads: int, n_kv_heads: int,
                                    head_dim: int) -> int:
    return N.check(N.load().paged_attention_workspace_bytes(batch, n_q_heads, n_kv_heads,
                                                            head_dim, 0))


def paged_decode_attention_fp8(q: torch.Tensor, k_pages: torch.Tensor, v_pages: torch.Tensor,
                               k_scale: float, v_scale: float, block_table: torch.Tensor,
                               lens: Sequence[int], out: torch.Tensor,
                               workspace: Optional[torch.Tensor] = None,
                               stream: Optional[torch.cuda.Stream] = None) -> torch.Tensor:
    """Isolated paged decode attention over E4M3 code pages (uint8
    [P][Hkv][16][Dh] and [P][Hkv][Dh][16]) with bf16 q; see include/pdec.h."""
    B, Hq, Dh = q.shape
    P, Hkv, page, Dh2 = k_pages.shape
    assert page == PAGE_TOKENS and Dh2 == Dh and tuple(v_pages.shape) == (P, Hkv, Dh, PAGE_TOKENS)
    assert q.dtype == torch.bfloat16 and k_pages.dtype == v_pages.dtype == torch.uint8
    assert q.is_contiguous() and k_pages.is_contiguous() and v_pages.is_contiguous()
    assert block_table.dtype == torch.int32 and block_table.dim() == 2
    assert block_table.shape[0] == B and block_table.is_contiguous()
    assert out.dtype == torch.float32 and tuple(out.shape) == (B, Hq, Dh) and out.is_contiguous()
    ln = np.ascontiguousarray(np.asarray(lens, dtype=np.int32))
    assert ln.shape == (B,) and (ln >= 1).all() and (ln <= block_table.shape[1] * PAGE_TOKENS).all()
    bt = block_table.cpu().numpy()
    for b in range(B):
        used = bt[b, :(int(ln[b]) + PAGE_TOKENS - 1) // PAGE_TOKENS]
        if used.size and (used.min() < 0 or used.max() >= P):
            raise PdecError(N.INVALID_ARG, f"block table row {b} names a page outside the pool")
    need = paged_attention_workspace_bytes(B, Hq, Hkv, Dh)
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    N.check(N.load().paged_decode_attention_fp8(
        B, Hq, Hkv, Dh, q.data_ptr(), k_pages.data_ptr(), v_pages.data_ptr(), float(k_scale),
        float(v_scale), block_table.data_ptr(), block_table.shape[1],
        ln.ctypes.data_as(POINTER(c_int32)), out.data_ptr(), workspace.data_ptr(),
        workspace.numel(), _stream_handle(stream)))
    return out


def paged_decode_attention(q: torch.Tensor, k_pages: torch.Tensor, v_pages: torch.Tensor,
                           block_table: torch.Tensor, lens: Sequence[int], out: torch.Tensor,
                           workspace: Optional[torch.Tensor] = None,
                           stream: Optional[torch.cuda.Stream] = None,
                           check_pages: bool = True) -> torch.Tensor:
    """Isolated paged decode attention; see include/pdec.h.

    q [B][Hq][Dh] (bf16 or fp32), k_pages [P][Hkv][16][Dh], v_pages
    [P][Hkv][Dh][16], block_table int32 [B][stride] on the device, lens on
    the host, out fp32 [B][Hq][Dh].  With ``check_pages`` the page ids the
    kernel will read are checked against the pool size first (one copy of the
    block table to the host).
    """
    B, Hq, Dh = q.shape
    P, Hkv, page, Dh2 = k_pages.shape
    assert page == PAGE_TOKENS and Dh2 == Dh and tuple(v_pages.shape) == (P, Hkv, Dh, PAGE_TOKENS)
    assert q.dtype == k_pages.dtype == v_pages.dtype
    assert q.is_contiguous() and k_pages.is_contiguous() and v_pages.is_contiguous()
    assert block_table.dtype == torch.int32 and block_table.dim() == 2
    assert block_table.shape[0] == B and block_table.is_contiguous()
    assert out.dtype == torch.float32 and tuple(out.shape) == (B, Hq, Dh) and out.is_contiguous()
    dtype = N.BF16 if q.dtype == torch.bfloat16 else N.F32
    assert dtype == N.BF16 or q.dtype == torch.float32
    ln = np.ascontiguousarray(np.asarray(lens, dtype=np.int32))
    assert ln.shape == (B,) and (ln >= 1).all() and (ln <= block_table.shape[1] * PAGE_TOKENS).all()
    if check_pages:
        bt = block_table.cpu().numpy()
        for b in range(B):
            used = bt[b, :(int(ln[b]) + PAGE_TOKENS - 1) // PAGE_TOKENS]
            if used.size and (used.min() < 0 or used.max() >= P):
                raise PdecError(N.INVALID_ARG, f"block table row {b} names a page outside the pool")
    need = paged_attention_workspace_bytes(B, Hq, Hkv, Dh)
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    N.check(N.load().paged_decode_attention(
        dtype, B, Hq, Hkv, Dh, q.data_ptr(), k_pages.data_ptr(), v_pages.data_ptr(),
        block_table.data_ptr(), block_table.shape[1], ln.ctypes.data_as(POINTER(c_int32)),
        out.data_ptr(), workspace.data_ptr(), workspace.numel(), _stream_handle(stream)))
    return out
