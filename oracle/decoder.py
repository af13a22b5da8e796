"""Plain decoder oracle: one trajectory at a time, contiguous KV, float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What it computes, for one trajectory with t the input token at position p
(p = number of tokens already cached, positions 0-indexed):

  x = E[t]
  per layer:
    h  = rmsnorm(x) * g1
    q, k, v = Wq h, Wk h, Wv h            reshaped to (Hq,Dh), (Hkv,Dh), (Hkv,Dh)
    [q/k-norm variant: q = rmsnorm(q) * gq, k = rmsnorm(k) * gk per head,
     over Dh, when the layer carries q_norm / k_norm gains]
    q, k = rope(q, p), rope(k, p)         rotate-half pairs (i, i + Dh/2),
                                          angle p * base^(-2i/Dh)
    append k, v to the trajectory's cache (the rotated k is cached)
    o_h = softmax(q_h . K_g^T / sqrt(Dh)) V_g   over positions 0..p,
                                          g = floor(h / (Hq/Hkv))
    x  = x + Wo concat(o)
    h2 = rmsnorm(x) * g2
    x  = x + Wd (silu(Wg h2) * (Wu h2)),  silu(z) = z / (1 + e^-z)
  logits = Wlm (rmsnorm(x) * gf);  greedy token = argmax, ties to the lowest id.

Readings of points the paper leaves open (it names dense Qwen3 models run by
its inference backend, Evaluation: experimental setup, and gives no layer
definition):
  * Llama-style pre-norm block, no biases, untied LM head and a final RMSNorm.
    The per-head q/k RMSNorm of the Qwen3 family (its public model
    definition, not the paper) is an option: a layer with ``q_norm`` and
    ``k_norm`` gains normalises each q and k head over Dh before RoPE.
  * RoPE in the rotate-half pairing with base 10000.
  * Contiguous GQA groups: query head h reads KV head floor(h*Hkv/Hq).
  * Attention is causal and includes the current token; scale 1/sqrt(Dh);
    no soft-cap, window or ALiBi.
  * A prefix occupies positions 0..n-1, and the first decode step after it is
    at position n.
  * fp8 KV variant (``kv_fp8=(k_scale, v_scale)``): the cache holds k and v as
    e4m3 codes (oracle/fp8.py), so attention reads value(code) * scale for
    every cached position, the current one included.
"""

from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence, Tuple

import numpy as np

from .fp8 import quantize_dequantize


@dataclasses.dataclass
class ModelWeights:
    """Decoder weights in the nn.Linear ``[out, in]`` layout, held as one dtype."""

    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    rms_eps: float
    rope_base: float
    embed: np.ndarray
    lm_head: np.ndarray
    final_norm: np.ndarray
    layers: List[dict]

    @classmethod
    def from_arrays(cls, shape, arrays: dict, dtype=np.float64) -> "ModelWeights":
        cast = lambda a: np.asarray(a, dtype=dtype)
        layers = [{k: cast(v) for k, v in lay.items()} for lay in arrays["layers"]]
        return cls(n_layers=shape.n_layers, n_q_heads=shape.n_q_heads,
                   n_kv_heads=shape.n_kv_heads, head_dim=shape.head_dim,
                   rms_eps=shape.rms_eps, rope_base=shape.rope_base,
                   embed=cast(arrays["embed"]), lm_head=cast(arrays["lm_head"]),
                   final_norm=cast(arrays["final_norm"]), layers=layers)


def rmsnorm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * gain over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gain


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def rope(z: np.ndarray, positions, base: float) -> np.ndarray:
    """Rotate-half rotary embedding.

    ``z`` has shape ``[..., n_heads, Dh]`` with the leading axes matching
    ``positions`` (a scalar or an array broadcast over the heads).  The pair
    (z_i, z_{i+Dh/2}) is rotated by the angle pos * base^(-2i/Dh).
    """
    dh = z.shape[-1]
    half = dh // 2
    i = np.arange(half, dtype=np.float64)
    theta = base ** (-2.0 * i / dh)
    pos = np.asarray(positions, dtype=np.float64)
    ang = pos[..., None, None] * theta  # broadcast over heads
    c, s = np.cos(ang).astype(z.dtype), np.sin(ang).astype(z.dtype)
    a, b = z[..., :half], z[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def attention(q: np.ndarray, keys: np.ndarray, values: np.ndarray) -> np.ndarray:
    """Decode attention of one query position over T cached positions.

    q: [Hq, Dh]; keys, values: [T, Hkv, Dh].  Returns [Hq, Dh].  Softmax is
    the two-pass max-subtracted form.
    """
    hq, dh = q.shape
    hkv = keys.shape[1]
    group = hq // hkv
    out = np.empty_like(q)
    scale = 1.0 / np.sqrt(dh)
    for h in range(hq):
        g = h // group
        s = keys[:, g, :] @ q[h] * scale
        a = np.exp(s - s.max())
        a = a / a.sum()
        out[h] = a @ values[:, g, :]
    return out


def greedy(logits: np.ndarray) -> np.ndarray:
    """Argmax over the last axis; numpy returns the first (lowest) index on ties."""
    if np.isnan(logits).any():
        raise ValueError("NaN logits")
    return np.argmax(logits, axis=-1)


class Decoder:
    """Incremental decoder with a contiguous per-trajectory KV cache."""

    def __init__(self, weights: ModelWeights, kv_fp8: Optional[Tuple[float, float]] = None):
        self.w = weights
        self.kv_fp8 = kv_fp8

    def new_state(self) -> dict:
        w = self.w
        return {"k": [np.zeros((0, w.n_kv_heads, w.head_dim), dtype=w.embed.dtype)
                      for _ in range(w.n_layers)],
                "v": [np.zeros((0, w.n_kv_heads, w.head_dim), dtype=w.embed.dtype)
                      for _ in range(w.n_layers)],
                "len": 0}

    def step(self, state: dict, token: int) -> np.ndarray:
        """Consume one token at position state['len'] and return its logits."""
        w = self.w
        p = state["len"]
        x = w.embed[int(token)].copy()
        for li, lay in enumerate(w.layers):
            h = rmsnorm(x, lay["attn_norm"], w.rms_eps)
            q = (lay["wq"] @ h).reshape(w.n_q_heads, w.head_dim)
            k = (lay["wk"] @ h).reshape(w.n_kv_heads, w.head_dim)
            v = (lay["wv"] @ h).reshape(w.n_kv_heads, w.head_dim)
            if "q_norm" in lay:
                q = rmsnorm(q, lay["q_norm"], w.rms_eps)
                k = rmsnorm(k, lay["k_norm"], w.rms_eps)
            q = rope(q, p, w.rope_base)
            k = rope(k, p, w.rope_base)
            if self.kv_fp8 is not None:
                k = quantize_dequantize(k, self.kv_fp8[0])
                v = quantize_dequantize(v, self.kv_fp8[1])
            state["k"][li] = np.concatenate([state["k"][li], k[None]], axis=0)
            state["v"][li] = np.concatenate([state["v"][li], v[None]], axis=0)
            o = attention(q, state["k"][li], state["v"][li])
            x = x + lay["wo"] @ o.reshape(-1)
            h2 = rmsnorm(x, lay["ffn_norm"], w.rms_eps)
            x = x + lay["w_down"] @ (silu(lay["w_gate"] @ h2) * (lay["w_up"] @ h2))
        state["len"] = p + 1
        return w.lm_head @ rmsnorm(x, w.final_norm, w.rms_eps)

    def prefill(self, state: dict, tokens: Sequence[int]) -> Optional[np.ndarray]:
        """Consume a prefix token by token; return the last position's logits."""
        logits = None
        for t in tokens:
            logits = self.step(state, t)
        return logits


def recompute_logits(weights: ModelWeights, tokens: Sequence[int],
                     kv_fp8: Optional[Tuple[float, float]] = None) -> np.ndarray:
    """Logits at every position of ``tokens``, recomputed without any KV cache.

    Full causal attention over the whole sequence with dense matrices; this is
    the definition the cached decoder must reproduce.
    """
    w = weights
    n = len(tokens)
    pos = np.arange(n)
    x = w.embed[np.asarray(tokens, dtype=np.int64)].copy()
    group = w.n_q_heads // w.n_kv_heads
    mask = np.tril(np.ones((n, n), dtype=bool))
    for lay in w.layers:
        h = rmsnorm(x, lay["attn_norm"], w.rms_eps)
        q = (h @ lay["wq"].T).reshape(n, w.n_q_heads, w.head_dim)
        k = (h @ lay["wk"].T).reshape(n, w.n_kv_heads, w.head_dim)
        v = (h @ lay["wv"].T).reshape(n, w.n_kv_heads, w.head_dim)
        if "q_norm" in lay:
            q = rmsnorm(q, lay["q_norm"], w.rms_eps)
            k = rmsnorm(k, lay["k_norm"], w.rms_eps)
        q = rope(q, pos, w.rope_base)
        k = rope(k, pos, w.rope_base)
        if kv_fp8 is not None:
            k = quantize_dequantize(k, kv_fp8[0])
            v = quantize_dequantize(v, kv_fp8[1])
        o = np.empty_like(q)
        for hh in range(w.n_q_heads):
            g = hh // group
            s = (q[:, hh, :] @ k[:, g, :].T) / np.sqrt(w.head_dim)
            s = np.where(mask, s, -np.inf)
            a = np.exp(s - s.max(axis=1, keepdims=True))
            a = a / a.sum(axis=1, keepdims=True)
            o[:, hh, :] = a @ v[:, g, :]
        x = x + o.reshape(n, -1) @ lay["wo"].T
        h2 = rmsnorm(x, lay["ffn_norm"], w.rms_eps)
        x = x + (silu(h2 @ lay["w_gate"].T) * (h2 @ lay["w_up"].T)) @ lay["w_down"].T
    return rmsnorm(x, w.final_norm, w.rms_eps) @ w.lm_head.T
