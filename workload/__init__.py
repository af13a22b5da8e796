"""Seeded synthetic inputs shared by the CPU oracle's tests and the GPU path.

This module only draws random numbers and lays them out: model shapes,
weights, token ids, context lengths, paged-pool block tables and raw
attention operands.  It contains none of the decoder's arithmetic, so both
sides of a parity test can take their inputs from here without sharing any
part of the computation under test.

The workloads stand in for the paper's RL rollout traces (its Evaluation
section, experimental setup), which are not available: long-horizon decode
over a batch whose context lengths differ by orders of magnitude
(Background, workload evolution).  Every generator is a pure function of its
seed, drawn with numpy's PCG64 ``default_rng``.
"""

from __future__ import annotations

import dataclasses
from typing import Dict, List

import numpy as np

PAGE_TOKENS = 16


@dataclasses.dataclass(frozen=True)
class ModelShape:
    """Shape of a Llama-style pre-norm decoder (RMSNorm, RoPE, GQA, SwiGLU)."""

    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rms_eps: float = 1e-6
    rope_base: float = 10000.0
    # Qwen3-style per-head RMSNorm of q and k (over head_dim) before RoPE.
    qk_norm: bool = False

    @property
    def q_dim(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim


# The 2-layer fp32 decoder used for end-to-end parity.
TINY = ModelShape(n_layers=2, d_model=256, n_q_heads=4, n_kv_heads=2, head_dim=64,
                  ffn_dim=688, vocab=1024)
# The 8B-shaped decoder (Llama-3-8B-like shape) used for throughput work.
EIGHT_B = ModelShape(n_layers=32, d_model=4096, n_q_heads=32, n_kv_heads=8, head_dim=128,
                     ffn_dim=14336, vocab=128256)
# A small bf16 decoder with the 8B model's head geometry (head_dim 128, GQA 4),
# small enough for a float64 oracle to run in seconds.
SMALL_BF16 = ModelShape(n_layers=2, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=128,
                        ffn_dim=1408, vocab=2048)
# The same two with Qwen3-style q/k norm.
TINY_QK = dataclasses.replace(TINY, qk_norm=True)
SMALL_BF16_QK = dataclasses.replace(SMALL_BF16, qk_norm=True)
# Decoders with the dimensions of the paper's larger rollout models (Qwen3-14B
# and Qwen3-32B, as their public configurations give them; the paper states no
# hyperparameters): per-head q/k norm, RoPE base 1e6, untied LM head.  Random
# init like the others; used for throughput at those widths and depths.
QWEN3_14B_SHAPED = ModelShape(n_layers=40, d_model=5120, n_q_heads=40, n_kv_heads=8,
                              head_dim=128, ffn_dim=17408, vocab=151936, rope_base=1e6,
                              qk_norm=True)
QWEN3_32B_SHAPED = ModelShape(n_layers=64, d_model=5120, n_q_heads=64, n_kv_heads=8,
                              head_dim=128, ffn_dim=25600, vocab=151936, rope_base=1e6,
                              qk_norm=True)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); float32 result."""
    a = np.ascontiguousarray(x, dtype=np.float32)
    bits = a.view(np.uint32).astype(np.uint64)
    rounded = ((bits + 0x7FFF + ((bits >> 16) & 1)) >> 16) << 16
    return rounded.astype(np.uint32).view(np.float32).reshape(a.shape)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """uint16 bit patterns of float32 values that are already bf16-representable."""
    a = np.ascontiguousarray(x, dtype=np.float32)
    return (a.view(np.uint32) >> 16).astype(np.uint16)


def layer_matrix_names() -> List[str]:
    return ["wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down"]


def make_weights(shape: ModelShape, seed: int = 0, bf16: bool = False,
                 std: float = 0.02) -> Dict[str, object]:
    """Seeded random weights in the nn.Linear ``[out, in]`` layout.

    Every matrix is drawn N(0, std) in the fixed order: embedding, then per
    layer q, k, v, o, gate, up, down, then the LM head.  Norm gains are 1.0,
    except that a shape with q/k norm then draws per-layer q and k gains
    1 + 0.1 N(0, 1) (so that the gains are exercised), after everything else.
    With ``bf16`` the float32 draws are rounded to bf16 (RNE); both sides
    then use exactly the same representable values.
    """
    rng = np.random.default_rng(seed)
    s = shape

    def draw(rows, cols):
        w = (rng.standard_normal((rows, cols), dtype=np.float32) * np.float32(std))
        return round_to_bf16(w) if bf16 else w

    weights: Dict[str, object] = {"embed": draw(s.vocab, s.d_model), "layers": []}
    for _ in range(s.n_layers):
        layer = {
            "wq": draw(s.q_dim, s.d_model),
            "wk": draw(s.kv_dim, s.d_model),
            "wv": draw(s.kv_dim, s.d_model),
            "wo": draw(s.d_model, s.q_dim),
            "w_gate": draw(s.ffn_dim, s.d_model),
            "w_up": draw(s.ffn_dim, s.d_model),
            "w_down": draw(s.d_model, s.ffn_dim),
            "attn_norm": np.ones(s.d_model, dtype=np.float32),
            "ffn_norm": np.ones(s.d_model, dtype=np.float32),
        }
        weights["layers"].append(layer)
    weights["lm_head"] = draw(s.vocab, s.d_model)
    weights["final_norm"] = np.ones(s.d_model, dtype=np.float32)
    if s.qk_norm:
        for layer in weights["layers"]:
            for name in ("q_norm", "k_norm"):
                layer[name] = (1.0 + 0.1 * rng.standard_normal(s.head_dim)).astype(np.float32)
    return weights


def make_weights_parallel(shape: ModelShape, seed: int = 0, bf16: bool = True,
                          std: float = 0.02, threads: int = 16,
                          chunk: int = 1 << 25) -> Dict[str, object]:
    """The same layout and distributions as make_weights, drawn in parallel for
    full-size models: every matrix is cut into chunks of ``chunk`` elements in
    the fixed order of make_weights, and chunk i is filled by its own PCG64
    stream ``SeedSequence(seed).spawn(...)[i]`` (N(0, std), float32, then bf16
    RNE with ``bf16``) on a thread pool.  The values differ from
    make_weights' (another stream layout) and do not depend on ``threads``.
    A shape with q/k norm also gets per-layer q and k gains 1 + 0.1 N(0, 1),
    drawn from one further stream."""
    import concurrent.futures as cf
    s = shape
    dims = [("embed", s.vocab, s.d_model)]
    for l in range(s.n_layers):
        dims += [((l, "wq"), s.q_dim, s.d_model), ((l, "wk"), s.kv_dim, s.d_model),
                 ((l, "wv"), s.kv_dim, s.d_model), ((l, "wo"), s.d_model, s.q_dim),
                 ((l, "w_gate"), s.ffn_dim, s.d_model), ((l, "w_up"), s.ffn_dim, s.d_model),
                 ((l, "w_down"), s.d_model, s.ffn_dim)]
    dims.append(("lm_head", s.vocab, s.d_model))
    mats = {key: np.empty((r, c), dtype=np.float32) for key, r, c in dims}
    jobs = []
    for key, r, c in dims:
        flat = mats[key].reshape(-1)
        for o in range(0, flat.size, chunk):
            jobs.append(flat[o:o + chunk])
    streams = np.random.SeedSequence(seed).spawn(len(jobs))

    def fill(i):
        out = jobs[i]
        np.random.default_rng(streams[i]).standard_normal(out.size, dtype=np.float32, out=out)
        out *= np.float32(std)
        if bf16:
            out[:] = round_to_bf16(out)

    with cf.ThreadPoolExecutor(max_workers=threads) as ex:
        list(ex.map(fill, range(len(jobs))))
    weights: Dict[str, object] = {"embed": mats["embed"], "lm_head": mats["lm_head"],
                                  "final_norm": np.ones(s.d_model, dtype=np.float32), "layers": []}
    for l in range(s.n_layers):
        lay = {k: mats[(l, k)] for k in layer_matrix_names()}
        lay["attn_norm"] = np.ones(s.d_model, dtype=np.float32)
        lay["ffn_norm"] = np.ones(s.d_model, dtype=np.float32)
        weights["layers"].append(lay)
    if s.qk_norm:  # as in make_weights, from one more stream after the matrices
        rng = np.random.default_rng(np.random.SeedSequence(seed).spawn(len(jobs) + 1)[-1])
        for lay in weights["layers"]:
            for name in ("q_norm", "k_norm"):
                lay[name] = (1.0 + 0.1 * rng.standard_normal(s.head_dim)).astype(np.float32)
    return weights


def cached_kv(n_tokens: int, n_kv_heads: int, head_dim: int, seed: int, k_std: float = 1.0,
              bf16: bool = True):
    """Seeded K and V values of one layer's cache, ``[n_tokens][Hkv][Dh]`` each:
    K ~ N(0, k_std^2), V ~ N(0, 1), float32 (bf16-representable with ``bf16``).
    Used to stage long contexts directly into pages (and into the oracle's
    contiguous cache) instead of running a long prefill."""
    rng = np.random.default_rng(seed)
    k = rng.standard_normal((n_tokens, n_kv_heads, head_dim), dtype=np.float32) * np.float32(k_std)
    v = rng.standard_normal((n_tokens, n_kv_heads, head_dim), dtype=np.float32)
    if bf16:
        k, v = round_to_bf16(k), round_to_bf16(v)
    return k, v


def random_tokens(n: int, vocab: int, seed: int) -> np.ndarray:
    return np.random.default_rng(seed).integers(0, vocab, size=n, dtype=np.int64).astype(np.int32)


# ---------------------------------------------------------------------------
# Context-length distributions of the decode workloads.
# ---------------------------------------------------------------------------

def lengths_uniform(batch: int, lo: int, hi: int, seed: int) -> np.ndarray:
    """Integer lengths uniform on [lo, hi] inclusive."""
    return np.random.default_rng(seed).integers(lo, hi + 1, size=batch).astype(np.int64)


def lengths_lognormal(batch: int, median: float, sigma: float, lo: int, hi: int,
                      seed: int) -> np.ndarray:
    """Lognormal lengths (given median and log-sigma), clamped to [lo, hi]."""
    x = np.random.default_rng(seed).lognormal(np.log(median), sigma, size=batch)
    return np.clip(np.floor(x), lo, hi).astype(np.int64)


def lengths_pareto(batch: int, alpha: float, xmin: int, cap: int, seed: int) -> np.ndarray:
    """Pareto type I lengths by inverse CDF, floor(xmin * U^(-1/alpha)), capped."""
    u = np.random.default_rng(seed).random(batch)
    u = np.maximum(u, np.finfo(np.float64).tiny)
    return np.minimum(np.floor(xmin * u ** (-1.0 / alpha)), cap).astype(np.int64)


def lengths_skewed(batch: int, mean: int, sigma: float, seed: int) -> np.ndarray:
    """Within-batch skew at a fixed mean: lengths mean * exp(sigma z - sigma^2 / 2),
    z ~ N(0, 1), rescaled so the batch mean is `mean`, clamped to [16, 16 mean].
    sigma = 0 gives every trajectory the same length."""
    if sigma == 0.0 or batch == 1:
        return np.full(batch, int(mean), dtype=np.int64)
    z = np.random.default_rng(seed).standard_normal(batch)
    x = np.exp(sigma * z - 0.5 * sigma * sigma)
    x = x / x.mean() * mean
    return np.clip(np.round(x), 16, 16 * mean).astype(np.int64)


# ---------------------------------------------------------------------------
# Isolated paged decode attention operands.
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class PagedAttentionCase:
    """Operands of one isolated paged decode-attention call.

    ``k_pool`` is ``[n_pages][Hkv][16][Dh]``; ``v_pool`` holds the same
    logical ``[n_pages][Hkv][16][Dh]`` values (the GPU side stores V pages
    transposed, which is a layout choice of that side).  ``block_table[b]``
    lists the physical pages of sequence b in logical order; only the first
    ``ceil(lens[b]/16)`` entries are meaningful and the rest are -1.
    """

    q: np.ndarray           # [B, Hq, Dh] float32 (bf16-representable when bf16)
    k_pool: np.ndarray      # [P, Hkv, 16, Dh] float32
    v_pool: np.ndarray      # [P, Hkv, 16, Dh] float32
    block_table: np.ndarray  # [B, max_pages] int32
    lens: np.ndarray        # [B] int64, number of cached keys per sequence


def paged_attention_case(batch: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                         lens: np.ndarray, n_pool_pages: int, seed: int, bf16: bool = True,
                         poison_tail: bool = True) -> PagedAttentionCase:
    """Random Q/K/V ~ N(0,1) and block tables drawn from a random page permutation.

    The pages of sequence b are the next ceil(lens[b]/16) entries of one
    random permutation of the pool, so no page is shared.  Slots beyond a
    sequence's length in its last page are filled with NaN when
    ``poison_tail`` is set: a correct kernel never reads them.
    """
    rng = np.random.default_rng(seed)
    lens = np.asarray(lens, dtype=np.int64)
    npages = (lens + PAGE_TOKENS - 1) // PAGE_TOKENS
    if int(npages.sum()) > n_pool_pages:
        raise ValueError("pool too small for the requested lengths")
    perm = rng.permutation(n_pool_pages).astype(np.int32)
    max_pages = int(npages.max()) if batch else 0
    bt = np.full((batch, max(max_pages, 1)), -1, dtype=np.int32)
    cursor = 0
    for b in range(batch):
        bt[b, :npages[b]] = perm[cursor:cursor + npages[b]]
        cursor += int(npages[b])
    used = perm[:cursor]
    k_pool = np.zeros((n_pool_pages, n_kv_heads, PAGE_TOKENS, head_dim), dtype=np.float32)
    v_pool = np.zeros_like(k_pool)
    kdraw = rng.standard_normal((cursor, n_kv_heads, PAGE_TOKENS, head_dim), dtype=np.float32)
    vdraw = rng.standard_normal((cursor, n_kv_heads, PAGE_TOKENS, head_dim), dtype=np.float32)
    q = rng.standard_normal((batch, n_q_heads, head_dim), dtype=np.float32)
    if bf16:
        kdraw, vdraw, q = round_to_bf16(kdraw), round_to_bf16(vdraw), round_to_bf16(q)
    k_pool[used] = kdraw
    v_pool[used] = vdraw
    if poison_tail:
        for b in range(batch):
            tail = int(lens[b] % PAGE_TOKENS)
            if tail:
                last = bt[b, npages[b] - 1]
                k_pool[last, :, tail:, :] = np.nan
                v_pool[last, :, tail:, :] = np.nan
    return PagedAttentionCase(q=q, k_pool=k_pool, v_pool=v_pool, block_table=bt, lens=lens)


@dataclasses.dataclass
class PagedAttentionCaseFp8:
    """Isolated decode-attention operands with E4M3 code pages (uint8)."""

    q: np.ndarray          # [B, Hq, Dh] float32, bf16-representable
    k_codes: np.ndarray    # [P, Hkv, 16, Dh] uint8
    v_codes: np.ndarray    # [P, Hkv, 16, Dh] uint8
    block_table: np.ndarray
    lens: np.ndarray


def paged_attention_case_fp8(batch: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                             lens: np.ndarray, n_pool_pages: int, seed: int,
                             exponents=(4, 9), all_codes: bool = False) -> PagedAttentionCaseFp8:
    """Random E4M3 K/V codes built from their bit fields, and block tables.

    Each code is sign << 7 | e << 3 | m with a random sign, e uniform in
    ``exponents`` (inclusive; bias 7, so (4, 9) spans about 2^-3 .. 2^2.9) and
    m uniform in 0..7; with ``all_codes`` every finite code (all but
    0x7F and 0xFF) is equally likely.  Pages come from one random permutation
    of the pool as in paged_attention_case, and slots past a sequence's length
    hold the NaN code 0x7F, which a correct kernel never reads.
    """
    rng = np.random.default_rng(seed)
    lens = np.asarray(lens, dtype=np.int64)
    npages = (lens + PAGE_TOKENS - 1) // PAGE_TOKENS
    if int(npages.sum()) > n_pool_pages:
        raise ValueError("pool too small for the requested lengths")
    perm = rng.permutation(n_pool_pages).astype(np.int32)
    bt = np.full((batch, max(int(npages.max()), 1)), -1, dtype=np.int32)
    cursor = 0
    for b in range(batch):
        bt[b, :npages[b]] = perm[cursor:cursor + npages[b]]
        cursor += int(npages[b])
    shape = (n_pool_pages, n_kv_heads, PAGE_TOKENS, head_dim)

    def codes():
        if all_codes:
            finite = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], dtype=np.uint8)
            return finite[rng.integers(0, finite.size, size=shape)]
        sign = rng.integers(0, 2, size=shape, dtype=np.uint8)
        e = rng.integers(exponents[0], exponents[1] + 1, size=shape, dtype=np.uint8)
        m = rng.integers(0, 8, size=shape, dtype=np.uint8)
        return (sign << 7) | (e << 3) | m

    k_codes, v_codes = codes(), codes()
    q = round_to_bf16(rng.standard_normal((batch, n_q_heads, head_dim), dtype=np.float32))
    for b in range(batch):
        tail = int(lens[b] % PAGE_TOKENS)
        if tail:
            last = bt[b, npages[b] - 1]
            k_codes[last, :, tail:, :] = 0x7F
            v_codes[last, :, tail:, :] = 0x7F
    return PagedAttentionCaseFp8(q=q, k_codes=k_codes, v_codes=v_codes, block_table=bt, lens=lens)


@dataclasses.dataclass
class LazyPagedAttentionCase:
    """Isolated decode-attention operands for a big pool, drawn per sequence.

    The block table comes from one random permutation of the pool; the
    K/V of sequence b (``[n_pages_b, Hkv, 16, Dh]``, float32,
    bf16-representable, tail slots NaN) and its query are drawn from a
    generator seeded by (seed, b), so any subset of sequences can be
    regenerated on its own.
    """

    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    lens: np.ndarray
    block_table: np.ndarray
    n_pool_pages: int
    seed: int

    def sequence(self, b: int):
        rng = np.random.default_rng([self.seed, int(b)])
        n = int(self.lens[b])
        npg = (n + PAGE_TOKENS - 1) // PAGE_TOKENS
        shp = (npg, self.n_kv_heads, PAGE_TOKENS, self.head_dim)
        k = round_to_bf16(rng.standard_normal(shp, dtype=np.float32))
        v = round_to_bf16(rng.standard_normal(shp, dtype=np.float32))
        q = round_to_bf16(rng.standard_normal((self.n_q_heads, self.head_dim), dtype=np.float32))
        tail = n % PAGE_TOKENS
        if tail:
            k[-1, :, tail:, :] = np.nan
            v[-1, :, tail:, :] = np.nan
        return q, k, v


def lazy_paged_attention_case(batch: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                              lens: np.ndarray, n_pool_pages: int,
                              seed: int) -> LazyPagedAttentionCase:
    lens = np.asarray(lens, dtype=np.int64)
    npages = (lens + PAGE_TOKENS - 1) // PAGE_TOKENS
    if int(npages.sum()) > n_pool_pages:
        raise ValueError("pool too small for the requested lengths")
    perm = np.random.default_rng(seed).permutation(n_pool_pages).astype(np.int32)
    bt = np.zeros((batch, int(npages.max())), dtype=np.int32)
    cursor = 0
    for b in range(batch):
        bt[b, :npages[b]] = perm[cursor:cursor + npages[b]]
        cursor += int(npages[b])
    return LazyPagedAttentionCase(n_q_heads, n_kv_heads, head_dim, lens, bt, n_pool_pages, seed)
