"""Pins of the CPU oracle against things other than itself.

* closed forms typed in ``tests/golden/closed_forms.txt`` (RoPE, RMSNorm, SiLU);
* mathematical invariants (RoPE norm and relative-position property, unit
  RMS, softmax weights summing to one, single-key and equal-key attention);
* library routines: torch's scaled-dot-product attention, and the whole
  decoder against transformers' LlamaForCausalLM built with the same weights;
* the cached step against a full recompute without a cache;
* planted mistakes: each plausible bug in the oracle must break a pin.
"""

import dataclasses
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import decoder as od
from workload import PAGE_TOKENS, ModelShape, TINY, TINY_QK, make_weights, random_tokens

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "closed_forms.txt")


def golden():
    vals = {}
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            name, *nums = line.split()
            vals[name] = np.array([float(x) for x in nums])
    return vals


# ---------------------------------------------------------------- elementary ops

def test_rope_closed_form():
    g = golden()
    e0 = np.array([[1.0, 0.0, 0.0, 0.0]])
    e1 = np.array([[0.0, 1.0, 0.0, 0.0]])
    np.testing.assert_allclose(od.rope(e0, 2, 10000.0)[0], g["rope_e0_p2"], atol=1e-15)
    np.testing.assert_allclose(od.rope(e1, 3, 10000.0)[0], g["rope_e1_p3"], atol=1e-15)


def test_rope_invariants():
    rng = np.random.default_rng(5)
    z = rng.standard_normal((3, 64))
    np.testing.assert_array_equal(od.rope(z, 0, 10000.0), z)          # identity at p=0
    for p in (1, 17, 4097, 131071):
        r = od.rope(z, p, 10000.0)
        np.testing.assert_allclose(np.linalg.norm(r, axis=-1), np.linalg.norm(z, axis=-1),
                                   rtol=1e-12)                           # norm preserving
    q, k = rng.standard_normal((1, 64)), rng.standard_normal((1, 64))
    d1 = od.rope(q, 50, 1e4)[0] @ od.rope(k, 20, 1e4)[0]
    d2 = od.rope(q, 1030, 1e4)[0] @ od.rope(k, 1000, 1e4)[0]
    np.testing.assert_allclose(d1, d2, rtol=1e-9)                      # depends on m-n only


def test_rmsnorm_and_silu_closed_forms():
    g = golden()
    np.testing.assert_allclose(od.rmsnorm(np.array([3.0, 4.0]), np.ones(2), 0.0),
                               g["rmsnorm_3_4"], rtol=1e-15)
    np.testing.assert_allclose(od.silu(np.array([1.0, -1.0])),
                               np.concatenate([g["silu_1"], g["silu_m1"]]), rtol=1e-15)
    assert od.silu(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(od.silu(np.array([40.0])), [40.0], rtol=1e-15)
    x = np.random.default_rng(1).standard_normal((5, 300)) * 7
    y = od.rmsnorm(x, np.ones(300), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=-1)), 1.0, rtol=1e-13)


# ------------------------------------------------------------------- attention

def test_attention_single_key_and_equal_keys():
    rng = np.random.default_rng(2)
    q = rng.standard_normal((8, 32))
    k1, v1 = rng.standard_normal((1, 2, 32)), rng.standard_normal((1, 2, 32))
    o = od.attention(q, k1, v1)
    for h in range(8):
        np.testing.assert_allclose(o[h], v1[0, h // 4], rtol=1e-15)   # L=1 => o = v
    keys = np.repeat(rng.standard_normal((1, 2, 32)), 9, axis=0)
    vals = rng.standard_normal((9, 2, 32))
    o = od.attention(q, keys, vals)
    for h in range(8):
        np.testing.assert_allclose(o[h], vals[:, h // 4].mean(axis=0), rtol=1e-12)


def test_attention_weights_sum_to_one():
    rng = np.random.default_rng(3)
    t, dh = 40, 64
    q = rng.standard_normal((4, dh)) * 3
    keys = rng.standard_normal((t, 1, dh))
    vals = np.zeros((t, 1, dh))
    vals[:, 0, :t] = np.eye(t)  # value j is the unit vector e_j: output = weights
    o = od.attention(q, keys, vals)
    np.testing.assert_allclose(o[:, :t].sum(axis=1), 1.0, rtol=1e-13)
    assert (o[:, :t] >= 0).all()


@pytest.mark.parametrize("hq,hkv", [(8, 2), (4, 4), (32, 8)])
def test_attention_matches_torch_sdpa(hq, hkv):
    rng = np.random.default_rng(4)
    t, dh = 37, 64
    q = rng.standard_normal((hq, dh))
    keys, vals = rng.standard_normal((t, hkv, dh)), rng.standard_normal((t, hkv, dh))
    o = od.attention(q, keys, vals)
    rep = hq // hkv
    kt = torch.from_numpy(keys).permute(1, 0, 2).repeat_interleave(rep, dim=0)
    vt = torch.from_numpy(vals).permute(1, 0, 2).repeat_interleave(rep, dim=0)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[:, None, :], kt, vt)[:, 0, :].numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-13)


def test_paged_gather_equals_contiguous():
    rng = np.random.default_rng(6)
    hkv, dh, n = 2, 16, 53
    hist_k = rng.standard_normal((n, hkv, dh))
    hist_v = rng.standard_normal((n, hkv, dh))
    npages = (n + PAGE_TOKENS - 1) // PAGE_TOKENS
    pool_k = np.full((11, hkv, PAGE_TOKENS, dh), np.nan)
    pool_v = np.full_like(pool_k, np.nan)
    row = rng.permutation(11)[:npages]
    for j in range(n):
        pool_k[row[j // 16], :, j % 16] = hist_k[j]
        pool_v[row[j // 16], :, j % 16] = hist_v[j]
    np.testing.assert_array_equal(oracle.gather_pages(pool_k, row, n), hist_k)
    q = rng.standard_normal((1, 8, dh))
    out = oracle.paged_decode_attention(q, pool_k, pool_v, row[None, :], [n])
    np.testing.assert_allclose(out[0], od.attention(q[0], hist_k, hist_v), rtol=1e-15)


def test_greedy_ties_and_nan():
    assert od.greedy(np.array([1.0, 3.0, 3.0, 2.0])) == 1
    with pytest.raises(ValueError):
        od.greedy(np.array([1.0, np.nan]))


# --------------------------------------------------------------- whole decoder

SMALL = ModelShape(n_layers=2, d_model=64, n_q_heads=8, n_kv_heads=2, head_dim=16,
                   ffn_dim=96, vocab=97)


def _hf_logits(shape, arrays, tokens):
    """Logits from transformers' Llama built with the same weights (float64)."""
    from transformers import LlamaConfig, LlamaForCausalLM
    cfg = LlamaConfig(vocab_size=shape.vocab, hidden_size=shape.d_model,
                      intermediate_size=shape.ffn_dim, num_hidden_layers=shape.n_layers,
                      num_attention_heads=shape.n_q_heads, num_key_value_heads=shape.n_kv_heads,
                      head_dim=shape.head_dim, rms_norm_eps=shape.rms_eps,
                      rope_theta=shape.rope_base, tie_word_embeddings=False,
                      attention_bias=False, mlp_bias=False, max_position_embeddings=4096)
    torch.manual_seed(0)
    m = LlamaForCausalLM(cfg).double().eval()
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(t(arrays["embed"]))
        m.lm_head.weight.copy_(t(arrays["lm_head"]))
        m.model.norm.weight.copy_(t(arrays["final_norm"]))
        for lay, hl in zip(arrays["layers"], m.model.layers):
            hl.self_attn.q_proj.weight.copy_(t(lay["wq"]))
            hl.self_attn.k_proj.weight.copy_(t(lay["wk"]))
            hl.self_attn.v_proj.weight.copy_(t(lay["wv"]))
            hl.self_attn.o_proj.weight.copy_(t(lay["wo"]))
            hl.mlp.gate_proj.weight.copy_(t(lay["w_gate"]))
            hl.mlp.up_proj.weight.copy_(t(lay["w_up"]))
            hl.mlp.down_proj.weight.copy_(t(lay["w_down"]))
            hl.input_layernorm.weight.copy_(t(lay["attn_norm"]))
            hl.post_attention_layernorm.weight.copy_(t(lay["ffn_norm"]))
        out = m(torch.tensor([list(map(int, tokens))])).logits[0].numpy()
    return out


def _hf_arrays(shape, seed):
    # std 0.2 so every sub-block moves the residual stream visibly and a
    # dropped or mangled term changes the logits well beyond the tolerance.
    arrays = make_weights(shape, seed=seed, std=0.2)
    rng = np.random.default_rng(seed + 100)
    for lay in arrays["layers"]:  # non-trivial norm gains so gains are exercised
        lay["attn_norm"] = (1 + 0.3 * rng.standard_normal(shape.d_model)).astype(np.float32)
        lay["ffn_norm"] = (1 + 0.3 * rng.standard_normal(shape.d_model)).astype(np.float32)
    arrays["final_norm"] = (1 + 0.3 * rng.standard_normal(shape.d_model)).astype(np.float32)
    return arrays


def _oracle_all_logits(shape, arrays, tokens):
    dec = od.Decoder(od.ModelWeights.from_arrays(shape, arrays))
    st = dec.new_state()
    return np.stack([dec.step(st, t) for t in tokens])


def _close_to_hf(got, ref):
    # The library keeps RMSNorm and the rotary tables in float32 internally,
    # so agreement is to float32 rounding, far below any planted mistake.
    return np.max(np.abs(got - ref)) <= 2e-5 * np.max(np.abs(ref))


def _hf_qwen3_logits(shape, arrays, tokens):
    """Logits from transformers' Qwen3 (per-head q/k RMSNorm) with the same weights."""
    from transformers import Qwen3Config, Qwen3ForCausalLM
    cfg = Qwen3Config(vocab_size=shape.vocab, hidden_size=shape.d_model,
                      intermediate_size=shape.ffn_dim, num_hidden_layers=shape.n_layers,
                      num_attention_heads=shape.n_q_heads, num_key_value_heads=shape.n_kv_heads,
                      head_dim=shape.head_dim, rms_norm_eps=shape.rms_eps,
                      rope_theta=shape.rope_base, tie_word_embeddings=False,
                      attention_bias=False, max_position_embeddings=4096,
                      use_sliding_window=False)
    torch.manual_seed(0)
    m = Qwen3ForCausalLM(cfg).double().eval()
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(t(arrays["embed"]))
        m.lm_head.weight.copy_(t(arrays["lm_head"]))
        m.model.norm.weight.copy_(t(arrays["final_norm"]))
        for lay, hl in zip(arrays["layers"], m.model.layers):
            hl.self_attn.q_proj.weight.copy_(t(lay["wq"]))
            hl.self_attn.k_proj.weight.copy_(t(lay["wk"]))
            hl.self_attn.v_proj.weight.copy_(t(lay["wv"]))
            hl.self_attn.o_proj.weight.copy_(t(lay["wo"]))
            hl.self_attn.q_norm.weight.copy_(t(lay["q_norm"]))
            hl.self_attn.k_norm.weight.copy_(t(lay["k_norm"]))
            hl.mlp.gate_proj.weight.copy_(t(lay["w_gate"]))
            hl.mlp.up_proj.weight.copy_(t(lay["w_up"]))
            hl.mlp.down_proj.weight.copy_(t(lay["w_down"]))
            hl.input_layernorm.weight.copy_(t(lay["attn_norm"]))
            hl.post_attention_layernorm.weight.copy_(t(lay["ffn_norm"]))
        out = m(torch.tensor([list(map(int, tokens))])).logits[0].numpy()
    return out


@pytest.mark.parametrize("shape", [dataclasses.replace(SMALL, qk_norm=True), TINY_QK])
def test_decoder_matches_transformers_qwen3(shape):
    arrays = _hf_arrays(shape, seed=13)
    rng = np.random.default_rng(14)
    for lay in arrays["layers"]:  # q/k gains well away from 1
        lay["q_norm"] = (1 + 0.3 * rng.standard_normal(shape.head_dim)).astype(np.float32)
        lay["k_norm"] = (1 + 0.3 * rng.standard_normal(shape.head_dim)).astype(np.float32)
    tokens = random_tokens(23, shape.vocab, seed=15)
    ref = _hf_qwen3_logits(shape, arrays, tokens)
    got = _oracle_all_logits(shape, arrays, tokens)
    assert _close_to_hf(got, ref), np.max(np.abs(got - ref))
    # and the cached decoder equals its own recomputation
    full = od.recompute_logits(od.ModelWeights.from_arrays(shape, arrays), tokens)
    np.testing.assert_allclose(got, full, rtol=0, atol=1e-10 * np.max(np.abs(full)))


@pytest.mark.parametrize("shape", [SMALL, TINY])
def test_decoder_matches_transformers_llama(shape):
    arrays = _hf_arrays(shape, seed=11)
    tokens = random_tokens(23, shape.vocab, seed=12)
    ref = _hf_logits(shape, arrays, tokens)
    got = _oracle_all_logits(shape, arrays, tokens)
    assert _close_to_hf(got, ref), np.max(np.abs(got - ref))


def test_cached_step_equals_recompute():
    arrays = make_weights(SMALL, seed=3, std=0.2)
    w = od.ModelWeights.from_arrays(SMALL, arrays)
    tokens = random_tokens(40, SMALL.vocab, seed=4)
    inc = _oracle_all_logits(SMALL, arrays, tokens)
    full = od.recompute_logits(w, tokens)
    np.testing.assert_allclose(inc, full, rtol=0, atol=1e-10 * np.max(np.abs(full)))


def test_prefill_then_steps_equals_recompute():
    arrays = make_weights(TINY, seed=0)
    w = od.ModelWeights.from_arrays(TINY, arrays)
    tokens = random_tokens(30, TINY.vocab, seed=9)
    dec = od.Decoder(w)
    st = dec.new_state()
    last = dec.prefill(st, tokens[:17])
    full = od.recompute_logits(w, tokens)
    np.testing.assert_allclose(last, full[16], rtol=0, atol=1e-12)
    for i in range(17, 30):
        np.testing.assert_allclose(dec.step(st, tokens[i]), full[i], rtol=0, atol=1e-12)
    assert st["len"] == 30 and st["k"][0].shape == (30, TINY.n_kv_heads, TINY.head_dim)


# ------------------------------------------------------------- planted mistakes

def _mut_rope_interleaved(z, positions, base):
    dh = z.shape[-1]
    i = np.arange(dh // 2, dtype=np.float64)
    theta = base ** (-2.0 * i / dh)
    ang = np.asarray(positions, dtype=np.float64)[..., None, None] * theta
    c, s = np.cos(ang), np.sin(ang)
    a, b = z[..., 0::2], z[..., 1::2]
    out = np.empty_like(z)
    out[..., 0::2] = a * c - b * s
    out[..., 1::2] = a * s + b * c
    return out


_ROPE = od.rope
_ATTENTION = od.attention


def _mut_rope_sign(z, positions, base):
    return _ROPE(z, -np.asarray(positions, dtype=np.float64), base)


def _mut_gqa_modulo(q, keys, values):
    hq, dh = q.shape
    hkv = keys.shape[1]
    out = np.empty_like(q)
    for h in range(hq):
        g = h % hkv
        s = keys[:, g, :] @ q[h] / np.sqrt(dh)
        a = np.exp(s - s.max())
        out[h] = (a / a.sum()) @ values[:, g, :]
    return out


def _mut_no_scale(q, keys, values):
    return _ATTENTION(q * np.sqrt(q.shape[1]), keys, values)


def _mut_rmsnorm_no_gain(x, gain, eps):
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps)


def _mut_silu_sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


@pytest.mark.parametrize("name,attr,mutant", [
    ("rope pairing", "rope", _mut_rope_interleaved),
    ("rope sign", "rope", _mut_rope_sign),
    ("gqa mapping", "attention", _mut_gqa_modulo),
    ("attention scale", "attention", _mut_no_scale),
    ("norm gain dropped", "rmsnorm", _mut_rmsnorm_no_gain),
    ("silu -> sigmoid", "silu", _mut_silu_sigmoid),
])
def test_planted_mistake_breaks_library_pin(monkeypatch, name, attr, mutant):
    arrays = _hf_arrays(SMALL, seed=11)
    tokens = random_tokens(23, SMALL.vocab, seed=12)
    ref = _hf_logits(SMALL, arrays, tokens)
    monkeypatch.setattr(od, attr, mutant)
    got = _oracle_all_logits(SMALL, arrays, tokens)
    assert not _close_to_hf(got, ref), name


_RMSNORM = od.rmsnorm


def _mut_qk_norm_whole_vector(x, gain, eps):
    """Per-head norm done over all heads of q (or k) at once."""
    if x.ndim >= 2 and gain.shape[-1] != x.shape[-1] * x.shape[-2]:
        flat = x.reshape(*x.shape[:-2], -1)
        ms = np.mean(flat * flat, axis=-1, keepdims=True)[..., None]
        return x / np.sqrt(ms + eps) * gain
    return _RMSNORM(x, gain, eps)


def _qwen3_case():
    shape = dataclasses.replace(SMALL, qk_norm=True)
    arrays = _hf_arrays(shape, seed=13)
    rng = np.random.default_rng(14)
    for lay in arrays["layers"]:
        lay["q_norm"] = (1 + 0.3 * rng.standard_normal(shape.head_dim)).astype(np.float32)
        lay["k_norm"] = (1 + 0.3 * rng.standard_normal(shape.head_dim)).astype(np.float32)
    tokens = random_tokens(23, shape.vocab, seed=15)
    return shape, arrays, tokens


def test_planted_qk_norm_mistakes_break_qwen3_pin(monkeypatch):
    shape, arrays, tokens = _qwen3_case()
    ref = _hf_qwen3_logits(shape, arrays, tokens)
    with monkeypatch.context() as mp:
        mp.setattr(od, "rmsnorm", _mut_qk_norm_whole_vector)
        assert not _close_to_hf(_oracle_all_logits(shape, arrays, tokens), ref)
    swapped = {**arrays, "layers": [{**lay, "q_norm": lay["k_norm"], "k_norm": lay["q_norm"]}
                                    for lay in arrays["layers"]]}
    assert not _close_to_hf(_oracle_all_logits(shape, swapped, tokens), ref)
