"""The full 8B-shaped decoder (32 layers, d 4096, 32/8 heads, Dh 128, FFN 14336,
vocabulary 128256; random bf16 weights) against the float64 oracle (GPU).

Two trajectories: prefixes of 16 and 9 tokens appended in one batched call
(with their last-position logits), then three decode steps of both.  Every
logits row is compared with the oracle's full recompute over the same bf16
weights, and with a float64 model of the bf16 path's rounding points (below).

Through 32 layers the bf16 activations alone move the logits by a few percent
of max|ref| (that model drifts 3.1-3.8% from the exact oracle on these
weights), so the exact oracle's 2e-2 bar cannot hold at this depth for this
arithmetic; the 2-layer full-width test holds it.  Asserted per row:
  * max|gpu - model| <= 3e-2 max|ref| (the GPU follows the bf16 arithmetic),
  * max|gpu - exact| <= max|model - exact| + 2e-2 max|ref|,
  * greedy agreement with the exact oracle where its top-2 gap is clear.

Host memory: ~100 GB (float32 draw and the float64 weights).
"""

import sys
import time

import numpy as np
import pytest
import torch

from oracle import decoder as od
from workload import EIGHT_B, make_weights_parallel, random_tokens, round_to_bf16

pytestmark = pytest.mark.gpu

TOL = 2e-2       # the bf16 bar
TOL_MODEL = 3e-2  # GPU against the float64 model of its rounding points


def _bf16(a):
    """Round float64 values to the nearest bf16 (ties to even), as float64."""
    return round_to_bf16(np.asarray(a, dtype=np.float32)).astype(np.float64)


def recompute_logits_bf16_activations(w, tokens):
    """The oracle's full recompute with the bf16 path's rounding points
    (written out from the path's definition: weights and KV stored in bf16,
    activations rounded to bf16 where they enter a matrix product: h, q, k,
    v, the softmax weights P with the normaliser summing the rounded weights,
    the attention output o, the SwiGLU output u, and the final h).  Float64
    otherwise.  A diagnostic reference: it shows how far the exact oracle and
    the GPU drift apart through 32 layers of bf16 activations."""
    n = len(tokens)
    pos = np.arange(n)
    x = w.embed[np.asarray(tokens, dtype=np.int64)].copy()
    group = w.n_q_heads // w.n_kv_heads
    mask = np.tril(np.ones((n, n), dtype=bool))
    for lay in w.layers:
        h = _bf16(od.rmsnorm(x, lay["attn_norm"], w.rms_eps))
        q = (h @ lay["wq"].T).reshape(n, w.n_q_heads, w.head_dim)
        k = (h @ lay["wk"].T).reshape(n, w.n_kv_heads, w.head_dim)
        v = _bf16((h @ lay["wv"].T).reshape(n, w.n_kv_heads, w.head_dim))
        q = _bf16(od.rope(q, pos, w.rope_base))
        k = _bf16(od.rope(k, pos, w.rope_base))
        o = np.empty_like(q)
        for hh in range(w.n_q_heads):
            g = hh // group
            sc = (q[:, hh, :] @ k[:, g, :].T) / np.sqrt(w.head_dim)
            sc = np.where(mask, sc, -np.inf)
            p = _bf16(np.exp(sc - sc.max(axis=1, keepdims=True)))
            o[:, hh, :] = (p @ v[:, g, :]) / p.sum(axis=1, keepdims=True)
        x = x + _bf16(o.reshape(n, -1)) @ lay["wo"].T
        h2 = _bf16(od.rmsnorm(x, lay["ffn_norm"], w.rms_eps))
        u = _bf16(od.silu(h2 @ lay["w_gate"].T) * (h2 @ lay["w_up"].T))
        x = x + u @ lay["w_down"].T
    return _bf16(od.rmsnorm(x, w.final_norm, w.rms_eps)) @ w.lm_head.T


def _say(msg):
    sys.stderr.write(f"[full-8b] {msg}\n")
    sys.stderr.flush()


def test_full_8b_decoder_matches_oracle():
    import paper_2609_36899_amd as P
    t0 = time.time()
    arrays = make_weights_parallel(EIGHT_B, seed=21, bf16=True)
    _say(f"weights drawn ({time.time() - t0:.0f} s)")
    w = P.weights_to_device(arrays, P.BF16)
    torch.cuda.synchronize()
    _say(f"weights on the device ({time.time() - t0:.0f} s)")
    per_tok = P.kv_bytes_per_token(EIGHT_B, P.BF16)
    E = P.Engine(EIGHT_B, w, P.BF16, 256 * per_tok, max_seqs=2, max_seq_len=64, max_batch=2,
                 max_chunk=32)
    lens, n_steps = (16, 9), 3
    toks = [random_tokens(n + n_steps, EIGHT_B.vocab, seed=210 + i) for i, n in enumerate(lens)]
    seqs = [E.kv_alloc(0) for _ in lens]
    first = torch.empty((2, EIGHT_B.vocab), dtype=torch.float32, device="cuda")
    E.kv_append_prefix_batch(seqs, [t[:n] for t, n in zip(toks, lens)], chunk_tokens=32,
                             last_logits=first)
    rows = [[r] for r in first.cpu().numpy()]
    logits = torch.empty((2, EIGHT_B.vocab), dtype=torch.float32, device="cuda")
    for k in range(n_steps):
        step = np.array([t[n + k] for t, n in zip(toks, lens)], dtype=np.int32)
        E.decode_step(seqs, torch.from_numpy(step).cuda(), logits)
        got = logits.cpu().numpy()
        for i in range(2):
            rows[i].append(got[i].copy())
    E.close()
    del E, w
    torch.cuda.empty_cache()
    _say(f"GPU done ({time.time() - t0:.0f} s); float64 oracle")
    w64 = od.ModelWeights.from_arrays(EIGHT_B, arrays)
    del arrays
    worst, agreed = 0.0, 0
    for i, n in enumerate(lens):
        ref = od.recompute_logits(w64, toks[i])[n - 1:]
        emu = recompute_logits_bf16_activations(w64, toks[i])[n - 1:]
        _say(f"oracle trajectory {i} done ({time.time() - t0:.0f} s)")
        g = np.stack(rows[i])
        assert np.isfinite(g).all()
        for r in range(ref.shape[0]):
            nrm = float(np.max(np.abs(ref[r])))
            rel = float(np.max(np.abs(g[r] - ref[r]))) / nrm
            rel_emu = float(np.max(np.abs(g[r] - emu[r]))) / nrm
            rel_ref_emu = float(np.max(np.abs(emu[r] - ref[r]))) / nrm
            _say(f"trajectory {i} row {r}: gpu-exact {rel:.3e}  gpu-bf16acts {rel_emu:.3e}  "
                 f"bf16acts-exact {rel_ref_emu:.3e}")
            worst = max(worst, rel)
            assert rel_emu <= TOL_MODEL, (i, r, rel_emu)
            assert rel <= rel_ref_emu + TOL, (i, r, rel, rel_ref_emu)
            top2 = np.sort(ref[r])[-2:]
            if top2[1] - top2[0] > 4 * TOL * np.max(np.abs(ref[r])):
                assert int(np.argmax(g[r])) == int(od.greedy(ref[r])), (i, r)
                agreed += 1
    _say(f"worst row error {worst:.3e} of max|ref|; {agreed} clear greedy tokens agree")
