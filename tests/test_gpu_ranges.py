"""Parity at the workloads' own ranges, through the C ABI, against the float64
oracle (GPU).

* The LM head at the 8B shape's vocabulary (N = 128256, K = 4096) for
  M = 1, 16, 33, 256 and 512 rows: every kernel the planner picks for it (the
  streaming kernel, the 128- and 256-row tiles, the 256 x 256 tile).  bf16
  inputs, float64 products, per row max|gpu - ref| <= 1e-4 * max|ref|.
* Greedy argmax over 128256 logits with planted ties (lowest index wins),
  rows of equal values, a maximum only in the first or last slot, against
  numpy's argmax of the same float32 values: exact.
* A decoder with the full 128256-entry vocabulary: 33 prefixes appended in
  one multi-sequence call (LM-head rows gathered from several sequences of a
  pass) and decode steps, logits normwise 2e-2, greedy agreement where the
  oracle's top-2 gap is clear.
* Decode at positions 65K-131K: contexts staged with kv_extend_uninit, their
  pages filled with seeded K/V that the oracle's contiguous cache also holds;
  two decode steps.  The rotary angle at these positions, the page index
  arithmetic and the KV write are all exercised: logits and the K/V the GPU
  wrote at the new positions are compared (bf16: 2e-2 normwise; fp32: 1e-4).
* The multi-sequence append equals the oracle and the per-sequence append.
* Departure, re-admission with a reserve and growth before the block-table
  entries reach the device (the freed slot's stale entries must not win).
"""

import numpy as np
import pytest
import torch

from oracle import decoder as od
from workload import (EIGHT_B, TINY, ModelShape, cached_kv, make_weights, random_tokens,
                      round_to_bf16)

pytestmark = pytest.mark.gpu

F32_TOL = 1e-4
BF16_TOL = 2e-2
V8B, K8B = EIGHT_B.vocab, EIGHT_B.d_model


def _P():
    import paper_2609_36899_amd as P
    return P


def _engine(shape, arrays, bf16, pool_tokens, max_seqs=8, max_seq_len=1024, max_batch=8,
            max_chunk=64):
    P = _P()
    dt = P.BF16 if bf16 else P.F32
    w = P.weights_to_device(arrays, dt)
    per_tok = P.kv_bytes_per_token(shape, dt)
    return P.Engine(shape, w, dt, pool_tokens * per_tok, max_seqs, max_seq_len, max_batch,
                    max_chunk)


def _rows_close(got, ref, tol, tag):
    for r in range(ref.shape[0]):
        err = float(np.max(np.abs(got[r] - ref[r])))
        assert err <= tol * float(np.max(np.abs(ref[r]))), (tag, r, err)


# ---------------------------------------------------------------------------
# LM head and argmax at V = 128256
# ---------------------------------------------------------------------------

@pytest.fixture(scope="module")
def lm_head_8b():
    P = _P()
    rng = np.random.default_rng(2024)
    w = round_to_bf16(rng.standard_normal((V8B, K8B), dtype=np.float32) * np.float32(0.02))
    wd = P.pack_weight(torch.from_numpy(w).cuda().to(torch.bfloat16).contiguous())
    torch.cuda.synchronize()
    return w, wd


def _ref_rows(x_rows, w):
    x64 = x_rows.astype(np.float64)
    out = np.empty((x_rows.shape[0], w.shape[0]), dtype=np.float64)
    for c in range(0, w.shape[0], 16384):
        out[:, c:c + 16384] = x64 @ w[c:c + 16384].astype(np.float64).T
    return out


@pytest.mark.parametrize("M", [1, 16, 33, 256, 512])
def test_lm_head_full_vocab(lm_head_8b, M):
    P = _P()
    w, wd = lm_head_8b
    rng = np.random.default_rng(M)
    x = round_to_bf16(rng.standard_normal((M, K8B), dtype=np.float32))
    out = torch.empty((M, V8B), dtype=torch.float32, device="cuda")
    P.weight_projection(torch.from_numpy(x).cuda().to(torch.bfloat16).contiguous(), wd, out)
    got = out.cpu().numpy()
    rows = np.arange(M) if M <= 33 else np.array(sorted({0, 1, M // 2, M - 2, M - 1} |
                                                        set(rng.integers(0, M, 3).tolist())))
    assert np.isfinite(got).all()
    _rows_close(got[rows], _ref_rows(x[rows], w), 1e-4, ("lm_head", M))


VOCAB_SHAPE = ModelShape(n_layers=1, d_model=64, n_q_heads=1, n_kv_heads=1, head_dim=64,
                         ffn_dim=64, vocab=V8B)


def test_greedy_argmax_full_vocab_with_planted_ties():
    arrays = make_weights(VOCAB_SHAPE, seed=3, bf16=True)
    E = _engine(VOCAB_SHAPE, arrays, bf16=True, pool_tokens=256, max_batch=64)
    rng = np.random.default_rng(11)
    for B in (1, 7, 512):
        lg = (rng.standard_normal((B, V8B)) * 3).astype(np.float32)
        # Quantise so that ties are common, then plant specific ones.
        lg = np.round(lg * 4) / 4
        lg[0, :] = lg[0].max()  # all equal -> 0
        if B > 1:
            lg[1, :] = -np.inf
            lg[1, V8B - 1] = 5.0            # the maximum only in the last slot
        if B > 2:
            lg[2, :] = -np.inf
            lg[2, 0] = -1e30                # the maximum only in the first slot
        if B > 3:
            m = lg[3].max()
            lg[3, 70000] = m + 1
            lg[3, 123] = m + 1              # tie: the lower index wins
            lg[3, 128255] = m + 1
        for b in range(4, B):
            j = rng.integers(0, V8B, 3)
            lg[b, j] = lg[b].max() + rng.choice([0.0, 0.25])
        tok = torch.empty(B, dtype=torch.int32, device="cuda")
        E.sample(torch.from_numpy(lg).cuda(), tok)
        np.testing.assert_array_equal(tok.cpu().numpy(), np.argmax(lg, axis=1))
    E.close()


def test_decoder_with_full_vocab_batched_prefill_and_steps():
    """33 trajectories (the LM head's 33-row tile in decode, several LM rows
    per prefill pass): prefixes of 1..40 tokens appended in one call, then
    three decode steps; every row against the float64 oracle."""
    shape = VOCAB_SHAPE
    arrays = make_weights(shape, seed=4, bf16=True)
    w64 = od.ModelWeights.from_arrays(shape, arrays)
    E = _engine(shape, arrays, bf16=True, pool_tokens=4096, max_seqs=40, max_batch=40,
                max_chunk=96)
    n_seq, n_steps = 33, 3
    lens = np.random.default_rng(5).integers(1, 41, n_seq)
    toks = [random_tokens(int(n) + n_steps, shape.vocab, seed=500 + i) for i, n in enumerate(lens)]
    seqs = [E.kv_alloc(0) for _ in range(n_seq)]
    first = torch.empty((n_seq, shape.vocab), dtype=torch.float32, device="cuda")
    E.kv_append_prefix_batch(seqs, [t[:n] for t, n in zip(toks, lens)], chunk_tokens=96,
                             last_logits=first)
    rows = [[r] for r in first.cpu().numpy()]
    logits = torch.empty((n_seq, shape.vocab), dtype=torch.float32, device="cuda")
    gtok = torch.empty(n_seq, dtype=torch.int32, device="cuda")
    for k in range(n_steps):
        step = np.array([t[n + k] for t, n in zip(toks, lens)], dtype=np.int32)
        E.decode_step(seqs, torch.from_numpy(step).cuda(), logits)
        E.sample(logits, gtok)
        got, g = logits.cpu().numpy(), gtok.cpu().numpy()
        np.testing.assert_array_equal(g, np.argmax(got, axis=1))
        for i in range(n_seq):
            rows[i].append(got[i])
    agreed = 0
    for i, n in enumerate(lens):
        ref = od.recompute_logits(w64, toks[i])[n - 1:]
        g = np.stack(rows[i])
        _rows_close(g, ref, BF16_TOL, ("vocab decoder", i))
        for r in range(ref.shape[0]):
            top2 = np.sort(ref[r])[-2:]
            if top2[1] - top2[0] > 4 * BF16_TOL * np.max(np.abs(ref[r])):
                assert int(np.argmax(g[r])) == int(od.greedy(ref[r])), (i, r)
                agreed += 1
    assert agreed > 0
    E.close()


# ---------------------------------------------------------------------------
# Decode at positions 65K-131K
# ---------------------------------------------------------------------------

LONG_MAX = 131072


def _stage_long(E, shape, lens, seed, k_std, bf16):
    """Stage sequences of the given lengths with seeded K/V in their pages;
    returns the ids and the oracle states holding the same cache."""
    dt = torch.bfloat16 if bf16 else torch.float32
    dec_states, seqs = [], []
    Hkv, Dh = shape.n_kv_heads, shape.head_dim
    for i, L in enumerate(lens):
        s = E.kv_alloc(0)
        E.kv_extend_uninit(s, int(L))
        pages = E.kv_block_table(s)
        npg = -(-int(L) // 16)
        idx = torch.from_numpy(pages[:npg].astype(np.int64)).cuda()
        st = {"k": [], "v": [], "len": int(L)}
        for layer in range(shape.n_layers):
            k, v = cached_kv(int(L), Hkv, Dh, seed=seed + 100 * i + layer, k_std=k_std, bf16=bf16)
            kp = np.zeros((npg * 16, Hkv, Dh), dtype=np.float32)
            vp = np.zeros((npg * 16, Hkv, Dh), dtype=np.float32)
            kp[:L], vp[:L] = k, v
            kp = kp.reshape(npg, 16, Hkv, Dh).transpose(0, 2, 1, 3)   # [page][g][slot][d]
            vp = vp.reshape(npg, 16, Hkv, Dh).transpose(0, 2, 3, 1)   # [page][g][d][slot]
            E.k_pages(layer)[idx] = torch.from_numpy(np.ascontiguousarray(kp)).cuda().to(dt)
            E.v_pages(layer)[idx] = torch.from_numpy(np.ascontiguousarray(vp)).cuda().to(dt)
            st["k"].append(k.astype(np.float64))
            st["v"].append(v.astype(np.float64))
        seqs.append(s)
        dec_states.append(st)
    torch.cuda.synchronize()
    return seqs, dec_states


def _read_kv(E, shape, seq, pos, layer):
    """K and V the GPU holds for one position, [Hkv][Dh] each (float64)."""
    pages = E.kv_block_table(seq)
    pg, slot = int(pages[pos // 16]), pos % 16
    k = E.k_pages(layer)[pg, :, slot, :].float().cpu().numpy().astype(np.float64)
    v = E.v_pages(layer)[pg, :, :, slot].float().cpu().numpy().astype(np.float64)
    return k, v


def _long_context_parity(shape, arrays, bf16, lens, q_gain, k_std, tol, seed):
    # Sharpen attention so that the result depends on which cached keys the
    # rotated query aligns with: q is scaled up and the cached keys have a
    # larger spread (score standard deviation about 2).
    arrays = {**arrays, "layers": [dict(lay) for lay in arrays["layers"]]}
    for lay in arrays["layers"]:
        wq = lay["wq"] * np.float32(q_gain)
        lay["wq"] = round_to_bf16(wq) if bf16 else wq
    w64 = od.ModelWeights.from_arrays(shape, arrays)
    dec = od.Decoder(w64)
    pool = int(sum(lens)) + 16 * (len(lens) + 4)
    E = _engine(shape, arrays, bf16, pool_tokens=pool, max_seqs=len(lens),
                max_seq_len=LONG_MAX, max_batch=len(lens), max_chunk=16)
    seqs, states = _stage_long(E, shape, lens, seed, k_std, bf16)
    logits = torch.empty((len(lens), shape.vocab), dtype=torch.float32, device="cuda")
    for step in range(2):
        tok = random_tokens(len(lens), shape.vocab, seed=seed + 7 + step)
        E.decode_step(seqs, torch.from_numpy(tok).cuda(), logits)
        got = logits.cpu().numpy()
        for i, st in enumerate(states):
            ref = dec.step(st, int(tok[i]))
            if tol < 1e-3:  # fp32: absolute bound
                err = float(np.max(np.abs(got[i] - ref)))
                assert err <= tol, ("fp32 logits", lens[i], step, err)
            else:
                _rows_close(got[i][None], ref[None], tol, ("bf16 logits", lens[i], step))
            # The KV the step wrote at its position (rotated k, and v).
            pos = int(lens[i]) + step
            for layer in range(shape.n_layers):
                k, v = _read_kv(E, shape, seqs[i], pos, layer)
                for g in range(shape.n_kv_heads):
                    for name, a, b in (("k", k[g], st["k"][layer][pos, g]),
                                       ("v", v[g], st["v"][layer][pos, g])):
                        err = float(np.max(np.abs(a - b)))
                        assert err <= 2 * tol * max(float(np.max(np.abs(b))), 1e-3), \
                            (name, lens[i], step, layer, g, err)
    E.close()


def test_long_positions_bf16():
    """bf16, head_dim 128 with GQA groups of 4: contexts of 131070 (the last
    two steps end at position 131071), 120001 (mid-page) and 65537 tokens."""
    shape = ModelShape(n_layers=1, d_model=256, n_q_heads=8, n_kv_heads=2, head_dim=128,
                       ffn_dim=256, vocab=512)
    arrays = make_weights(shape, seed=31, bf16=True)
    _long_context_parity(shape, arrays, True, [131070, 120001, 65537], q_gain=5.0, k_std=4.0,
                         tol=BF16_TOL, seed=3100)


def test_long_positions_fp32():
    """The 2-layer fp32 decoder (head_dim 64) at 131070 and 98304 + 5 tokens."""
    arrays = make_weights(TINY, seed=32)
    _long_context_parity(TINY, arrays, False, [131070, 98309], q_gain=5.0, k_std=4.0,
                         tol=F32_TOL, seed=3200)


# ---------------------------------------------------------------------------
# Multi-sequence append; departure and re-admission
# ---------------------------------------------------------------------------

def test_append_batch_equals_oracle_and_single_appends():
    """fp32 decoder: four prefixes (1, 37, 200 and 95 tokens) appended in one
    call with 64-row passes (so passes hold pieces of several sequences and a
    sequence spans passes), onto sequences that already hold a few tokens;
    last-position logits of all four, then a decode step, within 1e-4 of the
    oracle; the KV equals the per-sequence append's within the same bound."""
    arrays = make_weights(TINY, seed=33)
    w64 = od.ModelWeights.from_arrays(TINY, arrays)
    E = _engine(TINY, arrays, bf16=False, pool_tokens=4096, max_seq_len=512)
    heads = [random_tokens(n, TINY.vocab, seed=330 + i) for i, n in enumerate([3, 0, 16, 1])]
    tails = [random_tokens(n, TINY.vocab, seed=340 + i) for i, n in enumerate([1, 37, 200, 95])]
    nxt = random_tokens(4, TINY.vocab, seed=350)

    def run(batched):
        seqs = []
        for h in heads:
            s = E.kv_alloc(0)
            if len(h):
                E.kv_append_prefix(s, h, chunk_tokens=8)
            seqs.append(s)
        last = torch.empty((4, TINY.vocab), dtype=torch.float32, device="cuda")
        if batched:
            E.kv_append_prefix_batch(seqs, tails, chunk_tokens=64, last_logits=last)
        else:
            for i, (s, t) in enumerate(zip(seqs, tails)):
                E.kv_append_prefix(s, t, chunk_tokens=64, last_logits=last[i])
        step = torch.empty((4, TINY.vocab), dtype=torch.float32, device="cuda")
        E.decode_step(seqs, torch.from_numpy(nxt).cuda(), step)
        kv = []
        for s in seqs:
            n = E.kv_len(s)
            kv.append([_read_kv(E, TINY, s, p, layer) for p in (0, n // 2, n - 1)
                       for layer in range(TINY.n_layers)])
        out = (last.cpu().numpy(), step.cpu().numpy(), kv)
        for s in seqs:
            E.kv_free(s)
        return out

    last_b, step_b, kv_b = run(True)
    last_s, step_s, kv_s = run(False)
    for i in range(4):
        toks = np.concatenate([heads[i], tails[i], nxt[i:i + 1]])
        ref = od.recompute_logits(w64, toks)
        n = len(heads[i]) + len(tails[i])
        assert np.max(np.abs(last_b[i] - ref[n - 1])) <= F32_TOL
        assert np.max(np.abs(step_b[i] - ref[n])) <= F32_TOL
        assert np.max(np.abs(last_b[i] - last_s[i])) <= F32_TOL
        for (kb, vb), (ks, vs) in zip(kv_b[i], kv_s[i]):
            assert np.max(np.abs(kb - ks)) <= F32_TOL and np.max(np.abs(vb - vs)) <= F32_TOL
    E.close()


def test_append_batch_errors_are_atomic():
    P = _P()
    arrays = make_weights(TINY, seed=34)
    E = _engine(TINY, arrays, bf16=False, pool_tokens=64, max_seq_len=200)  # 4 pages
    a, b = E.kv_alloc(0), E.kv_alloc(0)
    E.kv_append_prefix(a, random_tokens(20, TINY.vocab, 1), chunk_tokens=16)
    head = E.kv_headroom()
    cases = [([a, b], [random_tokens(30, TINY.vocab, 2), random_tokens(30, TINY.vocab, 3)], -2),
             ([a, a], [random_tokens(2, TINY.vocab, 2), random_tokens(2, TINY.vocab, 3)], -1),
             ([a, b], [random_tokens(2, TINY.vocab, 2), np.zeros(0, np.int32)], -1),
             ([a, b], [random_tokens(2, TINY.vocab, 2), np.array([TINY.vocab], np.int32)], -1),
             ([a, b], [random_tokens(190, TINY.vocab, 2), random_tokens(2, TINY.vocab, 3)], -4)]
    for ids, toks, code in cases:
        with pytest.raises(P.PdecError) as ei:
            E.kv_append_prefix_batch(ids, toks, chunk_tokens=16)
        assert ei.value.code == code, (code, str(ei.value))
        assert E.kv_len(a) == 20 and E.kv_len(b) == 0 and E.kv_headroom() == head
    E.close()


def test_free_readmit_with_reserve_then_step():
    """A departure and two admissions before any block-table entry reaches the
    device: the freed slot's unflushed entries must not overwrite its next
    occupant's (both sequences then hold a page the other once held)."""
    arrays = make_weights(TINY, seed=35)
    w64 = od.ModelWeights.from_arrays(TINY, arrays)
    E = _engine(TINY, arrays, bf16=False, pool_tokens=8 * 16, max_seq_len=100)  # 8 pages
    a = E.kv_alloc(32)
    E.kv_free(a)
    b = E.kv_alloc(16)
    c = E.kv_alloc(16)
    tb, tc = random_tokens(40, TINY.vocab, 36), random_tokens(30, TINY.vocab, 37)
    E.kv_append_prefix(b, tb[:17], chunk_tokens=16)
    E.kv_append_prefix(c, tc[:20], chunk_tokens=16)
    assert not set(E.kv_block_table(b)) & set(E.kv_block_table(c))
    logits = torch.empty((2, TINY.vocab), dtype=torch.float32, device="cuda")
    for k in range(3):
        nxt = np.array([tb[17 + k], tc[20 + k]], dtype=np.int32)
        E.decode_step([b, c], torch.from_numpy(nxt).cuda(), logits)
    got = logits.cpu().numpy()
    assert np.max(np.abs(got[0] - od.recompute_logits(w64, tb[:20])[-1])) <= F32_TOL
    assert np.max(np.abs(got[1] - od.recompute_logits(w64, tc[:23])[-1])) <= F32_TOL
    E.close()
