"""A seeded random lifecycle on the GPU against the float64 oracle.

Trajectories are admitted (with and without reserves), appended to (one
sequence or several in one batched call, random chunk sizes), decoded in
random subsets, moved by snapshot/restore into a fresh sequence, and
departed, in a 30-page pool, so that freed pages and sequence slots are
reused many times over.  Operations that do not fit the pool must fail with
OUT_OF_PAGES and leave every trajectory as it was; a departed trajectory's id
must be refused afterwards.  Every logits row the engine returns is compared
with the oracle's recompute over that trajectory's whole token history: the
tiny fp32 decoder within 1e-4, and a bf16 decoder with 128-dim heads (GQA
groups of 4: the LDS-staged prefill kernel) within the bf16 bars of the other
parity tests, 2e-2 of max|logit| with bf16 pages and 6e-2 with E4M3 pages.
This drives the host bookkeeping (free list, slot reuse, pending block-table
entries, work lists, undo on failure) and the kernels together.
"""

import numpy as np
import pytest
import torch

from oracle import decoder as od
from workload import TINY, ModelShape, make_weights

pytestmark = pytest.mark.gpu

MAX_SEQS = 6
MAX_SEQ_LEN = 512
# One layer, d 256, 8 query heads and 2 KV heads of 128 dims.
BF16_G4 = ModelShape(n_layers=1, d_model=256, n_q_heads=8, n_kv_heads=2, head_dim=128,
                     ffn_dim=256, vocab=512)


@pytest.mark.parametrize("case", ["fp32", "bf16", "bf16-fp8kv", "bf16-wide"])
def test_random_lifecycle_matches_oracle(case, monkeypatch):
    """bf16-wide: every prefill pass takes 256-row blocks (eight-wave kernel)."""
    import paper_2609_36899_amd as P
    from paper_2609_36899_amd import _native as N

    if case == "bf16-wide":
        monkeypatch.setenv("PDEC_PREFILL_WIDE_PAGES", "0")
    bf16 = case != "fp32"
    shape = BF16_G4 if bf16 else TINY
    kv_fp8 = (0.5, 0.25) if case == "bf16-fp8kv" else None
    dt = P.BF16 if bf16 else P.F32
    # fp32: absolute; bf16: relative to max|ref| per row
    tol = {"fp32": 1e-4, "bf16": 2e-2, "bf16-fp8kv": 6e-2, "bf16-wide": 2e-2}[case]
    rng = np.random.default_rng(2024)
    arrays = make_weights(shape, seed=30, bf16=bf16)
    w64 = od.ModelWeights.from_arrays(shape, arrays)
    per_tok = P.kv_bytes_per_token(shape, dt, kv_fp8)
    E = P.Engine(shape, P.weights_to_device(arrays, dt), dt, 480 * per_tok,
                 max_seqs=MAX_SEQS, max_seq_len=MAX_SEQ_LEN, max_batch=MAX_SEQS, max_chunk=48,
                 kv_fp8=kv_fp8)
    hist = {}  # live sequence id -> its token history
    buf = torch.empty((MAX_SEQS, shape.vocab), dtype=torch.float32, device="cuda")
    counts = dict(checks=0, out_of_pages=0, moves=0, departures=0)

    def draw(n):
        return [int(x) for x in rng.integers(0, shape.vocab, n)]

    def check(seq, row):
        ref = od.recompute_logits(w64, hist[seq], kv_fp8=kv_fp8)[-1]
        err = float(np.max(np.abs(row - ref)))
        bound = tol * (float(np.max(np.abs(ref))) if bf16 else 1.0)
        assert np.isfinite(row).all() and err <= bound, (seq, len(hist[seq]), err, bound)
        counts["checks"] += 1

    def lens_unchanged():
        for s, h in hist.items():
            assert E.kv_len(s) == len(h), (s, E.kv_len(s), len(h))

    def out_of_pages(e):
        assert e.code == N.OUT_OF_PAGES, e
        counts["out_of_pages"] += 1
        lens_unchanged()

    def room(s, n):
        return len(hist[s]) + n <= MAX_SEQ_LEN

    for _ in range(150):
        live = list(hist)
        op = rng.choice(["admit", "admit", "append", "append", "batch", "decode", "decode",
                         "decode", "free", "move"])
        if op == "admit" and len(live) < MAX_SEQS:
            try:
                s = E.kv_alloc(int(rng.choice([0, 16, 100])))
            except N.PdecError as e:
                out_of_pages(e)
                continue
            hist[s] = []
            toks = draw(int(rng.integers(1, 80)))
            try:
                E.kv_append_prefix(s, toks, chunk_tokens=int(rng.choice([7, 16, 48])),
                                   last_logits=buf[0])
            except N.PdecError as e:
                out_of_pages(e)
                E.kv_free(s)
                del hist[s]
                continue
            hist[s] = toks
            check(s, buf[0].cpu().numpy())
        elif op == "append" and live:
            s = int(rng.choice(live))
            toks = draw(int(rng.integers(1, 60)))
            if not room(s, len(toks)):
                continue
            try:
                E.kv_append_prefix(s, toks, chunk_tokens=int(rng.choice([5, 16, 48])),
                                   last_logits=buf[0])
            except N.PdecError as e:
                out_of_pages(e)
                continue
            hist[s] += toks
            check(s, buf[0].cpu().numpy())
        elif op == "batch" and live:
            pick = [int(x) for x in rng.permutation(live)[:int(rng.integers(1, len(live) + 1))]]
            parts = [draw(int(rng.integers(1, 30))) for _ in pick]
            if not all(room(s, len(t)) for s, t in zip(pick, parts)):
                continue
            try:
                E.kv_append_prefix_batch(pick, parts, chunk_tokens=int(rng.choice([8, 32, 48])),
                                         last_logits=buf)
            except N.PdecError as e:
                out_of_pages(e)
                continue
            got = buf.cpu().numpy()
            for i, (s, t) in enumerate(zip(pick, parts)):
                hist[s] += t
                check(s, got[i])
        elif op == "decode" and live:
            pick = [int(x) for x in rng.permutation(live)[:int(rng.integers(1, len(live) + 1))]]
            pick = [s for s in pick if room(s, 1)]
            if not pick:
                continue
            nxt = draw(len(pick))
            try:
                E.decode_step(pick, torch.tensor(nxt, dtype=torch.int32, device="cuda"), buf)
            except N.PdecError as e:
                out_of_pages(e)
                continue
            got = buf.cpu().numpy()
            for i, (s, t) in enumerate(zip(pick, nxt)):
                hist[s].append(t)
                check(s, got[i])
        elif op == "free" and live:
            s = int(rng.choice(live))
            E.kv_free(s)
            del hist[s]
            counts["departures"] += 1
            with pytest.raises(N.PdecError) as stale:
                E.kv_len(s)
            assert stale.value.code == N.BAD_SEQ
            lens_unchanged()
        elif op == "move" and live:
            s = int(rng.choice(live))
            n = len(hist[s])
            snap = torch.empty(E.kv_snapshot_bytes(n), dtype=torch.uint8).pin_memory()
            assert E.kv_export(s, snap) == n
            torch.cuda.synchronize()
            E.kv_free(s)
            t = E.kv_alloc(0)
            E.kv_import(t, snap, n)
            hist[t] = hist.pop(s)
            counts["moves"] += 1
            lens_unchanged()
    E.close()
    # The schedule must have exercised what the test is for.
    assert counts["checks"] >= 100, counts
    assert counts["out_of_pages"] >= 3 and counts["moves"] >= 3 and counts["departures"] >= 3, counts
