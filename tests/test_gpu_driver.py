"""Headroom-paced rollout through the C ABI on a pool too small for the
whole batch: trajectories are evicted (KV snapshot to host, or dropped for
re-prefill) and placed back, and every logits row they produce must match
the float64 oracle's recomputation of the same token stream (tiny fp32
decoder, 1e-4 absolute), whatever was evicted in between.
"""

import numpy as np
import pytest
import torch

from oracle import decoder as od
from workload import TINY, make_weights, random_tokens

pytestmark = pytest.mark.gpu

PROMPTS = [20, 40, 70, 33, 90, 12]
DECODE = 40


@pytest.mark.parametrize("restore", ["snapshot", "reprefill"])
def test_paced_rollout_matches_oracle(restore):
    import paper_2609_36899_amd as P
    arrays = make_weights(TINY, seed=4)
    w = P.weights_to_device(arrays, P.F32)
    per_tok = P.kv_bytes_per_token(TINY, P.F32)
    # 20 pages (320 tokens) for six trajectories that end at 505 tokens in all
    E = P.Engine(TINY, w, P.F32, 20 * 16 * per_tok, max_seqs=8, max_seq_len=256, max_batch=4,
                 max_chunk=64)
    drv = P.PacedRollout(E, h_min=4 * 16, delta=16, restore=restore, chunk_tokens=32)
    streams = {}
    for i, n in enumerate(PROMPTS):
        streams[i] = random_tokens(n + DECODE, TINY.vocab, seed=300 + i)
        drv.add(i, streams[i], prompt_len=n)
    got = {i: {} for i in streams}
    for _ in range(2000):
        if drv.finished:
            break
        for tid, (pos, row) in drv.step().items():
            got[tid][pos] = row.cpu().numpy().copy()
    assert drv.finished, "pacing made no progress"
    assert drv.stats["evictions"] > 0
    if restore == "snapshot":
        assert drv.stats["restores"] > 0
    w64 = od.ModelWeights.from_arrays(TINY, arrays)
    for i, n in enumerate(PROMPTS):
        ref = od.recompute_logits(w64, streams[i])
        assert sorted(got[i]) == list(range(n, n + DECODE))
        for pos, row in got[i].items():
            err = np.max(np.abs(row - ref[pos]))
            assert err <= 1e-4, (restore, i, pos, err)
    E.close()
