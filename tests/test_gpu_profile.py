"""Sampled launch timing (engine_profile / engine_profile_every) on the tiny
bf16 decoder: the count of timed launches follows the sampling rule, and
timing does not change the logits."""

import numpy as np
import pytest
import torch

from workload import SMALL_BF16, make_weights, random_tokens

pytestmark = pytest.mark.gpu


def _engine(arrays):
    import paper_2609_36899_amd as P
    w = P.weights_to_device(arrays, P.BF16)
    per_tok = P.kv_bytes_per_token(SMALL_BF16, P.BF16)
    return P, P.Engine(SMALL_BF16, w, P.BF16, 2048 * per_tok, 4, 512, 4, 64)


def _steps(E, seqs, n, vocab):
    toks = torch.tensor([1, 2, 3], dtype=torch.int32, device="cuda")
    logits = torch.empty((len(seqs), vocab), dtype=torch.float32, device="cuda")
    rows = []
    for _ in range(n):
        E.decode_step(seqs, toks, logits)
        rows.append(logits.cpu().numpy().copy())
    return rows


@pytest.mark.parametrize("every", [1, 3, 7])
def test_timed_launch_count_and_identical_logits(every):
    arrays = make_weights(SMALL_BF16, seed=3)
    P, E = _engine(arrays)
    seqs = [E.kv_alloc(0) for _ in range(3)]
    for i, s in enumerate(seqs):
        E.kv_append_prefix(s, random_tokens(20 + 7 * i, SMALL_BF16.vocab, seed=i), 64)
    n_steps = 5
    ref = _steps(E, seqs, n_steps, SMALL_BF16.vocab)
    # the same trajectories again from the same prefixes, now timed
    P2, E2 = _engine(arrays)
    seqs2 = [E2.kv_alloc(0) for _ in range(3)]
    for i, s in enumerate(seqs2):
        E2.kv_append_prefix(s, random_tokens(20 + 7 * i, SMALL_BF16.vocab, seed=i), 64)
    from paper_2609_36899_amd import _native as N
    E2.profile([N.TIMER_ATTENTION, N.TIMER_GEMM], every=every)
    got = _steps(E2, seqs2, n_steps, SMALL_BF16.vocab)
    E2.profile([])
    torch.cuda.synchronize()
    attn_ms, attn_n = E2.profile_read(N.TIMER_ATTENTION)
    gemm_ms, gemm_n = E2.profile_read(N.TIMER_GEMM)
    launches = n_steps * SMALL_BF16.n_layers
    assert attn_n == -(-launches // every)
    assert gemm_n == -(-4 * launches // every)
    assert attn_ms > 0 and gemm_ms > 0
    assert E2.profile_read(N.TIMER_ATTENTION) == (0.0, 0)  # records were cleared
    for a, b in zip(ref, got):
        np.testing.assert_array_equal(a, b)


def test_every_must_be_positive():
    import paper_2609_36899_amd as P
    from paper_2609_36899_amd import _native as N
    arrays = make_weights(SMALL_BF16, seed=3)
    _, E = _engine(arrays)
    assert E.lib.engine_profile_every(E.handle, 0) == N.INVALID_ARG
