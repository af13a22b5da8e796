"""Temperature / top-p sampling through the C ABI against the oracle.

After one float64 exponential per logit every decision of the rule is
integer arithmetic on both sides, so the sampled tokens must agree exactly:
random logits at several vocabulary sizes (ragged, below and above one
element per thread, the 8B vocabulary), heavy ties that put the nucleus
boundary inside a tie group, masked (-inf) entries, exact u boundaries, and
stratified frequencies over one batch.  Small batches run the split form
(several work groups per row, partial results in a workspace); it must give
the one-group form's tokens bit for bit, and both the oracle's.  Argument
errors are checked too.
"""

import numpy as np
import pytest
import torch

from oracle.sampling import sample_top_p as oracle_sample

pytestmark = pytest.mark.gpu


def _gpu(z, temperature, top_p, u, split=True):
    import paper_2609_36899_amd as P
    zd = torch.from_numpy(np.ascontiguousarray(z, dtype=np.float32)).cuda()
    ud = torch.from_numpy(np.asarray(u, dtype=np.float32)).cuda()
    out = torch.full((z.shape[0],), -1, dtype=torch.int32, device="cuda")
    P.sample_top_p(zd, out, temperature, top_p, ud, split=split)
    return out.cpu().numpy()


def _check(z, temperature, top_p, u):
    got = _gpu(z, temperature, top_p, u)
    want = np.array([oracle_sample(z[b], temperature, top_p, u[b]) for b in range(z.shape[0])])
    np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("vocab", [5, 1000, 4096, 128256])
@pytest.mark.parametrize("temperature,top_p", [(1.0, 1.0), (0.7, 0.9), (1.3, 0.5), (0.6, 1e-6)])
def test_random_logits(vocab, temperature, top_p):
    rng = np.random.default_rng(vocab + int(100 * temperature))
    z = (rng.standard_normal((6, vocab)) * 3.0).astype(np.float32)
    u = rng.random(6).astype(np.float32)
    _check(z, temperature, top_p, u)


def test_ties_masks_and_boundaries():
    rng = np.random.default_rng(11)
    z = rng.integers(0, 4, size=(8, 3000)).astype(np.float32)  # many exact ties
    z[1, ::3] = -np.inf                                          # masked vocabulary
    z[2] = 0.0                                                   # all equal
    u = rng.random(8).astype(np.float32)
    u[2] = 0.5
    for top_p in (1.0, 0.3, 0.7):
        _check(z, 1.0, top_p, u)
    zeros = np.zeros((4, 4), np.float32)
    np.testing.assert_array_equal(_gpu(zeros, 1.0, 1.0, [0.0, 0.25, 0.5, 0.75]), [0, 1, 2, 3])


def test_stratified_frequencies_in_one_batch():
    n, vocab = 2000, 40
    z0 = (np.random.default_rng(3).standard_normal(vocab) * 2.0).astype(np.float32)
    z = np.repeat(z0[None], n, axis=0)
    u = ((np.arange(n) + 0.5) / n).astype(np.float32)
    got = _gpu(z, 0.8, 1.0, u)
    p = np.exp((z0.astype(np.float64) - z0.max()) / np.float32(0.8))
    p /= p.sum()
    counts = np.bincount(got, minlength=vocab)
    assert np.all(np.abs(counts - n * p) <= 1.0 + 1e-6)
    again = _gpu(z, 0.8, 1.0, u)
    np.testing.assert_array_equal(got, again)


@pytest.mark.parametrize("batch,vocab", [(1, 128256), (3, 128255), (16, 128256), (24, 50001),
                                         (32, 7), (20, 4099)])
def test_split_form_matches_one_group_and_oracle(batch, vocab):
    import paper_2609_36899_amd as P
    rng = np.random.default_rng(batch * 7 + vocab)
    z = (rng.standard_normal((batch, vocab)) * 3.0).astype(np.float32)
    z[0, : vocab // 2] = np.round(z[0, : vocab // 2])   # ties spread over chunks
    if batch > 1:
        z[1, ::5] = -np.inf
    u = rng.random(batch).astype(np.float32)
    assert P.sample_top_p_workspace_bytes(batch) > 0
    for temperature, top_p in ((1.0, 1.0), (0.8, 0.95), (1.2, 0.3)):
        split = _gpu(z, temperature, top_p, u, split=True)
        one = _gpu(z, temperature, top_p, u, split=False)
        np.testing.assert_array_equal(split, one)
        rows = range(batch) if batch * vocab <= 400_000 else (0, batch - 1)
        want = [oracle_sample(z[b], temperature, top_p, u[b]) for b in rows]
        np.testing.assert_array_equal(split[list(rows)], want)


def test_split_form_tie_nucleus_across_chunks():
    # One row of equal logits: the nucleus boundary falls inside one tie
    # group that spans every chunk, so the member ties are ranked across
    # chunks in index order.
    z = np.zeros((2, 10000), np.float32)
    z[1, 5000:] = 1.0
    u = np.array([0.37, 0.999], np.float32)
    for top_p in (0.25, 0.5, 0.61, 1.0):
        _check(z, 1.0, top_p, u)
        np.testing.assert_array_equal(_gpu(z, 1.0, top_p, u, split=False),
                                      _gpu(z, 1.0, top_p, u, split=True))


def test_split_form_reused_workspace_and_no_split_above_32_rows():
    import paper_2609_36899_amd as P
    assert P.sample_top_p_workspace_bytes(33) == 0
    assert P.sample_top_p_workspace_bytes(512) == 0
    need = P.sample_top_p_workspace_bytes(4)
    ws = torch.full((need,), 0xAB, dtype=torch.uint8, device="cuda")
    rng = np.random.default_rng(5)
    for vocab in (128256, 1000):  # the second call sees the first one's contents
        z = (rng.standard_normal((4, vocab)) * 2.0).astype(np.float32)
        u = rng.random(4).astype(np.float32)
        zd = torch.from_numpy(z).cuda()
        ud = torch.from_numpy(u).cuda()
        out = torch.full((4,), -1, dtype=torch.int32, device="cuda")
        P.sample_top_p(zd, out, 0.9, 0.9, ud, workspace=ws)
        want = [oracle_sample(z[b], 0.9, 0.9, u[b]) for b in range(4)]
        np.testing.assert_array_equal(out.cpu().numpy(), want)


def test_argument_errors():
    import paper_2609_36899_amd as P
    from paper_2609_36899_amd import _native as N
    z = torch.zeros((2, 16), dtype=torch.float32, device="cuda")
    u = torch.zeros(2, dtype=torch.float32, device="cuda")
    out = torch.zeros(2, dtype=torch.int32, device="cuda")
    for t, p in ((0.0, 1.0), (float("inf"), 1.0), (1.0, 0.0), (1.0, 1.5)):
        with pytest.raises(P.PdecError) as ei:
            P.sample_top_p(z, out, t, p, u)
        assert ei.value.code == N.INVALID_ARG
    lib = N.load()
    assert lib.sample_top_p(0, 16, z.data_ptr(), 1.0, 1.0, u.data_ptr(), out.data_ptr(),
                            None, 0, None) == N.INVALID_ARG
    assert lib.sample_top_p(2, 16, None, 1.0, 1.0, u.data_ptr(), out.data_ptr(),
                            None, 0, None) == N.INVALID_ARG
    need = lib.sample_top_p_workspace_bytes(2)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    assert lib.sample_top_p(2, 16, z.data_ptr(), 1.0, 1.0, u.data_ptr(), out.data_ptr(),
                            ws.data_ptr(), need - 1, None) == N.INVALID_ARG
    assert lib.sample_top_p(2, 16, z.data_ptr(), 1.0, 1.0, u.data_ptr(), out.data_ptr(),
                            ws.data_ptr(), 0, None) == N.INVALID_ARG
    assert lib.sample_top_p_workspace_bytes(0) == N.INVALID_ARG
