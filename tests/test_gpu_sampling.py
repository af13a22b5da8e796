"""Temperature / top-p sampling through the C ABI against the oracle.

After one float64 exponential per logit every decision of the rule is
integer arithmetic on both sides, so the sampled tokens must agree exactly:
random logits at several vocabulary sizes (ragged, below and above one
element per thread, the 8B vocabulary), heavy ties that put the nucleus
boundary inside a tie group, masked (-inf) entries, exact u boundaries, and
stratified frequencies over one batch.  Argument errors are checked too.
"""

import numpy as np
import pytest
import torch

from oracle.sampling import sample_top_p as oracle_sample

pytestmark = pytest.mark.gpu


def _gpu(z, temperature, top_p, u):
    import paper_2609_36899_amd as P
    zd = torch.from_numpy(np.ascontiguousarray(z, dtype=np.float32)).cuda()
    ud = torch.from_numpy(np.asarray(u, dtype=np.float32)).cuda()
    out = torch.full((z.shape[0],), -1, dtype=torch.int32, device="cuda")
    P.sample_top_p(zd, out, temperature, top_p, ud)
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
                            None) == N.INVALID_ARG
    assert lib.sample_top_p(2, 16, None, 1.0, 1.0, u.data_ptr(), out.data_ptr(),
                            None) == N.INVALID_ARG
