"""sample_top_p_noalloc (the entry point that allocates nothing; its scratch is
a static device array) against sample_top_p with a caller workspace, through
the C ABI: the tokens must be the same, bit for bit, on two calls in a row,
the second with a smaller input, so that the second call runs over the
first one's leftover scratch contents.  A batch above the split form's
32 rows (no scratch) and the argument errors are checked too."""

import ctypes

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def _lib():
    from paper_2609_36899_amd import _native as N
    return N, N.load()


def _inputs(batch, vocab, seed):
    rng = np.random.default_rng(seed)
    z = (rng.standard_normal((batch, vocab)) * 2).astype(np.float32)
    z = np.round(z * 8) / 8  # many ties
    u = rng.random(batch).astype(np.float32)
    return torch.from_numpy(z).cuda(), torch.from_numpy(u).cuda()


def _with_workspace(z, u, temperature, top_p):
    N, lib = _lib()
    B, V = z.shape
    need = lib.sample_top_p_workspace_bytes(B)
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device="cuda")
    out = torch.full((B,), -1, dtype=torch.int32, device="cuda")
    N.check(lib.sample_top_p(B, V, z.data_ptr(), temperature, top_p, u.data_ptr(),
                             out.data_ptr(), ws.data_ptr() if need else None, need, None))
    return out


def _noalloc(z, u, temperature, top_p):
    N, lib = _lib()
    B, V = z.shape
    out = torch.full((B,), -1, dtype=torch.int32, device="cuda")
    N.check(lib.sample_top_p_noalloc(B, V, z.data_ptr(), temperature, top_p, u.data_ptr(),
                                     out.data_ptr(), None))
    return out


@pytest.mark.parametrize("first,second", [((32, 128256), (5, 50000)),
                                          ((16, 128256), (1, 4096)),
                                          ((64, 32000), (9, 128256))])
def test_noalloc_matches_workspace_form_on_two_calls(first, second):
    for (B, V), seed, (t, p) in ((first, 1, (0.8, 0.9)), (second, 2, (1.2, 0.6))):
        z, u = _inputs(B, V, seed + B)
        want = _with_workspace(z, u, t, p)
        got = _noalloc(z, u, t, p)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(got.cpu().numpy(), want.cpu().numpy())
        assert (got.cpu().numpy() >= 0).all() and (got.cpu().numpy() < V).all()


def test_noalloc_argument_errors():
    N, lib = _lib()
    z, u = _inputs(2, 100, 3)
    out = torch.empty(2, dtype=torch.int32, device="cuda")
    for args in ((0, 100, z.data_ptr(), 1.0, 0.9, u.data_ptr(), out.data_ptr(), None),
                 (2, 100, z.data_ptr(), 0.0, 0.9, u.data_ptr(), out.data_ptr(), None),
                 (2, 100, z.data_ptr(), 1.0, 1.5, u.data_ptr(), out.data_ptr(), None),
                 (2, 100, None, 1.0, 0.9, u.data_ptr(), out.data_ptr(), None)):
        with pytest.raises(N.PdecError) as ei:
            N.check(lib.sample_top_p_noalloc(*args))
        assert ei.value.code == N.INVALID_ARG
