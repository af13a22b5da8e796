"""Weight projections (out = x W^T) through the C ABI against a float64 matmul.

Covers every kernel the planner picks: the weight-streaming MFMA kernel (one
and two 16-row tiles), the 128-row and 256-row MFMA tiles, split-K, ragged M
and N (a zero-padded last group of the packed weight).  Inputs are
bf16-representable values, so the only difference from the float64 product
is fp32 accumulation: per row, max|gpu - ref| <= 1e-4 * max|ref|.
The packed layout itself is checked element by element against its
definition.
"""

import numpy as np
import pytest
import torch

from workload import round_to_bf16

pytestmark = pytest.mark.gpu

TOL = 1e-4


def _run(M, N, K, bf16=True, seed=0, rows=None):
    import paper_2609_36899_amd as P
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((M, K), dtype=np.float32)
    w = rng.standard_normal((N, K), dtype=np.float32) * np.float32(0.02)
    if bf16:
        x, w = round_to_bf16(x), round_to_bf16(w)
    td = torch.bfloat16 if bf16 else torch.float32
    xd = torch.from_numpy(x).cuda().to(td).contiguous()
    wd = P.pack_weight(torch.from_numpy(w).cuda().to(td).contiguous())
    out = torch.empty((M, N), dtype=torch.float32, device="cuda")
    P.weight_projection(xd, wd, out)
    got = out.cpu().numpy()
    rows = np.arange(M) if rows is None else np.asarray(rows)
    ref = x[rows].astype(np.float64) @ w.astype(np.float64).T
    for i, r in enumerate(rows):
        err = np.max(np.abs(got[r] - ref[i]))
        assert err <= TOL * np.max(np.abs(ref[i])), (M, N, K, r, err)


@pytest.mark.parametrize("M", [1, 2, 3, 4, 5, 8, 16, 17, 64, 100, 128, 129, 256, 300])
def test_bf16_ragged_shapes(M):
    _run(M, 1412, 576, seed=M)


@pytest.mark.parametrize("M", [1, 3, 4, 8, 64, 256, 512])
@pytest.mark.parametrize("N,K", [(6144, 4096), (4096, 14336)])
def test_bf16_8b_shapes_sampled_rows(M, N, K):
    rows = sorted(set([0, M - 1] + list(np.random.default_rng(M).integers(0, M, 6))))
    _run(M, N, K, seed=N + M, rows=rows)


@pytest.mark.parametrize("M", [257, 300, 520])
def test_bf16_wide_tiles(M):
    """256 x 256 tiles (two column groups per work group), taken above 256
    rows when their grid fills the GPU: N = 28736 is 225 groups, so the last
    work group's second group is clamped and writes nothing, the last group
    is half-filled, and 520 rows end in a partial third M-block."""
    rows = sorted(set([0, 1, M // 2, M - 2, M - 1]))
    _run(M, 28736, 320, seed=M, rows=rows)


@pytest.mark.parametrize("M", [1, 4, 33])
def test_f32(M):
    _run(M, 688, 256, bf16=False, seed=M)


@pytest.mark.parametrize("N,K", [(64, 64), (1412, 576), (40, 128), (256, 64)])
def test_pack_layout(N, K):
    """Element (n, k) sits at (((G*K/32 + b)*8 + s)*64 + q*16 + c)*8 + e with
    n = 128G + 16s + c, k = 32b + 8q + e; the columns of the padded last group
    are zero."""
    import paper_2609_36899_amd as P
    w = np.arange(N * K, dtype=np.int64).reshape(N, K) % 65521
    wd = torch.from_numpy(w.astype(np.int16)).cuda().view(torch.bfloat16)
    pw = P.pack_weight(wd.contiguous())
    torch.cuda.synchronize()
    got = pw.data.view(torch.int16).cpu().numpy().astype(np.int64) % 65536
    n_groups = (N + 127) // 128
    assert got.size == n_groups * 128 * K
    expect = np.zeros(n_groups * 128 * K, dtype=np.int64)
    for n in range(N):
        G, r = divmod(n, 128)
        s, c = divmod(r, 16)
        for k in range(K):
            b, r2 = divmod(k, 32)
            q, e = divmod(r2, 8)
            expect[(((G * (K // 32) + b) * 8 + s) * 64 + q * 16 + c) * 8 + e] = w[n, k] % 65536
    np.testing.assert_array_equal(got, expect)


def _swiglu_run(M, F, K, bf16=True, seed=0, rows=None):
    """u = silu(x Wg^T) * (x Wu^T) through swiglu_projection against the
    oracle's silu on float64 products of the same (bf16-representable)
    inputs.  bf16 u is rounded to nearest even: per row,
    max|gpu - ref| <= 2^-8 * max|ref| (half an ulp is 2^-9 of the element,
    fp32 accumulation adds < 1e-5); fp32 u: 1e-4 * max|ref|."""
    import paper_2609_36899_amd as P
    from oracle import decoder as od
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((M, K), dtype=np.float32) * np.float32(3.0)
    wg = rng.standard_normal((F, K), dtype=np.float32) * np.float32(0.02)
    wu = rng.standard_normal((F, K), dtype=np.float32) * np.float32(0.02)
    if bf16:
        x, wg, wu = round_to_bf16(x), round_to_bf16(wg), round_to_bf16(wu)
    td = torch.bfloat16 if bf16 else torch.float32
    xd = torch.from_numpy(x).cuda().to(td).contiguous()
    pg = P.pack_weight(torch.from_numpy(wg).cuda().to(td).contiguous())
    pu = P.pack_weight(torch.from_numpy(wu).cuda().to(td).contiguous())
    u = torch.full((M, F), float("nan"), dtype=td, device="cuda")
    P.swiglu_projection(xd, pg, pu, u)
    got = u.float().cpu().numpy()
    rows = np.arange(M) if rows is None else np.asarray(rows)
    x64 = x[rows].astype(np.float64)
    ref = od.silu(x64 @ wg.astype(np.float64).T) * (x64 @ wu.astype(np.float64).T)
    tol = 2.0 ** -8 if bf16 else 1e-4
    assert np.isfinite(got).all()
    for i, r in enumerate(rows):
        err = np.max(np.abs(got[r] - ref[i]))
        assert err <= tol * np.max(np.abs(ref[i])), (M, F, K, r, err)


@pytest.mark.parametrize("M", [1, 16, 17, 32, 33, 128, 129, 256, 300])
@pytest.mark.parametrize("F,K", [(8256, 320), (16320, 256)])
def test_swiglu_fused_epilogue(M, F, K):
    """Shapes whose bf16 plan has no K split: the SwiGLU runs in the GEMM's
    epilogue (streaming kernel up to 32 rows, 128- and 256-row tiles above,
    two M-blocks at 300 rows).  F = 8256 and 16320 end in a half-filled
    column group, whose empty half writes nothing."""
    import paper_2609_36899_amd as P
    from paper_2609_36899_amd import _native as N
    assert N.load().swiglu_projection_workspace_bytes(N.BF16, M, F, K) == 0
    _swiglu_run(M, F, K, seed=M + F)


@pytest.mark.parametrize("M", [1, 16, 32, 33, 128, 256])
@pytest.mark.parametrize("F,K", [(17408, 320), (16448, 256), (17400, 256)])
def test_swiglu_split_tail(M, F, K):
    """FFN widths whose fused grid would be whole rounds of 256 work groups
    plus a last round at most half full (272 and 258 half column-groups;
    17400 ends in a part-filled group): the columns of that last round take
    the split-K kernels and the SwiGLU pass (a workspace is needed), the
    others the fused epilogue, on the streaming kernel and both tiles."""
    from paper_2609_36899_amd import _native as N
    assert N.load().swiglu_projection_workspace_bytes(N.BF16, M, F, K) > 0
    _swiglu_run(M, F, K, seed=M + F + 1)


@pytest.mark.parametrize("M", [16, 128, 256])
def test_swiglu_14b_shape_split_tail_sampled_rows(M):
    """The 14B-shaped gate/up pair (F 17408, K 5120): 256 half-groups fused,
    the last 16 split 16 ways; rows sampled."""
    rows = sorted(set([0, M - 1] + list(np.random.default_rng(M).integers(0, M, 4))))
    _swiglu_run(M, 17408, 5120, seed=11 + M, rows=rows)


@pytest.mark.parametrize("M", [1, 16, 256, 512])
def test_swiglu_8b_shape_sampled_rows(M):
    """The 8B gate/up pair (F 14336, K 4096) as the decode step runs it: the
    streaming kernel, the 256 x 128 tile and the 256 x 256 tile, all with the
    SwiGLU epilogue; rows sampled."""
    rows = sorted(set([0, M - 1] + list(np.random.default_rng(M).integers(0, M, 4))))
    _swiglu_run(M, 14336, 4096, seed=7 + M, rows=rows)


@pytest.mark.parametrize("M", [4, 64])
def test_swiglu_split_k(M):
    """A narrow FFN (F = 256): the plan splits K, the partials go through the
    workspace and the separate SwiGLU kernel."""
    from paper_2609_36899_amd import _native as N
    assert N.load().swiglu_projection_workspace_bytes(N.BF16, M, 256, 512) > 0
    _swiglu_run(M, 256, 512, seed=M)


def test_swiglu_f32():
    _swiglu_run(4, 688, 256, bf16=False, seed=9)
