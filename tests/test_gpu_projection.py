"""Weight projections (out = x W^T) through the C ABI against a float64 matmul.

Covers every kernel the planner picks: the VALU GEMV (M <= 4 with small
activations), the register-ring MFMA kernel (M <= 4 with long K), the 128-row
and 256-row MFMA tiles, split-K and ragged M, N.  Inputs are bf16-representable
values, so the only difference from the float64 product is fp32 accumulation:
per row, max|gpu - ref| <= 1e-4 * max|ref|.
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
    wd = torch.from_numpy(w).cuda().to(td).contiguous()
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


@pytest.mark.parametrize("M", [1, 4, 33])
def test_f32(M):
    _run(M, 688, 256, bf16=False, seed=M)
