"""Paged decode attention over fp8 (E4M3) KV pages against the oracle.

Inputs are codes built from their bit fields (workload), so both sides read
exactly the same values: the oracle decodes them from the E4M3 definition and
applies the plain attention definition in float64; the GPU decodes them in
registers and runs the bf16 MFMA path.  Tolerance as for bf16 pages: per
(sequence, head) row, max|gpu - ref| <= 2e-2 * max|ref|.  Slots past each
length hold the NaN code, so a read beyond the sequence would show.
"""

import numpy as np
import pytest
import torch

import oracle
from workload import paged_attention_case_fp8

pytestmark = pytest.mark.gpu

TOL = 2e-2
EDGE_LENS = [1, 2, 15, 16, 17, 31, 32, 33, 48, 127, 128, 129, 300, 1000, 2049]


def _run(case, k_scale, v_scale):
    import paper_2609_36899_amd as P
    q = torch.from_numpy(case.q).cuda().to(torch.bfloat16).contiguous()
    k = torch.from_numpy(case.k_codes).cuda().contiguous()
    v = torch.from_numpy(np.ascontiguousarray(case.v_codes.transpose(0, 1, 3, 2))).cuda()
    bt = torch.from_numpy(case.block_table).cuda()
    out = torch.empty(q.shape, dtype=torch.float32, device="cuda")
    P.paged_decode_attention_fp8(q, k, v.contiguous(), k_scale, v_scale, bt, case.lens, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def _check(case, k_scale, v_scale):
    got = _run(case, k_scale, v_scale)
    ref = oracle.paged_decode_attention_fp8(case.q, case.k_codes, case.v_codes, k_scale,
                                            v_scale, case.block_table, case.lens)
    assert np.isfinite(got).all()
    for b in range(ref.shape[0]):
        for h in range(ref.shape[1]):
            err = np.max(np.abs(got[b, h] - ref[b, h]))
            assert err <= TOL * np.max(np.abs(ref[b, h])), (b, h, err)


@pytest.mark.parametrize("hq,hkv,dh", [(32, 8, 128), (8, 2, 128), (16, 1, 64), (40, 8, 128)])
def test_edge_lengths(hq, hkv, dh):
    lens = np.array(EDGE_LENS)
    case = paged_attention_case_fp8(len(lens), hq, hkv, dh, lens, n_pool_pages=700, seed=21)
    _check(case, 0.5, 1.0)


def test_every_finite_code_and_scales():
    """All 254 finite codes (subnormals, +-448) through the hardware decode."""
    lens = np.array([64, 200, 513])
    case = paged_attention_case_fp8(3, 8, 2, 128, lens, n_pool_pages=64, seed=22, all_codes=True)
    _check(case, 1.0 / 256, 0.25)  # small K scale keeps scores of +-448 codes moderate


def test_long_contexts_split_over_many_items():
    lens = np.array([70000, 5000, 33])
    case = paged_attention_case_fp8(3, 32, 8, 128, lens, n_pool_pages=4700, seed=23)
    _check(case, 0.75, 1.5)
