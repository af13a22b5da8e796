"""Paged split-K decode attention on the GPU against the float64 oracle.

All calls go through the C ABI (paged_decode_attention).  Tolerances:
bf16 inputs with fp32 accumulation, normwise per (sequence, head) row,
max|gpu - ref| <= 2e-2 * max|ref|; fp32, max|gpu - ref| <= 1e-4.
"""

import numpy as np
import pytest
import torch

import oracle
from workload import (PAGE_TOKENS, lazy_paged_attention_case, lengths_uniform,
                      paged_attention_case)

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2
F32_TOL = 1e-4


def _pdec():
    import paper_2609_36899_amd as P
    return P


def _upload(case, dtype):
    td = torch.bfloat16 if dtype == "bf16" else torch.float32
    q = torch.from_numpy(case.q).cuda().to(td).contiguous()
    k = torch.from_numpy(case.k_pool).cuda().to(td).contiguous()
    v = torch.from_numpy(np.ascontiguousarray(case.v_pool.transpose(0, 1, 3, 2))).cuda().to(td)
    bt = torch.from_numpy(case.block_table).cuda()
    return q, k, v.contiguous(), bt


def _run(case, dtype):
    P = _pdec()
    q, k, v, bt = _upload(case, dtype)
    out = torch.empty(q.shape, dtype=torch.float32, device="cuda")
    P.paged_decode_attention(q, k, v, bt, case.lens, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def _check_rows(got, ref, tol, normwise):
    assert np.isfinite(got).all()
    for b in range(ref.shape[0]):
        for h in range(ref.shape[1]):
            err = np.max(np.abs(got[b, h] - ref[b, h]))
            bound = tol * np.max(np.abs(ref[b, h])) if normwise else tol
            assert err <= bound, (b, h, err, bound)


EDGE_LENS = [1, 2, 15, 16, 17, 31, 32, 33, 48, 127, 128, 129, 300, 1000, 2049]


@pytest.mark.parametrize("hq,hkv,dh", [(32, 8, 128), (8, 2, 128), (16, 16, 128), (16, 1, 64),
                                        (40, 8, 128), (6, 2, 64)])
def test_bf16_edge_lengths(hq, hkv, dh):
    lens = np.array(EDGE_LENS)
    case = paged_attention_case(len(lens), hq, hkv, dh, lens, n_pool_pages=700, seed=1)
    got = _run(case, "bf16")
    ref = oracle.paged_decode_attention(case.q, case.k_pool, case.v_pool, case.block_table,
                                        case.lens)
    _check_rows(got, ref, BF16_TOL, normwise=True)


@pytest.mark.parametrize("hq,hkv,dh", [(4, 2, 64), (32, 8, 128), (15, 3, 128)])
def test_f32_edge_lengths(hq, hkv, dh):
    lens = np.array(EDGE_LENS[:12])
    case = paged_attention_case(len(lens), hq, hkv, dh, lens, n_pool_pages=120, seed=2,
                                bf16=False)
    got = _run(case, "f32")
    ref = oracle.paged_decode_attention(case.q, case.k_pool, case.v_pool, case.block_table,
                                        case.lens)
    _check_rows(got, ref, F32_TOL, normwise=False)


def test_bf16_config2_shape_small_batch():
    """Config-2 head geometry and length range on a batch of 6."""
    lens = lengths_uniform(6, 1024, 8192, seed=3)
    case = paged_attention_case(6, 32, 8, 128, lens, n_pool_pages=3500, seed=4)
    got = _run(case, "bf16")
    ref = oracle.paged_decode_attention(case.q, case.k_pool, case.v_pool, case.block_table,
                                        case.lens)
    _check_rows(got, ref, BF16_TOL, normwise=True)


@pytest.mark.parametrize("lens", [[2048], [2049, 100], [4096, 17], [4097], [25600, 5, 2049]])
def test_bf16_combine_wave_counts(lens):
    """Query blocks with 16 / 17 / 32 / 33 / 200 items of 8 pages (the
    combine's work group grows from 4 to 8 to 16 waves at those counts; 200
    items take several rounds)."""
    lens = np.array(lens)
    case = paged_attention_case(len(lens), 32, 8, 128, lens, n_pool_pages=2000, seed=11)
    got = _run(case, "bf16")
    ref = oracle.paged_decode_attention(case.q, case.k_pool, case.v_pool, case.block_table,
                                        case.lens)
    _check_rows(got, ref, BF16_TOL, normwise=True)


def test_page_permutation_is_bitwise_invariant():
    lens = np.array([5, 16, 17, 700, 1500, 33])
    case = paged_attention_case(len(lens), 32, 8, 128, lens, n_pool_pages=400, seed=5)
    a = _run(case, "bf16")
    # Move every page to a new physical slot; logical content is unchanged.
    perm = np.random.default_rng(9).permutation(case.k_pool.shape[0])
    inv = np.empty_like(perm)
    inv[perm] = np.arange(len(perm))
    case.k_pool = case.k_pool[perm]
    case.v_pool = case.v_pool[perm]
    case.block_table = np.where(case.block_table >= 0, inv[np.maximum(case.block_table, 0)], -1)
    case.block_table = case.block_table.astype(np.int32)
    b = _run(case, "bf16")
    np.testing.assert_array_equal(a, b)


def test_batch_permutation_is_bitwise_invariant():
    lens = np.array([3, 64, 65, 900, 2000, 31, 4096])
    case = paged_attention_case(len(lens), 32, 8, 128, lens, n_pool_pages=600, seed=6)
    a = _run(case, "bf16")
    order = np.array([4, 0, 6, 2, 1, 5, 3])
    case.q = case.q[order]
    case.block_table = case.block_table[order]
    case.lens = case.lens[order]
    b = _run(case, "bf16")
    np.testing.assert_array_equal(a[order], b)


def test_bf16_full_config2_sampled():
    """B=64, lengths U[1024, 8192], a 200k-page pool: the full isolated
    attention workload, in the launch configuration the benchmark times.
    Eight sequences are checked against the oracle row by row."""
    B, HQ, HKV, DH, POOL = 64, 32, 8, 128, 200000
    lens = lengths_uniform(B, 1024, 8192, seed=21)
    case = lazy_paged_attention_case(B, HQ, HKV, DH, lens, POOL, seed=22)
    k = torch.zeros((POOL, HKV, PAGE_TOKENS, DH), dtype=torch.bfloat16, device="cuda")
    v = torch.zeros((POOL, HKV, DH, PAGE_TOKENS), dtype=torch.bfloat16, device="cuda")
    q = torch.empty((B, HQ, DH), dtype=torch.bfloat16, device="cuda")
    for b in range(B):
        qb, kb, vb = case.sequence(b)
        npg = kb.shape[0]
        idx = torch.from_numpy(case.block_table[b, :npg].astype(np.int64)).cuda()
        k[idx] = torch.from_numpy(kb).cuda().to(torch.bfloat16)
        v[idx] = torch.from_numpy(np.ascontiguousarray(vb.transpose(0, 1, 3, 2))).cuda().to(
            torch.bfloat16)
        q[b] = torch.from_numpy(qb).cuda().to(torch.bfloat16)
    bt = torch.from_numpy(case.block_table).cuda()
    out = torch.empty((B, HQ, DH), dtype=torch.float32, device="cuda")
    _pdec().paged_decode_attention(q, k, v, bt, lens, out)
    got = out.cpu().numpy()
    assert np.isfinite(got).all()
    for b in [0, 7, 19, 31, 40, 52, 60, 63]:
        qb, kb, vb = case.sequence(b)
        n = int(lens[b])
        keys = kb.transpose(0, 2, 1, 3).reshape(-1, HKV, DH)[:n].astype(np.float64)
        vals = vb.transpose(0, 2, 1, 3).reshape(-1, HKV, DH)[:n].astype(np.float64)
        ref = oracle.attention(qb.astype(np.float64), keys, vals)
        for h in range(HQ):
            err = np.max(np.abs(got[b, h] - ref[h]))
            assert err <= BF16_TOL * np.max(np.abs(ref[h])), (b, h, err)


def _full_size_sampled(lens, sampled, seed):
    """The attention pass at a decode workload's full size, in the launch
    configuration of the decode step (the same planner and kernels): every
    sequence's pages are filled on the GPU (torch's seeded generator), then
    the pages and query of the sampled sequences are overwritten with the
    seeded host draws of the lazy case, and those sequences' outputs are
    checked against the oracle row by row.  Attention is per sequence, so
    the filler around them shapes only the work split, not their result."""
    from workload import EIGHT_B
    B, HQ, HKV, DH = len(lens), EIGHT_B.n_q_heads, EIGHT_B.n_kv_heads, EIGHT_B.head_dim
    pages = int(np.sum((np.asarray(lens) + PAGE_TOKENS - 1) // PAGE_TOKENS))
    pool = pages + 64
    case = lazy_paged_attention_case(B, HQ, HKV, DH, lens, pool, seed=seed)
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    k = torch.empty((pool, HKV, PAGE_TOKENS, DH), dtype=torch.bfloat16, device="cuda")
    v = torch.empty((pool, HKV, DH, PAGE_TOKENS), dtype=torch.bfloat16, device="cuda")
    k.normal_(generator=g)
    v.normal_(generator=g)
    q = torch.empty((B, HQ, DH), dtype=torch.bfloat16, device="cuda").normal_(generator=g)
    for b in sampled:
        qb, kb, vb = case.sequence(b)
        idx = torch.from_numpy(case.block_table[b, :kb.shape[0]].astype(np.int64)).cuda()
        k[idx] = torch.from_numpy(kb).cuda().to(torch.bfloat16)
        v[idx] = torch.from_numpy(np.ascontiguousarray(vb.transpose(0, 1, 3, 2))).cuda().to(
            torch.bfloat16)
        q[b] = torch.from_numpy(qb).cuda().to(torch.bfloat16)
    bt = torch.from_numpy(case.block_table).cuda()
    out = torch.empty((B, HQ, DH), dtype=torch.float32, device="cuda")
    _pdec().paged_decode_attention(q, k, v, bt, lens, out)
    got = out.cpu().numpy()
    for b in sampled:
        qb, kb, vb = case.sequence(b)
        n = int(lens[b])
        keys = kb.transpose(0, 2, 1, 3).reshape(-1, HKV, DH)[:n].astype(np.float64)
        vals = vb.transpose(0, 2, 1, 3).reshape(-1, HKV, DH)[:n].astype(np.float64)
        ref = oracle.attention(qb.astype(np.float64), keys, vals)
        assert np.isfinite(got[b]).all()
        for h in range(HQ):
            err = np.max(np.abs(got[b, h] - ref[h]))
            assert err <= BF16_TOL * np.max(np.abs(ref[h])), (b, h, err)


def test_bf16_full_size_b256_lognormal_sampled():
    """B=256, contexts lognormal (median 4096, sigma 0.8, clipped to
    [256, 32768]), the default decode workload's draw: 1.27 M keys, 5.2 GB of
    K and V pages.  Sampled: the shortest, the longest and six others."""
    from workload import lengths_lognormal
    lens = lengths_lognormal(256, 4096, 0.8, 256, 32768, 1)
    order = np.argsort(lens)
    sampled = sorted({int(order[0]), int(order[-1]), 3, 64, 100, 128, 200, 255})
    _full_size_sampled(lens, sampled, seed=31)


def test_bf16_full_size_b8_long_sampled():
    """B=8, contexts U[65536, 131072], the long-context decode workload's
    draw: ~0.8 M keys, 3.2 GB of pages, each sequence cut into dozens of
    items.  Sampled: three sequences, including the longest."""
    lens = lengths_uniform(8, 65536, 131072, 1)
    sampled = sorted({int(np.argmax(lens)), 0, 5})
    _full_size_sampled(lens, sampled, seed=32)
