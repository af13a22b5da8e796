"""KV snapshot to host memory and restore (kv_export / kv_import), through the
C ABI: the prepared-KV alternative to re-prefill for a departing trajectory.

A trajectory snapshotted, freed and restored into new pages must continue
bitwise identically to one that never left (the KV bytes are the same and
the attention result does not depend on physical page placement).
"""

import numpy as np
import pytest
import torch

from workload import SMALL_BF16, TINY, make_weights, random_tokens

pytestmark = pytest.mark.gpu


def _P():
    import paper_2609_36899_amd as P
    return P


def _engine(shape, bf16, pool_tokens=2048, kv_fp8=None):
    P = _P()
    dt = P.BF16 if bf16 else P.F32
    w = P.weights_to_device(make_weights(shape, seed=7, bf16=bf16), dt)
    per_tok = P.kv_bytes_per_token(shape, dt, kv_fp8)
    return P.Engine(shape, w, dt, pool_tokens * per_tok, max_seqs=8, max_seq_len=1024,
                    max_batch=4, max_chunk=32, kv_fp8=kv_fp8)


@pytest.mark.parametrize("shape,bf16,kv_fp8", [(TINY, False, None), (SMALL_BF16, True, None),
                                               (SMALL_BF16, True, (0.5, 0.5))])
def test_snapshot_restore_continues_bitwise(shape, bf16, kv_fp8):
    E = _engine(shape, bf16, kv_fp8=kv_fp8)
    toks = random_tokens(90, shape.vocab, seed=3)
    logits = torch.empty((1, shape.vocab), dtype=torch.float32, device="cuda")
    a = E.kv_alloc(0)
    E.kv_append_prefix(a, toks[:70], chunk_tokens=32)
    for t in toks[70:85]:
        E.decode_step([a], torch.tensor([int(t)], dtype=torch.int32, device="cuda"), logits)
    n = E.kv_len(a)
    assert n == 85
    snap = torch.empty(E.kv_snapshot_bytes(n), dtype=torch.uint8).pin_memory()
    assert E.kv_export(a, snap) == n
    torch.cuda.synchronize()
    # the snapshot's first page equals the pool's pages, block by block
    page0 = int(E.kv_block_table(a)[0])
    per_block = E.kv_token_bytes * 16 // (2 * shape.n_layers)
    for layer in (0, shape.n_layers - 1):
        k_dev = E.k_pages(layer)[page0].contiguous().view(torch.uint8).cpu()
        v_dev = E.v_pages(layer)[page0].contiguous().view(torch.uint8).cpu()
        k_off = (layer * 2) * per_block
        assert torch.equal(snap[k_off:k_off + per_block], k_dev.reshape(-1))
        assert torch.equal(snap[k_off + per_block:k_off + 2 * per_block], v_dev.reshape(-1))
    # the trajectory that stays
    stay = []
    for t in toks[85:]:
        E.decode_step([a], torch.tensor([int(t)], dtype=torch.int32, device="cuda"), logits)
        stay.append(logits.cpu().numpy().copy())
    h0 = E.kv_headroom()
    E.kv_free(a)
    assert E.kv_headroom() > h0
    # occupy the freed pages so the restore lands on different physical pages
    filler = E.kv_alloc(0)
    E.kv_append_prefix(filler, toks[:40], chunk_tokens=32)
    b = E.kv_alloc(0)
    E.kv_import(b, snap, n)
    assert E.kv_len(b) == n
    assert set(E.kv_block_table(b).tolist()).isdisjoint(E.kv_block_table(filler).tolist())
    moved = []
    for t in toks[85:]:
        E.decode_step([b], torch.tensor([int(t)], dtype=torch.int32, device="cuda"), logits)
        moved.append(logits.cpu().numpy().copy())
    for s, m in zip(stay, moved):
        np.testing.assert_array_equal(s, m)


def test_snapshot_errors():
    P = _P()
    E = _engine(TINY, False, pool_tokens=256)
    a = E.kv_alloc(0)
    E.kv_append_prefix(a, random_tokens(40, TINY.vocab, 1), chunk_tokens=16)
    small = torch.empty(E.kv_snapshot_bytes(40) - 16, dtype=torch.uint8).pin_memory()
    with pytest.raises(P.PdecError) as ei:
        E.kv_export(a, small)
    assert ei.value.code == P.engine.N.INVALID_ARG
    snap = torch.empty(E.kv_snapshot_bytes(40), dtype=torch.uint8).pin_memory()
    with pytest.raises(AssertionError):  # the binding accepts pinned host tensors only
        E.kv_export(a, torch.empty(E.kv_snapshot_bytes(40), dtype=torch.uint8))
    assert E.kv_export(a, snap) == 40
    torch.cuda.synchronize()
    with pytest.raises(P.PdecError) as ei:
        E.kv_import(a, snap, 40)  # not an empty sequence
    assert ei.value.code == P.engine.N.INVALID_ARG
    # 256-token pool: 3 pages held by a, 13 free; a 15-page import cannot fit
    b = E.kv_alloc(0)
    big = torch.empty(E.kv_snapshot_bytes(240), dtype=torch.uint8).pin_memory()
    h0 = E.kv_headroom()
    with pytest.raises(P.PdecError) as ei:
        E.kv_import(b, big, 240)
    assert ei.value.code == P.engine.N.OUT_OF_PAGES
    assert E.kv_len(b) == 0 and E.kv_headroom() == h0
    E.kv_import(b, snap, 40)
    assert E.kv_len(b) == 40
