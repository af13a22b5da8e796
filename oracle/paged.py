"""Paged-gather form of decode attention (oracle side).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The inference backend keeps each trajectory's KV history in fixed-size pages
indexed by a per-trajectory block table (the paged memory manager the paper's
backend uses for memory management, Design: separating departure from
placement).  Logical position j of trajectory b lives in page
``block_table[b][j // 16]`` at slot ``j % 16``.  Paging changes where values
live, not what attention computes: the oracle gathers the pages back into a
contiguous history and applies the plain attention definition.
"""

from __future__ import annotations

import numpy as np

from .decoder import attention

PAGE = 16


def gather_pages(pool: np.ndarray, block_row: np.ndarray, length: int) -> np.ndarray:
    """Contiguous ``[length, Hkv, Dh]`` history from a ``[P, Hkv, 16, Dh]`` pool."""
    out = np.empty((length, pool.shape[1], pool.shape[3]), dtype=pool.dtype)
    for j in range(length):
        out[j] = pool[int(block_row[j // PAGE]), :, j % PAGE, :]
    return out


def paged_decode_attention(q: np.ndarray, k_pool: np.ndarray, v_pool: np.ndarray,
                           block_table: np.ndarray, lens) -> np.ndarray:
    """Decode attention for a batch: q ``[B, Hq, Dh]`` against paged K/V.

    Sequence b attends over its ``lens[b]`` cached positions.  Returns
    ``[B, Hq, Dh]`` in the dtype of the inputs (float64 for parity).
    """
    out = np.empty(q.shape, dtype=np.float64)
    for b in range(q.shape[0]):
        n = int(lens[b])
        keys = gather_pages(k_pool, block_table[b], n).astype(np.float64)
        vals = gather_pages(v_pool, block_table[b], n).astype(np.float64)
        out[b] = attention(q[b].astype(np.float64), keys, vals)
    return out
