"""Headroom pacing on one worker (oracle side).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's pacing algorithm (Design, "Separating Departure from Placement":
pacing thresholds; Alg. pacing) restricted to one worker, the only one a
single GPU holds:

* Phase 1, restore headroom: while the headroom H is below the floor H_min
  and residents remain, evict the longest resident (ties: lower id) to the
  pending pool; H rises by the tokens its pages held.
* Phase 2, place shortest first: take pending trajectories in ascending
  length (ties: lower id); r is placed when the headroom left after placing
  it, H - footprint(r), is at least H_min + (|A| + 1) * delta, with |A| the
  residents before placing r.  H then falls by footprint(r).

With one worker the prefix-affine sticky table and the tight-fit choice
among feasible workers both name the same worker.  A trajectory's footprint
is its KV in whole 16-token pages: ceil(len / 16) * 16 tokens.
"""

from __future__ import annotations

from typing import List, Sequence, Tuple

PAGE = 16


def footprint(length: int) -> int:
    return -(-int(length) // PAGE) * PAGE


def pacing_plan(headroom: int, h_min: int, delta: int,
                active: Sequence[Tuple[int, int, int]],
                pending: Sequence[Tuple[int, int]]) -> Tuple[List[int], List[int]]:
    """active: (id, length, held_tokens); pending: (id, length).

    Returns (evicted ids in eviction order, placed ids in placement order).
    """
    h = int(headroom)
    residents = {rid: (int(length), int(held)) for rid, length, held in active}
    waiting = {rid: int(length) for rid, length in pending}
    evicted: List[int] = []
    # Phase 1: longest first while below the floor.
    while h < h_min and residents:
        rid = max(residents, key=lambda r: (residents[r][0], -r))
        length, held = residents.pop(rid)
        h += held
        waiting[rid] = length
        evicted.append(rid)
    # Phase 2: shortest first, placement threshold with the decode reserve.
    placed: List[int] = []
    n_active = len(residents)
    for rid in sorted(waiting, key=lambda r: (waiting[r], r)):
        after = h - footprint(waiting[rid])
        if after >= h_min + (n_active + 1) * delta:
            h = after
            n_active += 1
            placed.append(rid)
    return evicted, placed
