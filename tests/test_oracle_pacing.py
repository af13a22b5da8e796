"""Pins of the single-worker pacing oracle (CPU).

* hand-worked cases (tests/golden/pacing_examples.txt);
* the algorithm's defining properties on random states (hypothesis):
  after Phase 1 the headroom is at the floor or nobody is left; the evicted
  are the longest residents, and no shorter prefix of them would have
  sufficed; every placement met the threshold when it was made; every
  trajectory left pending misses the threshold in the final state; placements
  go shortest first.
* planted mistakes (shortest-first eviction, a missing +1 in the reserve,
  longest-first placement) break a pin.
"""

import os

import pytest
from hypothesis import given, settings, strategies as st

from oracle import pacing as op

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "pacing_examples.txt")


def _parse_ids(field):
    field = field.strip()
    return [] if field == "-" else [int(x) for x in field.split()]


def golden_cases():
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        name, hd, act, pend, ev, pl = [f.strip() for f in line.split("|")]
        h, h_min, delta = (int(x) for x in hd.split())
        active = [] if act == "-" else [tuple(int(y) for y in a.split(":")) for a in act.split()]
        pending = [] if pend == "-" else [tuple(int(y) for y in p.split(":")) for p in pend.split()]
        yield name, (h, h_min, delta, active, pending), (_parse_ids(ev), _parse_ids(pl))


def golden_ok(plan):
    return all(tuple(plan(*args)) == tuple(want) for _, args, want in golden_cases())


def properties_hold(plan, h, h_min, delta, active, pending):
    evicted, placed = plan(h, h_min, delta, active, pending)
    held = {rid: hd for rid, _, hd in active}
    length = {rid: ln for rid, ln, _ in active}
    length.update(dict(pending))
    hh = h + sum(held[r] for r in evicted)
    remaining = [r for r, _, _ in active if r not in evicted]
    # Phase 1: floor restored or nobody left; longest first; minimal
    if hh < h_min and remaining:
        return False
    order = sorted((r for r, _, _ in active), key=lambda r: (-length[r], r))
    if evicted != order[:len(evicted)]:
        return False
    if evicted and h + sum(held[r] for r in evicted[:-1]) >= h_min:
        return False
    # Phase 2: each placement feasible when made, shortest first
    n = len(remaining)
    for r in placed:
        after = hh - op.footprint(length[r])
        if after < h_min + (n + 1) * delta:
            return False
        hh, n = after, n + 1
    if [length[r] for r in placed] != sorted(length[r] for r in placed):
        return False
    left = set(length) - set(remaining) - set(placed)
    return all(hh - op.footprint(length[r]) < h_min + (n + 1) * delta for r in left)


states = st.integers(0, 5000).flatmap(lambda h: st.tuples(
    st.just(h), st.integers(0, 4000), st.integers(0, 300),
    st.lists(st.tuples(st.integers(1, 3000), st.integers(0, 64)), max_size=12),
    st.lists(st.integers(1, 3000), max_size=8)))


def _unpack(s):
    h, h_min, delta, act, pend = s
    # held tokens: the whole pages of the length, sometimes one reserved page more
    active = [(i, ln, op.footprint(ln) + (16 if extra % 5 == 0 else 0))
              for i, (ln, extra) in enumerate(act)]
    pending = [(100 + j, ln) for j, ln in enumerate(pend)]
    return h, h_min, delta, active, pending


def test_golden_cases():
    for name, args, want in golden_cases():
        assert tuple(op.pacing_plan(*args)) == tuple(want), name


@settings(max_examples=300, deadline=None)
@given(states)
def test_properties(s):
    assert properties_hold(op.pacing_plan, *_unpack(s))


def _mut_shortest_evicted(h, h_min, delta, active, pending):
    rev = [(r, -ln, hd) for r, ln, hd in active]  # flips the eviction order
    ev, _ = op.pacing_plan(h, h_min, delta, rev, [])
    lengths = {r: ln for r, ln, _ in active}
    act2 = [a for a in active if a[0] not in ev]
    held = sum(hd for r, _, hd in active if r in ev)
    _, pl = op.pacing_plan(h + held, h_min, delta, act2,
                           list(pending) + [(r, lengths[r]) for r in ev])
    return ev, pl


def _mut_reserve_without_incoming(h, h_min, delta, active, pending):
    ev, _ = op.pacing_plan(h, h_min, delta, active, [])
    hh = h + sum(hd for r, _, hd in active if r in ev)
    n = len(active) - len(ev)
    waiting = dict(pending)
    waiting.update({r: ln for r, ln, _ in active if r in ev})
    placed = []
    for r in sorted(waiting, key=lambda r: (waiting[r], r)):
        after = hh - op.footprint(waiting[r])
        if after >= h_min + n * delta:  # missing the +1 for the incoming one
            hh, n = after, n + 1
            placed.append(r)
    return ev, placed


def _mut_longest_placed_first(h, h_min, delta, active, pending):
    ev, _ = op.pacing_plan(h, h_min, delta, active, [])
    hh = h + sum(hd for r, _, hd in active if r in ev)
    n = len(active) - len(ev)
    waiting = dict(pending)
    waiting.update({r: ln for r, ln, _ in active if r in ev})
    placed = []
    for r in sorted(waiting, key=lambda r: (-waiting[r], r)):
        after = hh - op.footprint(waiting[r])
        if after >= h_min + (n + 1) * delta:
            hh, n = after, n + 1
            placed.append(r)
    return ev, placed


@pytest.mark.parametrize("mutant", [_mut_shortest_evicted, _mut_reserve_without_incoming,
                                    _mut_longest_placed_first])
def test_planted_mistakes_break_a_pin(mutant):
    assert not golden_ok(mutant)
