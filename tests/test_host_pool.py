"""Host bookkeeping of the paged KV cache, tested on the CPU.

The page pool, the resident-set table and the attention work planner are
plain C++ (libpdec_host.so, built by g++).  They are checked against a small
Python model of the same rules: admission with a token reserve, growth that
is all-or-nothing, departure that raises the headroom at once, stale ids, and
a work list that covers every key of every query block exactly once.
"""

import ctypes
import os
from ctypes import POINTER, byref, c_int32, c_int64, c_void_p

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
# PDEC_HOST_LIB selects another build of the host library (the sanitizer
# build, see tests/test_sanitizers.py).
HOST_LIB = os.environ.get("PDEC_HOST_LIB") or os.path.join(ROOT, "paper_2609_36899_amd",
                                                           "libpdec_host.so")

OK, INVALID_ARG, OUT_OF_PAGES, BAD_SEQ, SEQ_TOO_LONG = 0, -1, -2, -3, -4


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(HOST_LIB):
        from paper_2609_36899_amd import build
        build.build_host()
    L = ctypes.CDLL(HOST_LIB)
    L.pp_create.restype = c_void_p
    L.pp_create.argtypes = [c_int32, c_int32, c_int32]
    L.pp_destroy.argtypes = [c_void_p]
    L.pp_alloc.argtypes = [c_void_p, c_int32, POINTER(c_int32)]
    L.pp_free.argtypes = [c_void_p, c_int32]
    L.pp_len.argtypes = [c_void_p, c_int32, POINTER(c_int32)]
    L.pp_headroom.restype = c_int64
    L.pp_headroom.argtypes = [c_void_p]
    L.pp_grow.argtypes = [c_void_p, POINTER(c_int32), c_int32, c_int32, c_int32]
    L.pp_pages.argtypes = [c_void_p, c_int32, POINTER(c_int32), c_int32]
    L.pp_slot.argtypes = [c_void_p, c_int32]
    L.pp_pending.argtypes = [c_void_p, POINTER(c_int32), c_int32]
    L.pp_clear_pending.argtypes = [c_void_p]
    L.pp_choose_split.argtypes = [c_int64, c_int32]
    L.pp_target_items.restype = c_int64
    L.pp_target_items.argtypes = [c_int32]
    L.pp_plan.argtypes = [POINTER(c_int32), c_int32, c_int32, POINTER(c_int32),
                          POINTER(c_int32), c_int32]
    L.pp_total_key_pages.restype = c_int64
    L.pp_total_key_pages.argtypes = [POINTER(c_int32), c_int32]
    L.pp_last_error.restype = ctypes.c_char_p
    L.pp_validate_pass.argtypes = [c_void_p, POINTER(c_int32), c_int32, POINTER(c_int32),
                                   c_int32, POINTER(c_int32), c_int32, c_int32, c_int32, c_int32]
    L.pp_validate_deltas.argtypes = [POINTER(c_int32), c_int32, c_int32, c_int32, c_int32]
    L.pp_pacing_plan.argtypes = [c_int64, c_int64, c_int64, c_int32, POINTER(c_int32),
                                 POINTER(c_int32), POINTER(ctypes.c_int64), c_int32,
                                 POINTER(c_int32), POINTER(c_int32), POINTER(c_int32),
                                 POINTER(c_int32), POINTER(c_int32), POINTER(c_int32)]
    return L


class Pool:
    def __init__(self, lib, n_pages, max_seqs, max_len):
        self.lib = lib
        self.h = lib.pp_create(n_pages, max_seqs, max_len)
        assert self.h

    def __del__(self):
        self.lib.pp_destroy(self.h)

    def alloc(self, reserve):
        out = c_int32(-1)
        rc = self.lib.pp_alloc(self.h, reserve, byref(out))
        return rc, out.value

    def free(self, sid):
        return self.lib.pp_free(self.h, sid)

    def len(self, sid):
        out = c_int32(-1)
        rc = self.lib.pp_len(self.h, sid, byref(out))
        return rc, out.value

    def headroom(self):
        return self.lib.pp_headroom(self.h)

    def grow(self, ids, extra, undo_after=0):
        a = (c_int32 * len(ids))(*ids)
        return self.lib.pp_grow(self.h, a, len(ids), extra, undo_after)

    def pages(self, sid):
        buf = (c_int32 * 4096)()
        n = self.lib.pp_pages(self.h, sid, buf, 4096)
        return list(buf[:n]) if n >= 0 else n

    def pending(self):
        buf = (c_int32 * (3 * 65536))()
        n = self.lib.pp_pending(self.h, buf, 65536)
        return [tuple(buf[3 * i:3 * i + 3]) for i in range(n)]


def test_admission_reserve_and_headroom(lib):
    p = Pool(lib, n_pages=10, max_seqs=4, max_len=1000)
    assert p.headroom() == 160
    rc, a = p.alloc(33)           # 3 pages reserved
    assert rc == OK and p.headroom() == 7 * 16
    rc, b = p.alloc(7 * 16 + 1)   # needs 8 pages, 7 free: refused, nothing changes
    assert rc == OUT_OF_PAGES and p.headroom() == 7 * 16
    rc, b = p.alloc(0)
    assert rc == OK and p.pages(b) == []
    assert p.len(a) == (OK, 0)
    # growth uses the reserve first
    assert p.grow([a], 48) == OK and p.headroom() == 7 * 16 and len(p.pages(a)) == 3
    assert p.grow([a], 1) == OK and p.headroom() == 6 * 16
    assert p.len(a) == (OK, 49)


def test_departure_and_stale_ids(lib):
    p = Pool(lib, n_pages=8, max_seqs=2, max_len=1000)
    rc, a = p.alloc(64)
    assert p.headroom() == 4 * 16
    assert p.free(a) == OK and p.headroom() == 8 * 16   # departure frees at once
    assert p.free(a) == BAD_SEQ                          # double free rejected
    assert p.len(a)[0] == BAD_SEQ
    rc, b = p.alloc(0)
    assert rc == OK and b != a                           # same slot, new generation
    assert p.grow([a], 1) == BAD_SEQ
    rc, c = p.alloc(0)
    rc, d = p.alloc(0)
    assert rc == INVALID_ARG                             # no free slot


def test_grow_is_atomic_across_batch(lib):
    p = Pool(lib, n_pages=5, max_seqs=4, max_len=100)
    ids = [p.alloc(0)[1] for _ in range(3)]
    assert p.grow(ids, 16) == OK                  # 3 pages used, 2 free
    before = [p.len(i)[1] for i in ids], [p.pages(i) for i in ids], p.headroom()
    assert p.grow(ids, 1) == OUT_OF_PAGES         # needs 3 new pages
    after = [p.len(i)[1] for i in ids], [p.pages(i) for i in ids], p.headroom()
    assert before == after
    assert p.grow(ids[:2], 1) == OK
    assert p.grow([ids[2]], 100) == SEQ_TOO_LONG
    assert p.len(ids[2]) == (OK, 16)


def test_undo_restores_state(lib):
    p = Pool(lib, n_pages=50, max_seqs=4, max_len=1000)
    ids = [p.alloc(20)[1] for _ in range(3)]
    lib.pp_clear_pending(p.h)
    snap = ([p.len(i)[1] for i in ids], [p.pages(i) for i in ids], p.headroom())
    assert p.grow(ids, 37, undo_after=1) == OK
    assert ([p.len(i)[1] for i in ids], [p.pages(i) for i in ids], p.headroom()) == snap
    assert p.pending() == []


def test_pending_deltas_match_block_tables(lib):
    p = Pool(lib, n_pages=64, max_seqs=8, max_len=4096)
    ids = [p.alloc(r)[1] for r in (0, 17, 40)]
    p.grow(ids, 50)
    table = {}
    for slot, idx, page in p.pending():
        table[(slot, idx)] = page
    for i in ids:
        slot = lib.pp_slot(p.h, i)
        pages = p.pages(i)
        assert [table[(slot, k)] for k in range(len(pages))] == pages


class ModelPool:
    """Python model of the pool's rules."""

    def __init__(self, n_pages, max_seqs, max_len):
        self.free, self.max_seqs, self.max_len = n_pages, max_seqs, max_len
        self.seqs = {}

    def alloc(self, reserve):
        need = -(-reserve // 16)
        if reserve > self.max_len:
            return INVALID_ARG
        if len(self.seqs) >= self.max_seqs:
            return INVALID_ARG
        if need > self.free:
            return OUT_OF_PAGES
        self.free -= need
        return OK, need

    def grow(self, keys, extra):
        need = 0
        for k in keys:
            ln, npg = self.seqs[k]
            if ln + extra > self.max_len:
                return SEQ_TOO_LONG
            need += max(0, -(-(ln + extra) // 16) - npg)
        if need > self.free:
            return OUT_OF_PAGES
        for k in keys:
            ln, npg = self.seqs[k]
            new = -(-(ln + extra) // 16)
            self.free -= max(0, new - npg)
            self.seqs[k] = (ln + extra, max(npg, new))
        return OK


def test_free_then_realloc_leaves_no_stale_pending_entry(lib):
    # The device applies all pending entries in parallel, in no order, so a
    # freed slot's unflushed entry beside its next occupant's entry for the
    # same (slot, idx) could point that occupant at another sequence's page.
    p = Pool(lib, n_pages=8, max_seqs=4, max_len=256)
    rc, a = p.alloc(32)                      # slot 0, pages 0, 1
    assert rc == OK
    assert p.free(a) == OK
    rc, b = p.alloc(16)                      # slot 0 again
    rc2, c = p.alloc(16)                     # slot 1
    assert rc == rc2 == OK
    assert p.grow([b], 17) == OK             # slot 0 attaches a second page
    pend = p.pending()
    keys = [(s, i) for s, i, _ in pend]
    assert len(keys) == len(set(keys))
    table = {(s, i): pg for s, i, pg in pend}
    for sid in (b, c):
        slot = lib.pp_slot(p.h, sid)
        assert [table[(slot, k)] for k in range(len(p.pages(sid)))] == p.pages(sid)
    assert set(p.pages(b)).isdisjoint(p.pages(c))


ops = st.lists(st.tuples(st.sampled_from(["alloc", "free", "grow", "grow_all", "flush"]),
                         st.integers(0, 200), st.integers(0, 7)), min_size=1, max_size=60)


@settings(max_examples=150, deadline=None)
@given(ops)
def test_pool_matches_python_model(lib, seq_ops):
    n_pages, max_seqs, max_len = 40, 6, 300
    p = Pool(lib, n_pages, max_seqs, max_len)
    m = ModelPool(n_pages, max_seqs, max_len)
    live = []  # (id, key)
    key = 0
    device = {}  # the device block table: (slot, idx) -> page

    def flush():
        pend = p.pending()
        keys = [(s, i) for s, i, _ in pend]
        assert len(keys) == len(set(keys)), "a (slot, idx) pending twice"
        for s, i, pg in pend:
            device[(s, i)] = pg
        lib.pp_clear_pending(p.h)

    for op, a, b in seq_ops:
        if op == "flush":
            flush()
        if op == "alloc":
            rc, sid = p.alloc(a)
            exp = m.alloc(a)
            if isinstance(exp, tuple):
                assert rc == OK
                m.seqs[key] = (0, exp[1])
                live.append((sid, key))
                key += 1
            else:
                assert rc == exp
        elif op == "free" and live:
            sid, k = live.pop(b % len(live))
            assert p.free(sid) == OK
            m.free += m.seqs.pop(k)[1]
            assert p.free(sid) == BAD_SEQ
        elif op in ("grow", "grow_all") and live:
            chosen = live if op == "grow_all" else [live[b % len(live)]]
            extra = a % 70
            rc = p.grow([s for s, _ in chosen], extra)
            assert rc == m.grow([k for _, k in chosen], extra)
        assert p.headroom() == 16 * m.free
        for sid, k in live:
            assert p.len(sid) == (OK, m.seqs[k][0])
            assert len(p.pages(sid)) == m.seqs[k][1]
    # After the deltas reach the device, its table matches every live
    # sequence's pages.
    flush()
    for sid, _ in live:
        slot = lib.pp_slot(p.h, sid)
        assert [device[(slot, k)] for k in range(len(p.pages(sid)))] == p.pages(sid)
    # pages of live sequences are distinct and disjoint from each other
    allp = [pg for sid, _ in live for pg in p.pages(sid)]
    assert len(allp) == len(set(allp))
    assert all(0 <= x < n_pages for x in allp)


def _plan(lib, specs, split):
    arr = (c_int32 * (4 * len(specs)))(*[v for s in specs for v in s])
    cap = 200000
    qb = (c_int32 * (6 * len(specs)))()
    it = (c_int32 * (4 * cap))()
    n = lib.pp_plan(arr, len(specs), split, qb, it, cap)
    assert n >= 0
    qbs = [tuple(qb[6 * i:6 * i + 6]) for i in range(len(specs))]
    items = [tuple(it[4 * i:4 * i + 3]) for i in range(n)]
    order = [it[4 * i + 3] for i in range(n)]
    # The dispatch order is a permutation, longest items first.
    assert sorted(order) == list(range(n))
    sizes = [items[o][2] for o in order]
    assert sizes == sorted(sizes, reverse=True)
    return qbs, items


@settings(max_examples=100, deadline=None)
@given(st.lists(st.tuples(st.integers(0, 5000), st.integers(1, 8)), min_size=1, max_size=20),
       st.sampled_from([1, 2, 8, 16]))
def test_plan_covers_each_key_once(lib, blocks, hkv):
    specs = [(4 * i, nq, i, pos0) for i, (pos0, nq) in enumerate(blocks)]
    arr = (c_int32 * (4 * len(specs)))(*[v for s in specs for v in s])
    total = lib.pp_total_key_pages(arr, len(specs))
    assert total == sum(-(-(pos0 + nq) // 16) for pos0, nq in blocks)
    split = lib.pp_choose_split(total, hkv)
    assert split >= 8 and split % 2 == 0
    qbs, items = _plan(lib, specs, split)
    assert len(items) <= lib.pp_target_items(hkv) + len(specs)
    for i, (pos0, nq) in enumerate(blocks):
        q = qbs[i]
        assert q[:4] == specs[i]
        mine = items[q[4]:q[5]]
        assert all(x[0] == i for x in mine)
        covered = []
        for _, pb, npg in mine:
            assert 1 <= npg <= split
            covered.extend(range(pb, pb + npg))
        assert covered == list(range(-(-(pos0 + nq) // 16)))


def test_split_targets_work_group_count(lib):
    # A long-context batch gets enough items to fill the grid; a tiny one
    # falls back to the minimum split of 8 pages.
    assert lib.pp_choose_split(10, 8) == 8
    total = 64 * 6144
    s = lib.pp_choose_split(total, 8)
    items = -(-total // s)
    assert lib.pp_target_items(8) // 2 <= items <= lib.pp_target_items(8)


def _arr(vals):
    vals = [int(v) for v in vals]
    return (c_int32 * max(len(vals), 1))(*vals)


def _validate(lib, pool, rows, qbs, items, max_seqs=8, max_len=4096, bt_stride=256):
    return lib.pp_validate_pass(pool, _arr([v for r in rows for v in r]), len(rows),
                                _arr([v for q in qbs for v in q]), len(qbs),
                                _arr([v for it in items for v in it]), len(items),
                                max_seqs, max_len, bt_stride)


def _decode_pass(lib, p, ids):
    """Rows, query blocks and items of one decode step over ids (after growth)."""
    rows, specs = [], []
    for b, sid in enumerate(ids):
        slot, pos = lib.pp_slot(p.h, sid), p.len(sid)[1] - 1
        rows.append((slot, pos))
        specs.append((b, 1, slot, pos))
    arr = _arr([v for sp in specs for v in sp])
    split = lib.pp_choose_split(lib.pp_total_key_pages(arr, len(specs)), 8)
    qb = (c_int32 * (6 * len(specs)))()
    it = (c_int32 * (4 * 4096))()
    n = lib.pp_plan(arr, len(specs), split, qb, it, 4096)
    assert n > 0
    return (rows, [tuple(qb[6 * i:6 * i + 6]) for i in range(len(specs))],
            [tuple(it[4 * i:4 * i + 4]) for i in range(n)])


def test_validate_accepts_planned_passes_and_names_each_violation(lib):
    p = Pool(lib, n_pages=64, max_seqs=8, max_len=4096)
    ids = [p.alloc(0)[1] for _ in range(3)]
    for sid, n in zip(ids, (40, 300, 17)):
        assert p.grow([sid], n) == OK
    rows, qbs, items = _decode_pass(lib, p, ids)
    assert _validate(lib, p.h, rows, qbs, items) == OK
    assert _validate(lib, None, rows, qbs, items) == OK

    def rejects(rows_, qbs_, items_, pool=p.h, **kw):
        rc = _validate(lib, pool, rows_, qbs_, items_, **kw)
        assert rc == INVALID_ARG, rc
        return lib.pp_last_error().decode()

    # item range past the block's keys, and a gap in the covered keys
    bad = list(items)
    q, pb, npg, o = bad[qbs[0][4]]
    bad[qbs[0][4]] = (q, pb, npg + 1, o)
    assert "keys not covered" in rejects(rows, qbs, bad)
    bad = list(items)
    bad[qbs[1][4] + 1] = (1, bad[qbs[1][4] + 1][1] + 1, bad[qbs[1][4] + 1][2], bad[qbs[1][4] + 1][3])
    assert "item" in rejects(rows, qbs, bad)
    # dispatch order not a permutation
    bad = list(items)
    bad[0] = bad[0][:3] + (bad[1][3],)
    assert "dispatch order" in rejects(rows, qbs, bad)
    # a row past its sequence, a slot out of range, a position past the rope table
    assert "outside its sequence" in rejects([(rows[0][0], rows[0][1] + 1)] + rows[1:],
                                             [(0, 1, rows[0][0], rows[0][1] + 1) + qbs[0][4:]] +
                                             qbs[1:], items)
    assert "slot" in rejects([(9, 0)] + rows[1:], qbs, items, pool=None)
    assert "position" in rejects(rows, qbs, items, pool=None, max_len=100)
    # keys past the block-table row
    assert "block-table row" in rejects(rows, qbs, items, pool=None, bt_stride=2)
    # a freed sequence's block
    assert p.free(ids[2]) == OK
    assert "outside its sequence" in rejects(rows, qbs, items)


def test_validate_deltas(lib):
    ok = [(0, 0, 5), (0, 1, 6), (1, 0, 7)]
    flat = _arr([v for d in ok for v in d])
    assert lib.pp_validate_deltas(flat, 3, 4, 16, 8) == OK
    dup = ok + [(0, 1, 3)]
    assert lib.pp_validate_deltas(_arr([v for d in dup for v in d]), 4, 4, 16, 8) == INVALID_ARG
    assert "twice" in lib.pp_last_error().decode()
    for bad in ([(0, 0, 8)], [(4, 0, 1)], [(0, 16, 1)], [(0, -1, 1)], [(0, 0, -1)]):
        assert lib.pp_validate_deltas(_arr([v for d in bad for v in d]), 1, 4, 16, 8) == INVALID_ARG


@settings(max_examples=100, deadline=None)
@given(ops)
def test_every_decode_pass_of_a_random_history_validates(lib, seq_ops):
    p = Pool(lib, 40, 6, 300)
    live = []
    for op, a, b in seq_ops:
        if op == "alloc":
            rc, sid = p.alloc(a)
            if rc == OK:
                live.append(sid)
        elif op == "free" and live:
            assert p.free(live.pop(b % len(live))) == OK
        elif op in ("grow", "grow_all") and live:
            chosen = live if op == "grow_all" else [live[b % len(live)]]
            p.grow(chosen, a % 70)
        elif op == "flush":
            lib.pp_clear_pending(p.h)
        pend = p.pending()
        assert lib.pp_validate_deltas(_arr([v for d in pend for v in d]), len(pend), 6,
                                      19, 40) == OK
        nonempty = [s for s in live if p.len(s)[1] > 0]
        if nonempty:
            rows, qbs, items = _decode_pass(lib, p, nonempty)
            assert _validate(lib, p.h, rows, qbs, items, max_seqs=6, max_len=300,
                             bt_stride=19) == OK


@settings(max_examples=200, deadline=None)
@given(st.integers(0, 6000), st.integers(0, 5000), st.integers(0, 400),
       st.lists(st.tuples(st.integers(0, 4000), st.booleans()), max_size=20),
       st.lists(st.integers(0, 4000), max_size=12), st.integers(0, 1000))
def test_host_pacing_plan_equals_oracle(lib, h, h_min, delta, act, pend, seed):
    """The pacing decision in the host library (the same source the device
    library exports as pacing_plan) against the oracle."""
    from oracle import pacing as op
    ids = np.random.default_rng(seed).permutation(1000)[:len(act) + len(pend)].tolist()
    active = [(ids[i], ln, op.footprint(ln) + (16 if extra else 0))
              for i, (ln, extra) in enumerate(act)]
    pending = [(ids[len(act) + j], ln) for j, ln in enumerate(pend)]
    na, npd = len(active), len(pending)
    ev, pl = _arr([0] * na), _arr([0] * (na + npd))
    n_ev, n_pl = c_int32(), c_int32()
    held = (ctypes.c_int64 * max(na, 1))(*[a[2] for a in active])
    lib.pp_pacing_plan(h, h_min, delta, na, _arr([a[0] for a in active]),
                       _arr([a[1] for a in active]), held, npd, _arr([q[0] for q in pending]),
                       _arr([q[1] for q in pending]), ev, byref(n_ev), pl, byref(n_pl))
    got = (list(ev[:n_ev.value]), list(pl[:n_pl.value]))
    assert got == op.pacing_plan(h, h_min, delta, active, pending)
