"""Headroom-paced rollout on one engine (one worker's resident set).

The engine holds the resident trajectories' KV; a pending pool holds the
ones waiting for room.  Before every decode step the worker's pacing
decision (C ABI ``pacing_plan``: Alg. pacing restricted to one worker) names
the residents to evict and the pending trajectories to place:

* eviction snapshots the trajectory's KV into pinned host memory
  (``kv_export``) and frees its pages (``kv_free``), which raises the
  headroom at once (Design, "Separating Departure from Placement");
* placement restores the snapshot into fresh pages (``kv_import``), or
  prefills the tokens when there is none (``kv_append_prefix``, the
  re-prefill fallback; new trajectories arrive this way).

Placements beyond the engine's batch capacity (``max_batch`` residents)
wait for a later step: a resource limit of the worker next to its headroom.
The floor ``h_min`` should cover one new page per resident
(16 x the most residents a step can have), so that a decode step never runs
out of pages between two pacing decisions.
"""

from __future__ import annotations

from ctypes import byref, c_int32, c_int64
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch

from . import _native as N


def pacing_plan(headroom: int, h_min: int, delta: int,
                active: Sequence[Tuple[int, int, int]],
                pending: Sequence[Tuple[int, int]]) -> Tuple[List[int], List[int]]:
    """active: (id, length, held_tokens); pending: (id, length).
    Returns (evicted ids, placed ids) in order; see pacing_plan in include/pdec.h."""
    na, npd = len(active), len(pending)
    a_ids = (c_int32 * max(na, 1))(*[int(a[0]) for a in active])
    a_len = (c_int32 * max(na, 1))(*[int(a[1]) for a in active])
    a_held = (c_int64 * max(na, 1))(*[int(a[2]) for a in active])
    p_ids = (c_int32 * max(npd, 1))(*[int(p[0]) for p in pending])
    p_len = (c_int32 * max(npd, 1))(*[int(p[1]) for p in pending])
    ev = (c_int32 * max(na, 1))()
    pl = (c_int32 * max(na + npd, 1))()
    n_ev, n_pl = c_int32(), c_int32()
    N.check(N.load().pacing_plan(int(headroom), int(h_min), int(delta), na, a_ids, a_len, a_held,
                                 npd, p_ids, p_len, ev, byref(n_ev), pl, byref(n_pl)))
    return list(ev[:n_ev.value]), list(pl[:n_pl.value])


class _Traj:
    def __init__(self, tid: int, tokens: np.ndarray, prompt_len: int):
        self.id = tid
        self.tokens = np.asarray(tokens, dtype=np.int32)  # prompt + tokens to decode
        self.prompt_len = prompt_len
        self.cached = 0          # tokens whose KV exists (resident or in the snapshot)
        self.seq: Optional[int] = None
        self.snapshot: Optional[torch.Tensor] = None
        self.staged = False

    @property
    def done(self) -> bool:
        return self.cached >= len(self.tokens)


class PacedRollout:
    """Teacher-forced rollout of token streams under headroom pacing.

    Each trajectory is a prompt followed by the tokens it will decode (given
    up front, as in replaying a rollout); ``step`` decodes one token for
    every resident and returns the logits it produced per trajectory.
    """

    def __init__(self, engine, h_min: int, delta: int, restore: str = "snapshot",
                 chunk_tokens: int = 64):
        assert restore in ("snapshot", "reprefill")
        self.E = engine
        self.h_min, self.delta = int(h_min), int(delta)
        self.restore = restore
        self.chunk = int(chunk_tokens)
        self.trajs: Dict[int, _Traj] = {}
        self.resident: List[int] = []
        self.pending: List[int] = []
        self.stats = {"evictions": 0, "restores": 0, "prefills": 0, "snapshot_bytes": 0}
        self._logits = None

    def add(self, tid: int, tokens: Sequence[int], prompt_len: int, staged: bool = False) -> None:
        """Queue a trajectory.  ``staged`` places its prompt with
        kv_extend_uninit (positions without computed KV, for benchmarks
        whose cost does not depend on KV values) instead of a prefill."""
        assert tid not in self.trajs and 0 < prompt_len < len(tokens)
        self.trajs[tid] = _Traj(tid, np.asarray(tokens), prompt_len)
        self.trajs[tid].staged = staged
        self.pending.append(tid)

    def _length(self, t: _Traj) -> int:
        # tokens the trajectory's KV holds once placed
        return t.cached if t.cached else t.prompt_len

    def pace(self) -> Tuple[List[int], List[int]]:
        E = self.E
        active = []
        for tid in self.resident:
            t = self.trajs[tid]
            # placed with no reserve and grown a page at a time: whole pages of its length
            active.append((tid, t.cached, (t.cached + 15) // 16 * 16))
        pending = [(tid, self._length(self.trajs[tid])) for tid in self.pending]
        evicted, placed = pacing_plan(E.kv_headroom(), self.h_min, self.delta, active, pending)
        for tid in evicted:
            self._evict(self.trajs[tid])
        placed = placed[:max(0, E.max_batch - len(self.resident))]
        for tid in placed:
            self._place(self.trajs[tid])
        return evicted, placed

    def _evict(self, t: _Traj) -> None:
        E = self.E
        if self.restore == "snapshot":
            t.snapshot = torch.empty(E.kv_snapshot_bytes(t.cached), dtype=torch.uint8).pin_memory()
            E.kv_export(t.seq, t.snapshot)
            self.stats["snapshot_bytes"] += t.snapshot.numel()
        E.kv_free(t.seq)  # ordered after the export on the engine's stream
        t.seq = None
        self.resident.remove(t.id)
        self.pending.append(t.id)
        self.stats["evictions"] += 1

    def _place(self, t: _Traj) -> None:
        E = self.E
        t.seq = E.kv_alloc(0)
        if t.cached and t.snapshot is not None:
            E.kv_import(t.seq, t.snapshot, t.cached)
            self.stats["restores"] += 1
        elif not t.cached and t.staged:
            E.kv_extend_uninit(t.seq, t.prompt_len)
            t.cached = t.prompt_len
        else:
            n = t.cached if t.cached else t.prompt_len
            E.kv_append_prefix(t.seq, t.tokens[:n], chunk_tokens=self.chunk)
            t.cached = n
            self.stats["prefills"] += 1
        t.snapshot = None
        self.pending.remove(t.id)
        self.resident.append(t.id)

    def step(self) -> Dict[int, Tuple[int, torch.Tensor]]:
        """Pace, then decode one token for every resident.  Returns, per
        trajectory that decoded, the position of the token it consumed and the
        logits row it produced (a device view, valid until the next step)."""
        self.pace()
        live = [tid for tid in self.resident if not self.trajs[tid].done]
        if not live:
            return {}
        E = self.E
        vocab = E.shape.vocab
        if self._logits is None or self._logits.shape[0] < len(live):
            self._logits = torch.empty((max(len(live), E.max_batch), vocab), dtype=torch.float32,
                                       device="cuda")
        seqs = [self.trajs[tid].seq for tid in live]
        toks = torch.tensor([int(self.trajs[tid].tokens[self.trajs[tid].cached]) for tid in live],
                            dtype=torch.int32, device="cuda")
        logits = self._logits[:len(live)]
        E.decode_step(seqs, toks, logits)
        out = {}
        for i, tid in enumerate(live):
            t = self.trajs[tid]
            out[tid] = (t.cached, logits[i])
            t.cached += 1
        for tid in list(self.resident):  # finished trajectories depart
            t = self.trajs[tid]
            if t.done:
                E.kv_free(t.seq)
                t.seq = None
                self.resident.remove(tid)
        return out

    @property
    def finished(self) -> bool:
        return all(t.done for t in self.trajs.values())
