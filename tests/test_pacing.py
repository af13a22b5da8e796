"""The library's pacing decision (C ABI pacing_plan, host only) against the
oracle on random single-worker states (CPU)."""

import numpy as np
from hypothesis import given, settings, strategies as st

from oracle import pacing as op


def _plan(*args):
    from paper_2609_36899_amd.driver import pacing_plan
    return pacing_plan(*args)


@settings(max_examples=400, deadline=None)
@given(st.integers(0, 6000), st.integers(0, 5000), st.integers(0, 400),
       st.lists(st.tuples(st.integers(0, 4000), st.booleans()), max_size=20),
       st.lists(st.integers(0, 4000), max_size=12), st.integers(0, 1000))
def test_native_plan_equals_oracle(h, h_min, delta, act, pend, seed):
    ids = np.random.default_rng(seed).permutation(1000)[:len(act) + len(pend)].tolist()
    active = [(ids[i], ln, op.footprint(ln) + (16 if extra else 0))
              for i, (ln, extra) in enumerate(act)]
    pending = [(ids[len(act) + j], ln) for j, ln in enumerate(pend)]
    assert _plan(h, h_min, delta, active, pending) == op.pacing_plan(h, h_min, delta, active,
                                                                     pending)


def test_argument_errors():
    from paper_2609_36899_amd import _native as N
    import pytest
    with pytest.raises(N.PdecError):
        _plan(0, -1, 0, [], [])
    with pytest.raises(N.PdecError):
        _plan(0, 0, 0, [(1, -5, 0)], [])
