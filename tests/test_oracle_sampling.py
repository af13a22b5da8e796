"""Pins of the sampling oracle (CPU).

* a hand-worked example (tests/golden/sampling_worked_example.txt);
* stratified inverse-CDF frequencies equal softmax(z/T) probabilities, and
  with top_p < 1 the renormalised nucleus probabilities computed here
  independently from float64 softmax and a probability sort;
* limits: small T and small top_p give the argmax, ties to the lowest id;
* planted mistakes in the oracle must break one of these pins.
"""

import os

import numpy as np
import pytest

from oracle import sampling as osm

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "sampling_worked_example.txt")
_SAMPLE = osm.sample_top_p
_MASK = osm.nucleus_mask
_MASSES = osm.token_masses


CASES = {"ln1234": np.log(np.array([1, 2, 3, 4], dtype=np.float32)),
         "zeros4": np.zeros(4, dtype=np.float32)}


def worked_example_ok(sample):
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        case, t, p, u, want = line.split()
        if sample(CASES[case], float(t), float(p), float(u)) != int(want):
            return False
    return True


def frequencies_ok(sample, temperature, top_p, n=4000, seed=0, vocab=40):
    """Stratified u_i = (i + 1/2)/n hits token v about n * p_v times (within 1)."""
    z = (np.random.default_rng(seed).standard_normal(vocab) * 2.0).astype(np.float32)
    p = np.exp((z.astype(np.float64) - z.max()) / np.float32(temperature))
    p /= p.sum()
    order = np.argsort(-p, kind="stable")
    k = int(np.searchsorted(np.cumsum(p[order]), top_p - 1e-12)) + 1
    keep = np.zeros(vocab, dtype=bool)
    keep[order[:k]] = True
    want = np.where(keep, p, 0.0)
    want /= want.sum()
    counts = np.zeros(vocab)
    for i in range(n):
        counts[sample(z, temperature, top_p, (i + 0.5) / n)] += 1
    return bool(np.all(np.abs(counts - n * want) <= 1.0 + 1e-6))


def test_worked_example():
    assert worked_example_ok(_SAMPLE)


@pytest.mark.parametrize("temperature,top_p", [(1.0, 1.0), (0.7, 1.0), (1.3, 0.9), (0.8, 0.6)])
def test_stratified_frequencies(temperature, top_p):
    assert frequencies_ok(_SAMPLE, temperature, top_p)


def test_limits_give_argmax_with_lowest_tie():
    rng = np.random.default_rng(5)
    z = rng.standard_normal(1000).astype(np.float32)
    best = int(np.argmax(z))
    for u in (0.0, 0.3, 0.999):
        assert _SAMPLE(z, 1e-4, 1.0, u) == best
        assert _SAMPLE(z, 1.0, 1e-7, u) == best
    z[[17, 400, 800]] = z.max() + 1.0  # a three-way tie at the top
    for u in (0.0, 0.5, 0.999):
        assert _SAMPLE(z, 1.0, 1e-7, u) == 17
        assert _SAMPLE(z, 1e-4, 1.0, u) in (17, 400, 800)


def test_masses_and_clamping():
    q = _MASSES(np.array([0.0, -np.inf, 0.0, -1e9], np.float32), 1.0)
    assert list(q) == [1 << 40, 0, 1 << 40, 0]
    z = np.log(np.array([1, 3], np.float32))
    assert _SAMPLE(z, 1.0, 1.0, -0.5) == 0 and _SAMPLE(z, 1.0, 1.0, 1.5) == 1


# ------------------------------------------------------------- planted mistakes

def _mutant_ascending(z, temperature, top_p, u):
    """Nucleus built from the least likely tokens first."""
    q = _MASSES(z, temperature)
    order = np.lexsort((np.arange(q.size), q.astype(np.int64)))  # q ascending
    need = -((-int(np.rint(top_p * 2 ** 24)) * int(q.sum())) // (1 << 24))
    cum = np.cumsum(q[order].astype(object))
    mask = np.zeros(q.size, dtype=bool)
    mask[order[:int(np.argmax(cum >= need)) + 1]] = True
    return _sample_with_mask(q, mask, u)


def _sample_with_mask(q, mask, u):
    members = np.nonzero(mask)[0]
    Z = int(sum(int(x) for x in q[members]))
    target = (int(np.floor(np.float32(min(max(u, 0.0), 0.99999994)) * 2 ** 24)) * Z) >> 24
    run = 0
    for v in members:
        run += int(q[v])
        if run > target:
            return int(v)
    return int(members[-1])


def _mutant_temperature_multiplies(z, temperature, top_p, u):
    return _SAMPLE(z, 1.0 / temperature, top_p, u)


def _mutant_drops_crossing_token(z, temperature, top_p, u):
    q = _MASSES(z, temperature)
    mask = _MASK(q, top_p)
    order = np.lexsort((np.arange(q.size), -q.astype(np.int64)))
    last = [v for v in order if mask[v]][-1]
    if mask.sum() > 1:
        mask[last] = False
    return _sample_with_mask(q, mask, u)


def _mutant_greater_equal(z, temperature, top_p, u):
    q = _MASSES(z, temperature)
    mask = _MASK(q, top_p)
    members = np.nonzero(mask)[0]
    Z = int(sum(int(x) for x in q[members]))
    target = (int(np.floor(np.float32(u) * 2 ** 24)) * Z) >> 24
    run = 0
    for v in members:
        run += int(q[v])
        if run >= target:
            return int(v)
    return int(members[-1])


@pytest.mark.parametrize("mutant", [_mutant_ascending, _mutant_temperature_multiplies,
                                    _mutant_drops_crossing_token, _mutant_greater_equal])
def test_planted_mistakes_break_a_pin(mutant):
    caught = (not worked_example_ok(mutant)
              or not frequencies_ok(mutant, 0.7, 1.0)
              or not frequencies_ok(mutant, 1.3, 0.9))
    assert caught
