"""Temperature / nucleus (top-p) sampling (oracle side).

TEST INFRASTRUCTURE ONLY (see the package docstring).

RL rollouts sample their actions (Background, "RL Post-Training Workflow");
the paper does not state the sampler, so the library defines the common
temperature + top-p rule with exact integer decisions after one exponential,
and this oracle writes that definition out step by step:

1. e_v = exp((z_v - max z) * (1/T)) in float64, with z the float32 logits.
2. q_v = rint(e_v * 2^40): an integer mass per token; S = sum_v q_v.
3. The nucleus is the shortest prefix of the tokens ordered by q descending,
   ties by lower index, whose mass reaches ceil(p24 * S / 2^24), where
   p24 = rint(top_p * 2^24) (at least 1).
4. With u in [0, 1) (clamped), u24 = floor(u * 2^24), Z = the nucleus mass,
   target = floor(u24 * Z / 2^24): the sampled token is the first nucleus
   token in index order whose running nucleus mass exceeds target.

With top_p = 1 this is inverse-CDF sampling of softmax(z / T) (up to the
2^-40 quantisation of the masses); listing the nucleus in index order rather
than by probability changes which u maps to which token, not the
distribution.
"""

from __future__ import annotations

import numpy as np

_ONE_BELOW = float(np.nextafter(np.float32(1.0), np.float32(0.0)))


def token_masses(z, temperature: float) -> np.ndarray:
    """Steps 1-2: integer masses q_v (uint64) of a float32 logit row."""
    z = np.asarray(z, dtype=np.float32).astype(np.float64)
    inv_t = 1.0 / np.float64(np.float32(temperature))
    e = np.exp((z - z.max()) * inv_t)
    return np.rint(e * 2.0 ** 40).astype(np.uint64)


def nucleus_mask(q: np.ndarray, top_p: float) -> np.ndarray:
    """Step 3: boolean mask of the nucleus."""
    total = int(q.sum(dtype=np.uint64))
    p24 = int(np.rint(np.float64(np.float32(top_p)) * 2.0 ** 24))
    p24 = min(max(p24, 1), 1 << 24)
    need = -((-p24 * total) // (1 << 24))  # ceil
    order = np.lexsort((np.arange(q.size), -q.astype(np.int64)))  # q desc, index asc
    cum = np.cumsum(q[order].astype(object))
    k = int(np.argmax(cum >= need))  # first prefix reaching the mass
    mask = np.zeros(q.size, dtype=bool)
    mask[order[:k + 1]] = True
    return mask


def sample_top_p(z, temperature: float, top_p: float, u: float) -> int:
    """Step 4: the sampled token id of one logit row."""
    q = token_masses(z, temperature)
    mask = nucleus_mask(q, top_p)
    members = np.nonzero(mask)[0]  # ascending index order
    mass = q[members].astype(object)
    Z = int(sum(mass))
    u = min(max(float(np.float32(u)), 0.0), _ONE_BELOW)
    u24 = int(np.floor(np.float32(u) * np.float32(2.0 ** 24)))
    target = (u24 * Z) >> 24
    run = 0
    for v, m in zip(members, mass):
        run += int(m)
        if run > target:
            return int(v)
    raise AssertionError("target beyond the nucleus mass")
