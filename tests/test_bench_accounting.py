"""bench.py's algorithmic byte and flop accounting against independent counts.

The reported rooflines divide these counts by measured time, so a dropped
matrix or a doubled term would shift every reported fraction.  They are
checked against the sizes of the 8B-shaped decoder written out matrix by
matrix (15.01 GB of weights streamed per step besides the gathered embedding
rows), and against brute-force enumeration of the causal (query, key) pairs
on small inputs.
"""

import bench
from workload import EIGHT_B, TINY


def _matrices(shape):
    """(rows, cols) of every projection matrix of one layer, listed one by one."""
    d, qd, kvd, f = shape.d_model, shape.n_q_heads * shape.head_dim, \
        shape.n_kv_heads * shape.head_dim, shape.ffn_dim
    return [(qd, d), (kvd, d), (kvd, d), (d, qd), (f, d), (f, d), (d, f)]


def test_weight_bytes_per_step_8b():
    per_layer = sum(r * c for r, c in _matrices(EIGHT_B))
    assert per_layer == 4096 * 4096 * 2 + 1024 * 4096 * 2 + 14336 * 4096 * 3
    for batch in (1, 16, 256):
        want = 2 * (32 * per_layer + 128256 * 4096 + batch * 4096)
        assert bench.weight_bytes_per_step(EIGHT_B, batch) == want
    assert abs(bench.weight_bytes_per_step(EIGHT_B, 0) / 1e9 - 15.01) < 0.005


def test_prefill_flops_by_enumeration():
    for shape in (TINY, EIGHT_B):
        macs_per_token = shape.n_layers * sum(r * c for r, c in _matrices(shape))
        for n in (1, 2, 3, 7, 16):
            pairs = sum(1 for q in range(n) for k in range(n) if k <= q)
            # q.k and p.v: head_dim multiply-adds each, per pair, head and layer
            attn_macs = shape.n_layers * shape.n_q_heads * pairs * 2 * shape.head_dim
            assert bench.prefill_flops(shape, n) == 2 * (n * macs_per_token + attn_macs)


def test_prefill_flops_8b_magnitudes():
    # 4K tokens: 57.2 TFLOP of projections and 4.4 TFLOP of attention.
    assert abs(bench.prefill_flops(EIGHT_B, 4096) / 1e12 - 61.57) < 0.01
    # 64K tokens: the attention share overtakes the projections.
    n = 65536
    proj = 2.0 * n * EIGHT_B.n_layers * sum(r * c for r, c in _matrices(EIGHT_B))
    assert bench.prefill_flops(EIGHT_B, n) - proj > proj


def test_append_flops_by_enumeration():
    """Appending n tokens onto ctx0 cached ones: every new query sees the
    cached keys and the new keys up to itself."""
    for shape in (TINY, EIGHT_B):
        macs_per_token = shape.n_layers * sum(r * c for r, c in _matrices(shape))
        for ctx0, n in ((0, 5), (3, 1), (17, 4), (100, 9)):
            pairs = sum(1 for q in range(ctx0, ctx0 + n) for k in range(ctx0 + n) if k <= q)
            attn_macs = shape.n_layers * shape.n_q_heads * pairs * 2 * shape.head_dim
            assert bench.append_flops(shape, ctx0, n) == 2 * (n * macs_per_token + attn_macs)
        assert bench.append_flops(shape, 0, 12) == bench.prefill_flops(shape, 12)
