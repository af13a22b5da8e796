"""CPU oracle of the batched paged decode step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or links
anything in this package: only the tests, the smoke check and the benchmark's
CPU-baseline leg may use it.  It shares no code with the HIP kernels, the C ABI
or the Python binding.

It is a plain, slow, float64 (optionally float32 for timing) numpy rendering of
one Llama-style pre-norm decoder step over a batch of trajectories, each with
its own contiguous KV history, plus the paged-gather form of decode attention.
The paper runs this computation inside its inference backend without
specifying it (Introduction; Design Principles, specialization in
heterogeneous pools: each step reads the weights once for the active batch
and each trajectory's own KV history).  Every reading the paper leaves open
(architecture family, RoPE convention, GQA grouping, positions) is listed in
the module docstrings below.
"""

from .decoder import (Decoder, ModelWeights, attention, greedy, recompute_logits, rmsnorm,
                      rope, silu)
from .paged import gather_pages, paged_decode_attention
from .sampling import nucleus_mask, sample_top_p, token_masses
from .fp8 import e4m3_decode, e4m3_encode, paged_decode_attention_fp8, quantize_dequantize
from .pacing import footprint, pacing_plan

__all__ = [
    "Decoder", "ModelWeights", "attention", "greedy", "recompute_logits", "rmsnorm", "rope",
    "silu", "gather_pages", "paged_decode_attention", "nucleus_mask", "sample_top_p",
    "token_masses", "e4m3_decode", "e4m3_encode", "quantize_dequantize",
    "paged_decode_attention_fp8", "footprint", "pacing_plan",
]
