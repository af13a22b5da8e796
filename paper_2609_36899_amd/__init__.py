"""MI355X (gfx950) batched paged decode: HIP kernels behind a C ABI.

The compiled library (libpdec.so, see include/pdec.h) holds every kernel;
this package only builds it (``build``) and marshals torch tensors into its
calls (``engine``).
"""

from ._native import PAGE_TOKENS, PdecError, BF16, F32, FP8_E4M3  # noqa: F401


def __getattr__(name):
    # The torch-facing binding is imported lazily so that host-only tooling
    # (build, ABI checks) does not pay for importing torch.
    if name in ("Engine", "paged_decode_attention", "paged_attention_workspace_bytes",
                "kv_bytes_per_token", "weights_to_device", "model_cfg", "weight_projection",
                "weight_projection_workspace_bytes", "pack_weight", "swiglu_projection",
                "swiglu_projection_workspace_bytes",
                "PackedWeight", "sample_top_p", "sample_top_p_workspace_bytes",
                "paged_decode_attention_fp8"):
        from . import engine
        return getattr(engine, name)
    if name in ("PacedRollout", "pacing_plan"):
        from . import driver
        return getattr(driver, name)
    raise AttributeError(name)
