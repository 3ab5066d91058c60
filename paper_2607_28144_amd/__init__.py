"""MI355X (gfx950) window attention for a real-time generative video decoder.

Exact non-causal softmax attention for one GPU's share of a sequence-parallel
video diffusion transformer, its per-chunk partials and log-sum-exp merge,
cross-attention to conditioning tokens, and the q/k RMSNorm + 3D rotary
embedding that produce the attention inputs (plus a ring step that merges a
chunk's result straight into the running output) -- hand-written HIP kernels behind
a C ABI (include/regenvc_attn.h).  Import is cheap: the library and torch are
loaded on first use.
"""

__all__ = ["attn_fwd", "attn_partial_fwd", "lse_merge", "attn_ring_accumulate", "cross_attn_fwd",
           "cross_attn_dual_fwd", "attn_plan", "qk_norm_rope",
           "RegenvcError"]


def __getattr__(name):
    if name in __all__:
        from . import api
        return getattr(api, name)
    raise AttributeError(name)
