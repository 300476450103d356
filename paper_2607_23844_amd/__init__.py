"""OmniCache cached attention layer for MI355X (gfx950).

Token / Frame / Block Cache around one attention layer of a diffusion
denoiser (OmniCache §3.2-§3.3): cosine-similarity matching against
deterministic representatives, the most redundant items skipped, reduced
attention over the retained tokens on MFMA, cached activations restored at
their original positions.  Every step runs in the HIP library liboc.so
(C ABI in include/oc.h); this package only marshals torch tensors.  There is
no CPU fallback: a missing library raises OmniCacheError on first use.
"""
from ._lib import LIB_PATH, OmniCacheError, lib  # noqa: F401
from .api import (  # noqa: F401
    Cfg,
    LayerCache,
    PlanInfo,
    Shape,
    StageTimer,
    attn_full,
    block_cached,
    block_workspace,
    clock_ghz,
    clock_sample,
    attn_reduced,
    attn_workspace_bytes,
    ffn_reduced,
    ffn_workspace_bytes,
    gather,
    layer_cached,
    layer_cached_static,
    layered_schedule,
    match,
    plan,
    residual_add,
    restore,
    select,
    static_scratch_bytes,
    workspace,
)
