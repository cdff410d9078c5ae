"""MI355X (gfx950) implementation of the exact-reference-caching attention
path of arXiv 2608.21229: block-masked attention over
[static text anchors | live text | target | references], with a
once-per-request reference K/V prefill, per-step masked attention over fresh
plus cached K/V, and a full-recompute baseline.

The compute lives in ``librefcache.so`` (hand-written HIP, C ABI declared in
``include/refcache.h``); ``binding`` is its ctypes wrapper and ``chain``
drives a stack of synthetic layers (projection, attention, projection plus
residual) through it.
"""
from .binding import (  # noqa: F401
    Layout, RcError, lib, ref_kv_prefill, step_masked_attention, step_masked_attention_noalloc, full_attention,
    linear, NOALLOC_SCRATCH_BYTES,
    ref_kv_prefill_fp8, step_masked_attention_fp8, fp8_cache_shapes,
    SEG_ANCHOR, SEG_TEXT, SEG_TARGET, SEG_REF,
    MASK_PAPER, MASK_PERREF, MASK_ISOLATED, MASK_DENSE, MASKS,
    ENTRY_PREFILL, ENTRY_STEP, ENTRY_FULL,
    ROWS_STATIC, ROWS_LIVE, ROWS_CACHED, ROWS_ALL, SPLITS_BALANCED, SPLITS_TAIL, SPLITS_LAST_ROUND,
    RC_OK, RC_ERR_ARG, RC_ERR_UNSUPPORTED, RC_ERR_MASK_NOT_CACHEABLE, RC_ERR_WORKSPACE, RC_ERR_HIP,
)
from .chain import Chain  # noqa: F401,E402
