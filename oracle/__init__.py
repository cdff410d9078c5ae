"""Oracle for the exact-reference-caching attention path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import anything from this package.  It is a plain, slow,
fp64 CPU statement of what the GPU library computes, written from the paper
(arXiv 2608.21229) and sharing no code, table or helper with the HIP path.

Modules
-------
masks      block masks over the segmented sequence (Sec. 3.3, App. A)
attention  masked softmax attention and the prefill / step / full-recompute
           row subsets built on it (Eq. 2, Sec. 3.3, App. C)
cost       the attention-interaction cost model (App. C, Eq. 4)
graph      the unrolled layered dependency graph of App. A (Theorem 1)
chain      chained synthetic layers (projection -> attention -> projection +
           residual) with bf16 storage points (Eq. 2 across layers)
fp8        the e4m3fn reference cache: rounding, power-of-two scales,
           quantise / dequantise

Pinning: every function here is checked in ``tests/test_oracle*.py``
against values that do not come from this package (an mpmath brute force,
torch's fp64 scaled_dot_product_attention and its float8/bfloat16
conversions, closed forms, the paper's printed numbers and equations).  No function is "parity unpinned".
"""
