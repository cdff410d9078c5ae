"""Attention-interaction cost model (App. C) and visible-pair counts.

One unit per query-key interaction (App. C, derivation paragraph).  With
S = N_X + N_LT:
  C_pre  = (N_R + N_ST)^2          (Eq. cost-pre)
  C_step = S (N_R + S)             (Eq. cost-step)
  C_ours = C_pre + T C_step        (Eq. cost-ours)
  C_full = T (N_R + S)^2
  R(N_R) = C_full / C_ours         (Eq. speedup)
  R ~= T N_R / (N_R + T S)         (large-context approximation)
and the anchor overhead over an isolated cache is 2 N_R N_ST + N_ST^2 (Eq. 4).
"""
from __future__ import annotations

from typing import Sequence

from .masks import LIVE_KINDS, STATIC_KINDS, Mask


def c_pre(n_r, n_st):
    return (n_r + n_st) ** 2


def c_step(n_r, s):
    return s * (n_r + s)


def c_full(n_r, s, T):
    return T * (n_r + s) ** 2


def c_ours(n_r, n_st, s, T):
    return c_pre(n_r, n_st) + T * c_step(n_r, s)


def speedup(n_r, n_st, s, T):
    return c_full(n_r, s, T) / c_ours(n_r, n_st, s, T)


def speedup_large_context(n_r, s, T):
    return T * n_r / (n_r + T * s)


def anchor_overhead(n_r, n_st):
    return 2 * n_r * n_st + n_st ** 2


def visible_pairs(kinds: Sequence[int], lens: Sequence[int], vis: Mask, rows: str) -> int:
    """Visible query-key pairs per (batch, head) for the rows of one entry:
    rows = 'static' (prefill), 'live' (step) or 'all' (full recompute)."""
    pick = {"static": lambda kk: kk in STATIC_KINDS,
            "live": lambda kk: kk in LIVE_KINDS,
            "all": lambda kk: True}[rows]
    total = 0
    for qi, qk in enumerate(kinds):
        if pick(qk):
            total += lens[qi] * sum(lens[ki] for ki in range(len(kinds)) if vis[qi][ki])
    return total
