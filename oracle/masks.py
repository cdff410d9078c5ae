"""Block masks over the segmented in-context sequence.

Notation (Sec. 3.1, Eq. 1; Sec. 3.3): ST static text anchors, LT live text,
X denoising target, R^(k) the k-th reference.  A mask here is a boolean
matrix ``vis[q][k]`` over *segments*: True when the tokens of query segment
q attend to the tokens of key segment k.  (App. A writes the transpose,
M[b', b] = 1 meaning b attends to b'; this module is query-first.)

Kinds are the integers 0=ST, 1=LT, 2=X, 3=R.
"""
from __future__ import annotations

from typing import List, Sequence

ST, LT, X, R = 0, 1, 2, 3
STATIC_KINDS = (ST, R)      # fixed during denoising (Sec. 3.3: the static subgraph [ST, R])
LIVE_KINDS = (LT, X)        # change every denoising step

Mask = List[List[bool]]


def paper_mask(kinds: Sequence[int]) -> Mask:
    """The static-text-anchor mask of Sec. 3.3.

    R and ST see each other (both directions) and never receive LT or X;
    the original branch [LT, X_t] keeps its text-target interaction and
    attends to R but not to ST.  All references form one R block (Eq. 1
    concatenates them), so every R segment sees every R segment.
    """
    vis = []
    for qk in kinds:
        if qk in STATIC_KINDS:
            vis.append([kk in STATIC_KINDS for kk in kinds])
        else:
            vis.append([kk in (LT, X, R) for kk in kinds])
    return vis


def perref_mask(kinds: Sequence[int]) -> Mask:
    """Per-reference anchored mask used by the synthetic workloads.

    Reference queries see their own reference segment and the anchors,
    anchor queries see anchors only, text and target queries see every
    segment (anchors included).  It is structurally cacheable like the
    Sec. 3.3 mask: no static query sees LT or X.
    """
    vis = []
    for qi, qk in enumerate(kinds):
        row = []
        for ki, kk in enumerate(kinds):
            if qk == ST:
                row.append(kk == ST)
            elif qk == R:
                row.append(kk == ST or ki == qi)
            else:
                row.append(True)
        vis.append(row)
    return vis


def isolated_mask(kinds: Sequence[int]) -> Mask:
    """Prior-work isolated reference cache (Sec. 1, Sec. 2, Sec. 4.1).

    R is cut off from LT and X and there is no anchor path: R sees R only,
    [LT, X] see LT, X and R.  Anchor segments, if present, are detached:
    they attend to nothing and nobody attends to them, so the prefill
    interaction count is N_R^2 and the Sec. 3.3 mask adds exactly Eq. 4.
    """
    vis = []
    for qk in kinds:
        if qk == ST:
            vis.append([False for _ in kinds])
        elif qk == R:
            vis.append([kk == R for kk in kinds])
        else:
            vis.append([kk in (LT, X, R) for kk in kinds])
    return vis


def dense_mask(kinds: Sequence[int]) -> Mask:
    """Full attention: every segment sees every segment (the paper's Base, App. C)."""
    return [[True for _ in kinds] for _ in kinds]


def live_text_mask(kinds: Sequence[int]) -> Mask:
    """A mask on the original token set where R also reads live text.

    Used only as the negative control of Sec. 3.2 / Eq. 3: it opens the
    path X -> LT -> R, so R is not exactly cacheable.
    """
    vis = []
    for qk in kinds:
        if qk == R:
            vis.append([kk in (LT, R) for kk in kinds])
        elif qk == ST:
            vis.append([kk == ST for kk in kinds])
        else:
            vis.append([kk in (LT, X, R) for kk in kinds])
    return vis


PRESETS = {
    "paper": paper_mask,
    "perref": perref_mask,
    "isolated": isolated_mask,
    "dense": dense_mask,
}


def is_cacheable(kinds: Sequence[int], vis: Mask) -> bool:
    """No static query segment reads a live key segment (single-layer form
    of StructCacheable, App. A: with a layer-shared mask every path from X
    into R must enter the static set through such an edge)."""
    for qi, qk in enumerate(kinds):
        if qk in STATIC_KINDS:
            for ki, kk in enumerate(kinds):
                if vis[qi][ki] and kk in LIVE_KINDS:
                    return False
    return True


def cached_segments(kinds: Sequence[int], vis: Mask) -> List[int]:
    """Static segments whose K/V some live query reads, in sequence order:
    these are what the reference K/V cache holds (Eq. 2; Sec. 3.3)."""
    out = []
    for ki, kk in enumerate(kinds):
        if kk in STATIC_KINDS and any(vis[qi][ki] for qi, qk in enumerate(kinds) if qk in LIVE_KINDS):
            out.append(ki)
    return out
