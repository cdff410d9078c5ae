"""Unrolled layered dependency graph of App. A.

Nodes are (block, layer) for layer 0..L; edges are residual
(b, l-1) -> (b, l) and attention (b', l-1) -> (b, l) whenever b attends b'
(``vis[b][b']`` in this package's query-first convention).
"""
from __future__ import annotations

from typing import Sequence, Set, Tuple

from .masks import Mask


def reachable_from(vis: Mask, start_block: int, start_layer: int, L: int) -> Set[Tuple[int, int]]:
    """All nodes (b, l) reachable by a directed path from (start_block, start_layer)."""
    n = len(vis)
    seen = {(start_block, start_layer)}
    frontier = {start_block}
    for layer in range(start_layer + 1, L + 1):
        nxt = set(frontier)                       # residual edges
        for b in range(n):
            if any(vis[b][bp] for bp in frontier):  # attention edges
                nxt.add(b)
        for b in nxt:
            seen.add((b, layer))
        frontier = nxt
    return seen


def struct_cacheable(vis: Mask, x_blocks: Sequence[int], r_blocks: Sequence[int], L: int) -> bool:
    """No path (X, 0) ~> (R, l) for any l in 1..L (App. A, StructCacheable)."""
    for xb in x_blocks:
        reach = reachable_from(vis, xb, 0, L)
        if any((rb, l) in reach for rb in r_blocks for l in range(1, L + 1)):
            return False
    return True


def live_text_reachable(vis: Mask, lt_blocks: Sequence[int], r_blocks: Sequence[int], L: int) -> bool:
    """(LT, l) ~> (R, m) for some 1 <= l < m <= L (App. A, LiveTextReachable)."""
    for lb in lt_blocks:
        for layer in range(1, L):
            reach = reachable_from(vis, lb, layer, L)
            if any((rb, m) in reach for rb in r_blocks for m in range(layer + 1, L + 1)):
                return True
    return False
