"""Masked softmax attention in float64 -- the oracle's statement of the path.

What the method computes is exact (Sec. 3.1 "Exact reference caching",
Eq. 2; Sec. 3.3): with a structurally cacheable mask, attention over the
whole segmented sequence, recomputed from scratch, gives the same result as
(i) a once-per-request prefill over the static subgraph [ST, R] that also
stores the reference K/V, followed by (ii) per-step attention of the live
rows [LT, X_t] over fresh LT/X K/V plus the stored K/V (App. C, derivation
paragraph).  So the oracle is one plain definition -- softmax(Q K^T * scale) V
restricted, per query segment, to the visible key segments -- and each entry
point is a subset of its rows with the keys taken from a different buffer.

Arrays are numpy float64 ``[B, N, H, D]`` (token-major, like a fused QKV
projection output).  bf16 inputs convert to float64 exactly.
Rows with no visible key get O = 0 and lse = -inf (a convention; the
paper's masks always leave at least one key).
"""
from __future__ import annotations

from typing import List, Optional, Sequence, Tuple

import numpy as np

from .masks import LIVE_KINDS, STATIC_KINDS, Mask, cached_segments, is_cacheable

ROW_CHUNK = 1024   # rows per numpy matmul; bounds memory only, rows are independent


def softmax_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float):
    """One head: q [n, D], k [m, D], v [m, D] -> (O [n, D], lse [n]).

    O_i = sum_j exp(s_ij - m_i) v_j / sum_j exp(s_ij - m_i), s_ij = scale * q_i.k_j,
    m_i = max_j s_ij, lse_i = m_i + log sum_j exp(s_ij - m_i).
    """
    n, D = q.shape
    if k.shape[0] == 0:
        return np.zeros((n, v.shape[1])), np.full(n, -np.inf)
    s = (q @ k.T) * scale
    m = s.max(axis=1, keepdims=True)
    w = np.exp(s - m)
    l = w.sum(axis=1, keepdims=True)
    o = (w @ v) / l
    return o, m[:, 0] + np.log(l[:, 0])


def _attend(q: np.ndarray, keys: List[Tuple[np.ndarray, np.ndarray]], scale: float, Dv: int):
    """q [B, n, H, D]; keys: (K, V) blocks [B, m_i, H, D] / [B, m_i, H, Dv] in sequence order."""
    B, n, H, D = q.shape
    if keys:
        K = np.concatenate([kk for kk, _ in keys], axis=1)
        V = np.concatenate([vv for _, vv in keys], axis=1)
    else:
        K = np.zeros((B, 0, H, D))
        V = np.zeros((B, 0, H, Dv))
    O = np.zeros((B, n, H, Dv))
    lse = np.zeros((B, H, n))
    for b in range(B):
        for h in range(H):
            kbh = K[b, :, h, :]
            vbh = V[b, :, h, :]
            for r0 in range(0, n, ROW_CHUNK):
                r1 = min(n, r0 + ROW_CHUNK)
                o, ls = softmax_attention(q[b, r0:r1, h, :], kbh, vbh, scale)
                O[b, r0:r1, h, :] = o
                lse[b, h, r0:r1] = ls
    return O, lse


def _offsets(lens: Sequence[int], members: Sequence[int]):
    """Start of each member segment inside a buffer holding only the members, in order."""
    off, pos = {}, 0
    for i in members:
        off[i] = pos
        pos += lens[i]
    return off, pos


def _run(kinds, lens, vis: Mask, row_segs, q_buf, q_off, key_of, scale, rows, Dv):
    """Evaluate rows of the query segments ``row_segs``.

    ``q_buf`` holds the rows of ``row_segs`` in order (offsets ``q_off``);
    ``key_of(seg)`` returns that key segment's (K, V) rows.  ``rows`` (optional)
    lists row indices inside ``q_buf`` to evaluate.
    """
    B, N, H, D = q_buf.shape
    want = np.arange(N) if rows is None else np.asarray(rows, dtype=np.int64)
    outs_O, outs_lse, outs_rows = [], [], []
    for qs in row_segs:
        lo, hi = q_off[qs], q_off[qs] + lens[qs]
        sel = want[(want >= lo) & (want < hi)]
        if sel.size == 0:
            continue
        keys = [key_of(ks) for ks in range(len(kinds)) if vis[qs][ks]]
        O, lse = _attend(q_buf[:, sel], keys, scale, Dv)
        outs_O.append(O)
        outs_lse.append(lse)
        outs_rows.append(sel)
    if not outs_rows:
        return np.zeros((B, 0, H, Dv)), np.zeros((B, H, 0)), want[:0]
    O = np.concatenate(outs_O, axis=1)
    lse = np.concatenate(outs_lse, axis=2)
    r = np.concatenate(outs_rows)
    order = np.argsort(r, kind="stable")
    return O[:, order], lse[:, :, order], r[order]


def full_attention(kinds, lens, vis: Mask, q, k, v, scale: float, rows=None):
    """Every row of the whole sequence under ``vis`` (the recompute baseline;
    with the dense mask over [LT, X, R] it is the paper's Base, App. C).

    Returns (O [B, n, H, D], lse [B, H, n], row indices)."""
    segs = list(range(len(kinds)))
    off, total = _offsets(lens, segs)
    assert q.shape[1] == total and k.shape[1] == total and v.shape[1] == total
    key_of = lambda s: (k[:, off[s]:off[s] + lens[s]], v[:, off[s]:off[s] + lens[s]])
    return _run(kinds, lens, vis, segs, q, off, key_of, scale, rows, v.shape[3])


def static_segments(kinds) -> List[int]:
    return [i for i, kk in enumerate(kinds) if kk in STATIC_KINDS]


def live_segments(kinds) -> List[int]:
    return [i for i, kk in enumerate(kinds) if kk in LIVE_KINDS]


def reference_prefill(kinds, lens, vis: Mask, q_s, k_s, v_s, scale: float, rows=None):
    """Static-subgraph prefill (Sec. 3.3): rows of the ST and R segments,
    attending only to static keys, plus the K/V cache.

    q_s, k_s, v_s hold the static segments' tokens in sequence order.  The
    cache is ``[B, H, N_cached, D]``: the K and V rows of the segments that
    some live query reads (``masks.cached_segments``), in sequence order --
    an exact copy of the inputs, since Eq. 2's projections are given.

    Returns (O_s, lse_s, row indices, K_cache, V_cache)."""
    if not is_cacheable(kinds, vis):
        raise ValueError("mask lets a static query read a live segment: not cacheable")
    st = static_segments(kinds)
    off, total = _offsets(lens, st)
    assert q_s.shape[1] == total and k_s.shape[1] == total and v_s.shape[1] == total
    key_of = lambda s: (k_s[:, off[s]:off[s] + lens[s]], v_s[:, off[s]:off[s] + lens[s]])
    O, lse, r = _run(kinds, lens, vis, st, q_s, off, key_of, scale, rows, v_s.shape[3])
    cs = cached_segments(kinds, vis)
    if cs:
        kc = np.concatenate([k_s[:, off[s]:off[s] + lens[s]] for s in cs], axis=1)
        vc = np.concatenate([v_s[:, off[s]:off[s] + lens[s]] for s in cs], axis=1)
    else:
        B, _, H, D = k_s.shape
        kc = np.zeros((B, 0, H, D))
        vc = np.zeros((B, 0, H, v_s.shape[3]))
    return O, lse, r, np.ascontiguousarray(kc.transpose(0, 2, 1, 3)), np.ascontiguousarray(vc.transpose(0, 2, 1, 3))


def denoise_step(kinds, lens, vis: Mask, q_l, k_l, v_l, k_cache, v_cache, scale: float, rows=None):
    """Per-step attention (App. C): rows of LT and X attend to fresh LT/X
    keys (k_l, v_l, in sequence order) and to the cached static keys
    (``[B, H, N_cached, D]``).  Returns (O_l, lse_l, row indices)."""
    if not is_cacheable(kinds, vis):
        raise ValueError("mask lets a static query read a live segment: not cacheable")
    lv = live_segments(kinds)
    off_l, total_l = _offsets(lens, lv)
    cs = cached_segments(kinds, vis)
    off_c, total_c = _offsets(lens, cs)
    assert q_l.shape[1] == total_l and k_l.shape[1] == total_l
    assert k_cache.shape[2] == total_c and v_cache.shape[2] == total_c

    def key_of(s):
        if s in off_l:
            return k_l[:, off_l[s]:off_l[s] + lens[s]], v_l[:, off_l[s]:off_l[s] + lens[s]]
        a, b = off_c[s], off_c[s] + lens[s]
        return k_cache[:, :, a:b].transpose(0, 2, 1, 3), v_cache[:, :, a:b].transpose(0, 2, 1, 3)

    return _run(kinds, lens, vis, lv, q_l, off_l, key_of, scale, rows, v_l.shape[3])
