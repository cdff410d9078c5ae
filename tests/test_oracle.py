"""Pins for the fp64 oracle: none of the expected values below comes from the
oracle itself.  They come from an mpmath brute force, from torch's fp64
scaled_dot_product_attention (a library routine), from closed forms, from
algebraic identities of softmax attention, and from the structure the paper
states (Sec. 3.1-3.3, App. A)."""
import itertools
import math

import mpmath
import numpy as np
import pytest
import torch

from oracle import attention as oa
from oracle import masks as om

ST, LT, X, R = om.ST, om.LT, om.X, om.R
TINY_KINDS = [ST, LT, X, R, R]
TINY_LENS = [2, 3, 4, 3, 2]


def rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def token_mask(kinds, lens, vis):
    """Expand a segment mask to tokens: T[i, j] True when token i attends token j."""
    seg = np.concatenate([[s] * n for s, n in enumerate(lens)])
    return np.array([[vis[seg[i]][seg[j]] for j in range(len(seg))] for i in range(len(seg))])


def brute_force(q, k, v, tmask, scale):
    """50-digit mpmath masked softmax attention, one row at a time."""
    mpmath.mp.dps = 50
    B, N, H, D = q.shape
    O = np.zeros((B, N, H, v.shape[3]))
    lse = np.zeros((B, H, N))
    for b, h, i in itertools.product(range(B), range(H), range(N)):
        js = [j for j in range(N) if tmask[i, j]]
        if not js:
            lse[b, h, i] = -np.inf
            continue
        s = [mpmath.mpf(scale) * mpmath.fsum(mpmath.mpf(q[b, i, h, d]) * mpmath.mpf(k[b, j, h, d]) for d in range(D)) for j in js]
        e = [mpmath.exp(x) for x in s]
        z = mpmath.fsum(e)
        for d in range(v.shape[3]):
            O[b, i, h, d] = float(mpmath.fsum(e[t] * mpmath.mpf(v[b, js[t], h, d]) for t in range(len(js))) / z)
        lse[b, h, i] = float(mpmath.log(z))
    return O, lse


@pytest.mark.parametrize("preset", ["paper", "perref", "isolated", "dense"])
def test_full_vs_mpmath_brute_force(preset):
    vis = om.PRESETS[preset](TINY_KINDS)
    N = sum(TINY_LENS)
    B, H, D = 2, 2, 5
    q, k, v = rand((B, N, H, D), 1, 1.3), rand((B, N, H, D), 2, 1.1), rand((B, N, H, D + 2), 3)
    scale = 0.7
    O, lse, rows = oa.full_attention(TINY_KINDS, TINY_LENS, vis, q, k, v, scale)
    assert list(rows) == list(range(N))
    Ob, lseb = brute_force(q, k, v, token_mask(TINY_KINDS, TINY_LENS, vis), scale)
    np.testing.assert_allclose(O, Ob, rtol=0, atol=1e-12)
    fin = np.isfinite(lseb)
    assert np.array_equal(fin, np.isfinite(lse))
    np.testing.assert_allclose(lse[fin], lseb[fin], rtol=0, atol=1e-12)
    if preset == "isolated":  # anchors are detached: no visible key
        assert np.all(O[:, :2] == 0) and np.all(np.isneginf(lse[:, :, :2]))


@pytest.mark.parametrize("preset", ["paper", "perref", "isolated", "dense"])
def test_full_vs_torch_sdpa_fp64(preset):
    kinds = [ST, LT, X, R, R, R]
    lens = [5, 11, 37, 23, 16, 9]
    vis = om.PRESETS[preset](kinds)
    N = sum(lens)
    B, H, D = 2, 3, 16
    q, k, v = rand((B, N, H, D), 4), rand((B, N, H, D), 5), rand((B, N, H, D), 6)
    scale = 1 / math.sqrt(D)
    O, lse, _ = oa.full_attention(kinds, lens, vis, q, k, v, scale)
    tm = torch.from_numpy(token_mask(kinds, lens, vis))
    tq, tk, tv = (torch.from_numpy(a).permute(0, 2, 1, 3) for a in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=tm, scale=scale)
    ref = ref.permute(0, 2, 1, 3).numpy()
    live = tm.any(dim=1).numpy()                 # rows with at least one key
    np.testing.assert_allclose(O[:, live], ref[:, live], rtol=0, atol=1e-12)
    # lse against torch's logsumexp of the masked scores
    s = torch.einsum("bhid,bhjd->bhij", tq, tk) * scale
    s = s.masked_fill(~tm, float("-inf"))
    lse_ref = torch.logsumexp(s, dim=-1).numpy()
    np.testing.assert_allclose(lse[:, :, live], lse_ref[:, :, live], rtol=0, atol=1e-12)


def test_dense_is_plain_sdpa_non_square_heads():
    """Unmasked, with D_v != D and n_q != n_k in every block: a transposed
    operand or swapped K/V would not even have the right shape or value."""
    kinds, lens = [LT, X, R], [3, 8, 13]
    N = sum(lens)
    q, k, v = rand((1, N, 2, 6), 7), rand((1, N, 2, 6), 8), rand((1, N, 2, 3), 9)
    O, _, _ = oa.full_attention(kinds, lens, om.dense_mask(kinds), q, k, v, 0.5)
    tq, tk, tv = (torch.from_numpy(a).permute(0, 2, 1, 3) for a in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, scale=0.5).permute(0, 2, 1, 3).numpy()
    np.testing.assert_allclose(O, ref, rtol=0, atol=1e-13)


def test_closed_forms():
    kinds, lens = TINY_KINDS, TINY_LENS
    N = sum(lens)
    vis = om.perref_mask(kinds)
    tm = token_mask(kinds, lens, vis)
    q, v = rand((1, N, 2, 4), 10), rand((1, N, 2, 4), 11)
    # K = 0: every visible key scores 0 -> O is the mean of the visible V rows, lse = log(count)
    O, lse, _ = oa.full_attention(kinds, lens, vis, q, np.zeros_like(q), v, 0.9)
    for i in range(N):
        js = np.nonzero(tm[i])[0]
        np.testing.assert_allclose(O[0, i], v[0, js].mean(axis=0), rtol=0, atol=1e-14)
        np.testing.assert_allclose(lse[0, :, i], math.log(len(js)), rtol=0, atol=1e-14)
    # constant V = c -> O = c for every row
    O, _, _ = oa.full_attention(kinds, lens, vis, q, rand((1, N, 2, 4), 12), np.full((1, N, 2, 4), -2.5), 0.9)
    np.testing.assert_allclose(O, -2.5, rtol=0, atol=1e-14)
    # single visible key: O is that V row and lse is its score
    kinds1, lens1 = [ST, R], [1, 3]
    vis1 = [[True, False], [True, False]]
    q1, k1, v1 = rand((1, 4, 1, 4), 13), rand((1, 4, 1, 4), 14), rand((1, 4, 1, 4), 15)
    O, lse, _ = oa.full_attention(kinds1, lens1, vis1, q1, k1, v1, 0.3)
    for i in range(4):
        np.testing.assert_allclose(O[0, i, 0], v1[0, 0, 0], rtol=0, atol=1e-15)
        np.testing.assert_allclose(lse[0, 0, i], 0.3 * q1[0, i, 0] @ k1[0, 0, 0], rtol=0, atol=1e-15)


def test_lse_merge_identity():
    """Attention over A u B equals the LSE-weighted merge of A and B (the
    identity that split-KV relies on)."""
    q, k, v = rand((7, 8), 20), rand((50, 8), 21), rand((50, 8), 22)
    O, lse = oa.softmax_attention(q, k, v, 0.4)
    Oa, la = oa.softmax_attention(q, k[:19], v[:19], 0.4)
    Ob, lb = oa.softmax_attention(q, k[19:], v[19:], 0.4)
    M = np.maximum(la, lb)
    wa, wb = np.exp(la - M), np.exp(lb - M)
    np.testing.assert_allclose(O, (wa[:, None] * Oa + wb[:, None] * Ob) / (wa + wb)[:, None], rtol=0, atol=1e-14)
    np.testing.assert_allclose(lse, M + np.log(wa + wb), rtol=0, atol=1e-14)


def test_segment_order_invariance():
    """Results per segment do not depend on where the segment sits in the
    sequence (attention has no positional term once Q/K/V exist)."""
    kinds, lens = [ST, LT, X, R, R], [3, 4, 6, 5, 2]
    N = sum(lens)
    vis = om.perref_mask(kinds)
    q, k, v = rand((1, N, 2, 4), 30), rand((1, N, 2, 4), 31), rand((1, N, 2, 4), 32)
    O, lse, _ = oa.full_attention(kinds, lens, vis, q, k, v, 0.6)
    perm = [3, 1, 4, 0, 2]     # new order of segments
    offs = np.cumsum([0] + lens)
    idx = np.concatenate([np.arange(offs[s], offs[s + 1]) for s in perm])
    kinds2 = [kinds[s] for s in perm]
    lens2 = [lens[s] for s in perm]
    vis2 = [[vis[a][b] for b in perm] for a in perm]
    O2, lse2, _ = oa.full_attention(kinds2, lens2, vis2, q[:, idx], k[:, idx], v[:, idx], 0.6)
    np.testing.assert_allclose(O2, O[:, idx], rtol=0, atol=1e-13)
    np.testing.assert_allclose(lse2, lse[:, :, idx], rtol=0, atol=1e-13)


def _split(kinds, lens, arr):
    offs = np.cumsum([0] + list(lens))
    st = [i for i, kk in enumerate(kinds) if kk in (ST, R)]
    lv = [i for i, kk in enumerate(kinds) if kk in (LT, X)]
    cat = lambda segs: np.concatenate([arr[:, offs[s]:offs[s + 1]] for s in segs], axis=1)
    return cat(st), cat(lv), st, lv


@pytest.mark.parametrize("preset", ["paper", "perref", "isolated"])
def test_prefill_and_step_equal_full_recompute(preset):
    """Exactness (Eq. 2, Sec. 3.3): prefill rows + cache, then step rows from
    fresh live K/V + the cache, equal full recomputation of the same rows."""
    kinds, lens = [ST, LT, X, R, R], [4, 6, 9, 7, 5]
    vis = om.PRESETS[preset](kinds)
    N = sum(lens)
    q, k, v = rand((2, N, 3, 8), 40), rand((2, N, 3, 8), 41), rand((2, N, 3, 8), 42)
    Of, lsef, _ = oa.full_attention(kinds, lens, vis, q, k, v, 0.35)
    qs, ql, st, lv = _split(kinds, lens, q)
    ks, kl, _, _ = _split(kinds, lens, k)
    vs, vl, _, _ = _split(kinds, lens, v)
    Os, lses, _, kc, vc = oa.reference_prefill(kinds, lens, vis, qs, ks, vs, 0.35)
    Ol, lsel, _ = oa.denoise_step(kinds, lens, vis, ql, kl, vl, kc, vc, 0.35)
    _, Of_l, _, _ = _split(kinds, lens, Of)
    Of_s, _, _, _ = _split(kinds, lens, Of)
    np.testing.assert_allclose(Os, Of_s, rtol=0, atol=1e-14)
    np.testing.assert_allclose(Ol, Of_l, rtol=0, atol=1e-14)
    # cache = exact copy of the cached segments' K/V, [B, H, N_c, D]
    offs = np.cumsum([0] + lens)
    cs = om.cached_segments(kinds, vis)
    kc_ref = np.concatenate([k[:, offs[s]:offs[s + 1]] for s in cs], axis=1).transpose(0, 2, 1, 3)
    assert np.array_equal(kc, kc_ref)
    expect_cached = {"paper": [3, 4], "perref": [0, 3, 4], "isolated": [3, 4]}[preset]
    assert cs == expect_cached


@pytest.mark.parametrize("preset", ["paper", "perref", "isolated"])
def test_caching_invariant_bitwise(preset):
    """Redrawing LT/X Q/K/V leaves every ST/R output of a full recompute
    bit-identical under a cacheable mask (Sec. 3.1, exact reference caching)."""
    kinds, lens = [ST, LT, X, R, R], [3, 5, 8, 6, 4]
    vis = om.PRESETS[preset](kinds)
    N = sum(lens)
    q, k, v = rand((1, N, 2, 8), 50), rand((1, N, 2, 8), 51), rand((1, N, 2, 8), 52)
    O1, l1, _ = oa.full_attention(kinds, lens, vis, q, k, v, 0.5)
    live = np.concatenate([np.arange(3, 16)])
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    for a, s in ((q2, 53), (k2, 54), (v2, 55)):
        a[:, live] = rand(a[:, live].shape, s)
    O2, l2, _ = oa.full_attention(kinds, lens, vis, q2, k2, v2, 0.5)
    static = np.r_[0:3, 16:26]
    assert np.array_equal(O1[:, static], O2[:, static])
    assert np.array_equal(l1[:, :, static], l2[:, :, static])
    assert not np.allclose(O1[:, live], O2[:, live])


def test_non_cacheable_masks_rejected():
    kinds, lens = [ST, LT, X, R], [2, 2, 2, 2]
    vis = om.live_text_mask(kinds)
    assert not om.is_cacheable(kinds, vis)
    z = np.zeros((1, 4, 1, 2))
    with pytest.raises(ValueError):
        oa.reference_prefill(kinds, lens, vis, z, z, z, 1.0)
    for p in ("paper", "perref", "isolated", ):
        assert om.is_cacheable(kinds, om.PRESETS[p](kinds))
    assert not om.is_cacheable(kinds, om.dense_mask(kinds))


def _chained(kinds, lens, vis, x_seed, L=3, dm=8, H=2):
    """Toy stack: per layer Q/K/V = h W, h <- h + attn(h) W_o (weights fixed,
    seeded independently of the inputs).  Returns per-layer (K, V)."""
    N = sum(lens)
    rng = np.random.default_rng(1234)
    W = [[rng.standard_normal((dm, dm)) / math.sqrt(dm) for _ in range(4)] for _ in range(L)]
    h = rand((N, dm), 77)
    offs = np.cumsum([0] + lens)
    xs = [s for s, kk in enumerate(kinds) if kk == X][0]
    h[offs[xs]:offs[xs + 1]] = rand((lens[xs], dm), x_seed)
    kvs = []
    for layer in range(L):
        Wq, Wk, Wv, Wo = W[layer]
        qkv = [(h @ Wm).reshape(1, N, H, dm // H) for Wm in (Wq, Wk, Wv)]
        kvs.append((qkv[1].copy(), qkv[2].copy()))
        O, _, _ = oa.full_attention(kinds, lens, vis, *qkv, 1 / math.sqrt(dm // H))
        h = h + O.reshape(N, dm) @ Wo
    return kvs


def test_chained_layers_cache_invariant_and_negative_control():
    """Eq. 3 / App. A: with a cacheable mask R's K/V are bitwise independent
    of the target at every layer; when R reads live text (the mask of
    Sec. 3.2), target information reaches R's K/V from layer 3 on
    (X^(0) -> LT^(1) -> R^(2), and layer-3 K/V project R^(2))."""
    kinds, lens = [ST, LT, X, R, R], [2, 3, 4, 3, 3]
    rsl = np.r_[9:15]
    for p in ("paper", "perref", "isolated"):
        vis = om.PRESETS[p](kinds)
        a, b = _chained(kinds, lens, vis, 1), _chained(kinds, lens, vis, 2)
        for (ka, va), (kb, vb) in zip(a, b):
            assert np.array_equal(ka[:, rsl], kb[:, rsl]) and np.array_equal(va[:, rsl], vb[:, rsl])
    vis = om.live_text_mask(kinds)
    a, b = _chained(kinds, lens, vis, 1), _chained(kinds, lens, vis, 2)
    assert np.array_equal(a[0][0][:, rsl], b[0][0][:, rsl])
    assert np.array_equal(a[1][0][:, rsl], b[1][0][:, rsl])
    assert not np.allclose(a[2][0][:, rsl], b[2][0][:, rsl])


def test_row_subsets_match_full_rows():
    kinds, lens = [ST, LT, X, R, R], [3, 5, 8, 6, 4]
    vis = om.perref_mask(kinds)
    N = sum(lens)
    q, k, v = rand((1, N, 2, 8), 60), rand((1, N, 2, 8), 61), rand((1, N, 2, 8), 62)
    O, lse, _ = oa.full_attention(kinds, lens, vis, q, k, v, 0.5)
    rows = [0, 2, 7, 15, 16, 25]
    Os, lss, r = oa.full_attention(kinds, lens, vis, q, k, v, 0.5, rows=rows)
    assert list(r) == rows
    np.testing.assert_allclose(Os, O[:, rows], rtol=0, atol=1e-15)
    np.testing.assert_allclose(lss, lse[:, :, rows], rtol=0, atol=1e-15)
