"""Pins for the chained-layer oracle (oracle/chain.py).  The expected values
come from torch's float32 -> bfloat16 conversion (a library routine), from
worked rounding cases, from a 50-digit mpmath brute force of the whole chain,
from a closed form (uniform attention with permutation weights), from the
identity W_o = 0, and from the exactness of the cached path (Sec. 3.1,
Eq. 2; App. A)."""
import itertools

import mpmath
import numpy as np
import pytest
import torch

from oracle import chain as oc
from oracle import masks as om
from tests.test_oracle import token_mask

ST, LT, X, R = om.ST, om.LT, om.X, om.R


def bf16_arr(shape, seed, std=1.0):
    """Seeded values that are exact bf16 numbers, as float64."""
    g = torch.Generator().manual_seed(seed)
    return torch.randn(shape, generator=g).mul(std).to(torch.bfloat16).double().numpy()


# ----------------------------------------------------------------- round_bf16
def test_round_bf16_matches_torch_on_float32_values():
    g = torch.Generator().manual_seed(3)
    x = torch.randn(200_000, generator=g) * torch.exp(torch.randn(200_000, generator=g) * 8)
    # exact ties: low 16 bits 0x8000 on both even and odd kept bits
    bits = torch.randint(0, 2 ** 31, (4096,), generator=g, dtype=torch.int64)
    ties = ((bits & ~0xFFFF) | 0x8000).to(torch.int32).view(torch.float32)
    ties = ties[torch.isfinite(ties) & (ties.abs() >= 2.0 ** -126)]
    for xs in (x, ties, -ties):
        want = xs.to(torch.bfloat16).double().numpy()
        got = oc.round_bf16(xs.double().numpy())
        assert np.array_equal(got, want)


@pytest.mark.parametrize("x,want", [
    (1 + 2 ** -8, 1.0),                      # tie, kept bits even -> down
    (1 + 3 * 2 ** -8, 1 + 2 ** -6),          # tie, kept bits odd -> up
    (1 + 2 ** -8 + 2 ** -30, 1 + 2 ** -7),   # just above a tie: float32 would make it a tie first
    (-(1 + 2 ** -8 + 2 ** -30), -(1 + 2 ** -7)),
    (255.5, 256.0),                          # carry into the next binade
    (0.0, 0.0),
    (3.0, 3.0),
])
def test_round_bf16_worked_cases(x, want):
    assert oc.round_bf16(np.float64(x)) == want


# ------------------------------------------------------ mpmath brute force
def _bf(y):
    with mpmath.workprec(8):   # nearest, ties to even
        return +y


def brute_chain(kinds, lens, vis, h0, w_qkv, w_o, H, D, scale):
    """One token and one head at a time, 50 digits, bf16 rounding where the
    layer stores a tensor.  h0 [1, N, C]."""
    mpmath.mp.dps = 50
    tm = token_mask(kinds, lens, vis)
    N, C = h0.shape[1], H * D
    mp = mpmath.mpf
    h = [[mp(h0[0, i, c]) for c in range(C)] for i in range(N)]
    out = []
    for wq, wo in zip(w_qkv, w_o):
        qkv = [[_bf(mpmath.fsum(h[i][c] * mp(wq[n, c]) for c in range(C))) for n in range(3 * C)] for i in range(N)]
        o = [[mp(0)] * C for _ in range(N)]
        for i, hd in itertools.product(range(N), range(H)):
            js = [j for j in range(N) if tm[i, j]]
            if not js:
                continue
            s = [mp(scale) * mpmath.fsum(qkv[i][hd * D + d] * qkv[j][C + hd * D + d] for d in range(D)) for j in js]
            e = [mpmath.exp(x) for x in s]
            z = mpmath.fsum(e)
            for d in range(D):
                o[i][hd * D + d] = _bf(mpmath.fsum(e[t] * qkv[js[t]][2 * C + hd * D + d] for t in range(len(js))) / z)
        h = [[_bf(h[i][n] + mpmath.fsum(o[i][c] * mp(wo[n, c]) for c in range(C))) for n in range(C)] for i in range(N)]
        out.append(np.array([[float(x) for x in row] for row in h])[None])
    return out


TINY = ([ST, LT, X, R, R], [1, 2, 2, 2, 1])


@pytest.mark.parametrize("preset", ["perref", "paper", "dense"])
def test_chain_full_matches_brute_force(preset):
    kinds, lens = TINY
    vis = om.PRESETS[preset](kinds)
    H, D, L = 2, 2, 2
    C, N = H * D, sum(lens)
    h0 = bf16_arr((1, N, C), 11)
    w_qkv = [bf16_arr((3 * C, C), 20 + l, C ** -0.5) for l in range(L)]
    w_o = [bf16_arr((C, C), 30 + l, C ** -0.5) for l in range(L)]
    scale = D ** -0.5
    hs, kvs = oc.chain_full(kinds, lens, vis, h0, w_qkv, w_o, H, D, scale)
    want = brute_chain(kinds, lens, vis, h0, w_qkv, w_o, H, D, scale)
    for l in range(L):
        assert np.array_equal(hs[l], want[l]), (preset, l, np.abs(hs[l] - want[l]).max())


def test_chain_split_orders_q_k_v_heads():
    """Fused projection rows: Q heads, then K heads, then V heads, D each."""
    B, N, H, D = 1, 3, 2, 4
    qkv = np.arange(B * N * 3 * H * D, dtype=np.float64).reshape(B, N, 3 * H * D)
    q, k, v = oc.split_qkv(qkv, H, D)
    C = H * D
    for t, name in enumerate((q, k, v)):
        for n, h, d in itertools.product(range(N), range(H), range(D)):
            assert name[0, n, h, d] == qkv[0, n, t * C + h * D + d]


# --------------------------------------------------------------- closed forms
def test_chain_identity_when_output_projection_is_zero():
    kinds, lens = [ST, LT, X, R, R], [3, 4, 6, 5, 4]
    vis = om.perref_mask(kinds)
    H, D, L = 2, 4, 3
    C, N = H * D, sum(lens)
    h0 = bf16_arr((2, N, C), 5)
    w_qkv = [bf16_arr((3 * C, C), 40 + l, 0.3) for l in range(L)]
    w_o = [np.zeros((C, C)) for _ in range(L)]
    hs, _ = oc.chain_full(kinds, lens, vis, h0, w_qkv, w_o, H, D, D ** -0.5)
    for h in hs:
        assert np.array_equal(h, h0)


def test_chain_uniform_attention_with_permutation_weights():
    """W_Q = W_K = 0 gives uniform weights over the visible tokens; with
    W_V = P (a permutation) and W_O = I one layer gives
    h1[i] = bf16(h0[i] + bf16(mean_{j visible from i} P h0[j]))."""
    kinds, lens = [ST, LT, X, R, R], [2, 3, 4, 3, 2]
    vis = om.perref_mask(kinds)
    H, D = 2, 3
    C, N = H * D, sum(lens)
    h0 = bf16_arr((1, N, C), 9)
    perm = np.array([3, 0, 5, 1, 4, 2])
    P = np.zeros((C, C))
    P[np.arange(C), perm] = 1.0          # (P h)[n] = h[perm[n]]
    w_qkv = [np.concatenate([np.zeros((C, C)), np.zeros((C, C)), P])]
    w_o = [np.eye(C)]
    hs, _ = oc.chain_full(kinds, lens, vis, h0, w_qkv, w_o, H, D, D ** -0.5)
    tm = token_mask(kinds, lens, vis)
    want = np.zeros((1, N, C))
    for i in range(N):
        js = [j for j in range(N) if tm[i, j]]
        mean = sum(h0[0, j, perm] for j in js) / len(js)
        want[0, i] = oc.round_bf16(h0[0, i] + oc.round_bf16(mean))
    assert np.allclose(hs[0], want, rtol=0, atol=0)


# ------------------------------------------------ cached path = full recompute
@pytest.mark.parametrize("preset", ["perref", "paper", "isolated"])
def test_cached_chain_equals_full_recompute(preset):
    kinds, lens = [ST, LT, X, R, R, R], [5, 7, 12, 9, 6, 4]
    vis = om.PRESETS[preset](kinds)
    B, H, D, L = 2, 2, 4, 3
    C, N = H * D, sum(lens)
    w_qkv = [bf16_arr((3 * C, C), 60 + l, C ** -0.5) for l in range(L)]
    w_o = [bf16_arr((C, C), 70 + l, C ** -0.5) for l in range(L)]
    scale = D ** -0.5
    static = [i for i, k in enumerate(kinds) if k in (ST, R)]
    live = [i for i, k in enumerate(kinds) if k in (LT, X)]
    off = np.cumsum([0] + lens)
    rows_of = lambda segs: np.concatenate([np.arange(off[s], off[s + 1]) for s in segs])
    h_static = bf16_arr((B, len(rows_of(static)), C), 80)
    _, caches = oc.chain_prefill(kinds, lens, vis, h_static, w_qkv, w_o, H, D, scale)
    for step in range(2):
        h_live = bf16_arr((B, len(rows_of(live)), C), 90 + step)
        h0 = np.zeros((B, N, C))
        h0[:, rows_of(static)] = h_static
        h0[:, rows_of(live)] = h_live
        hs_full, kvs = oc.chain_full(kinds, lens, vis, h0, w_qkv, w_o, H, D, scale)
        hs_step = oc.chain_step(kinds, lens, vis, h_live, caches, w_qkv, w_o, H, D, scale)
        for l in range(L):
            np.testing.assert_allclose(hs_step[l], hs_full[l][:, rows_of(live)], rtol=0, atol=1e-12)
            cs = om.cached_segments(kinds, vis)
            if cs:
                kc = kvs[l][0][:, rows_of(cs)].transpose(0, 2, 1, 3)
                vc = kvs[l][1][:, rows_of(cs)].transpose(0, 2, 1, 3)
                assert np.array_equal(caches[l][0], kc) and np.array_equal(caches[l][1], vc)


def test_isolated_chain_live_rows_ignore_anchor_inputs():
    """Under the isolated mask nobody reads ST, so changing the anchor rows'
    hidden state changes no live row at any layer."""
    kinds, lens = [ST, LT, X, R], [4, 3, 5, 6]
    vis = om.isolated_mask(kinds)
    H, D, L = 1, 4, 2
    C, N = H * D, sum(lens)
    w_qkv = [bf16_arr((3 * C, C), 100 + l, 0.5) for l in range(L)]
    w_o = [bf16_arr((C, C), 110 + l, 0.5) for l in range(L)]
    h0 = bf16_arr((1, N, C), 120)
    h1 = h0.copy()
    h1[:, :4] = bf16_arr((1, 4, C), 121)
    a, _ = oc.chain_full(kinds, lens, vis, h0, w_qkv, w_o, H, D, 0.5)
    b, _ = oc.chain_full(kinds, lens, vis, h1, w_qkv, w_o, H, D, 0.5)
    assert np.array_equal(a[-1][:, 4:], b[-1][:, 4:])
    assert not np.array_equal(a[-1][:, :4], b[-1][:, :4])
