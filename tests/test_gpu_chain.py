"""GPU checks of the dense projection (rc_linear) and of chained synthetic
layers (projection -> masked attention -> projection + residual) built on the
C ABI, against the fp64 chain oracle on the same seeded inputs.

Tolerance.  Both sides round every stored tensor (hidden state, fused QKV,
attention output) to bf16 at the same points.  A projection differs from the
oracle only by fp32 accumulation order: within one bf16 ulp of the result
plus fp32's error on the terms.  The attention differs further, because the
kernel rounds the softmax weights to bf16 for the P V product (its own
tolerance: max-abs 2e-2, relative L2 5e-3 on O).  Through the residual
stream each layer carries the error of the layers before it forward with
gain one and adds its own, so after layer l (from 0) the bar per element is
(l + 1) max(2e-2, 2^-6 |ref|) -- one layer's share being the attention's
absolute bound or two bf16 ulps, whichever is larger -- and the relative L2
error of every tensor stays within 5e-3.

Exactness (Sec. 3.1, Eq. 2): with segment lengths on the 64-key tile grid and
no split-KV, the cached path's live rows equal the full recompute's bit for
bit at every layer, and every layer's cache equals the K/V rows the full
recompute projects."""
import numpy as np
import pytest
import torch

import paper_2608_21229_amd as rc
from oracle import chain as oc
from oracle import fp8 as of
from oracle import masks as om
from synthgen import ANCHOR, REF, TEXT, TARGET, Workload, bf16_normal, draw_chain_weights, draw_hidden, workload
from tests.parity_util import f64

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
REL_L2 = 5e-3


def ulp_bf16(x):
    """Spacing of bf16 numbers at |x| (x != 0): 2^(floor(log2|x|) - 7)."""
    e = np.floor(np.log2(np.maximum(np.abs(x), 2.0 ** -126)))
    return np.ldexp(1.0, (e - 7).astype(np.int64))


def check_projection(gpu, ref, what, a, w, r=None):
    """One bf16 ulp of the result plus the fp32 accumulation error, bounded by
    2^-16 times the sum of the magnitudes of the terms (|a| |w|^T + |r|): where
    the terms cancel, the ulp of the result is smaller than fp32's error."""
    g = f64(gpu)
    d = np.abs(g - ref)
    mag = np.abs(a) @ np.abs(w).T + (0 if r is None else np.abs(r))
    bad = d > ulp_bf16(ref) + 2.0 ** -16 * mag
    n_diff = int((d > 0).sum())
    over = d > ulp_bf16(ref)
    print(f"[parity] {what}: differing={n_diff}/{ref.size} max_abs={d.max():.3e} beyond_one_ulp={int(over.sum())}",
          flush=True)
    for i in np.argwhere(over)[:4]:
        i = tuple(i)
        print(f"    at {i}: ref={ref[i]:.6e} got={g[i]:.6e} term_magnitude={mag[i]:.3e}", flush=True)
    assert not bad.any(), f"{what}: {int(bad.sum())} elements beyond the bound"
    assert n_diff <= max(8, ref.size // 200), f"{what}: {n_diff} elements differ"


def check_chain(gpu, ref, what, layer):
    g = f64(gpu)
    assert g.shape == ref.shape, (what, g.shape, ref.shape)
    assert np.all(np.isfinite(g)), what
    d = np.abs(g - ref)
    lim = (layer + 1) * np.maximum(2e-2, 2.0 ** -6 * np.abs(ref))
    rel = float(np.linalg.norm(g - ref) / np.linalg.norm(ref))
    print(f"[parity] {what}: max_abs={d.max():.3e} worst/bound={(d / lim).max():.3f} rel_l2={rel:.3e}", flush=True)
    assert (d <= lim).all(), f"{what}: {int((d > lim).sum())} elements beyond {layer + 1} max(2e-2, 2^-6 |ref|)"
    assert rel <= REL_L2, f"{what}: rel_l2 {rel:.3e}"


# ------------------------------------------------------------------ rc_linear
def _bf(shape, seed, std=1.0):
    return bf16_normal(shape, seed, std)


@pytest.mark.parametrize("M,N,K,resid,strided", [
    (300, 256, 192, True, True),      # ragged M, odd number of K steps, strided views
    (1, 128, 64, False, False),        # one row, one K step
    (127, 384, 128, True, False),
    (129, 128, 256, False, True),
    (1000, 512, 320, True, False),
    (257, 768, 64, True, True),        # 256-wide tiles: one row past a tile, one K step
    (2100, 1024, 448, False, False),   # 256-wide tiles: 9 m-tiles (a partial group of 4), odd K steps
])
def test_linear_matches_oracle(M, N, K, resid, strided):
    a_full = _bf((M, K + (64 if strided else 0)), 1 + M)
    a = a_full[:, :K]
    w = _bf((N, K), 2 + N, K ** -0.5)
    r = _bf((M, N), 3 + K) if resid else None
    want = oc.project(f64(a), f64(w), None if r is None else f64(r))
    a_d = a_full.to(DEV)[:, :K]
    if strided:
        out_full = torch.full((M, N + 128), 7.0, dtype=torch.bfloat16, device=DEV)
        out = out_full[:, :N]
    else:
        out = None
    got = rc.linear(a_d, w.to(DEV), residual=None if r is None else r.to(DEV), out=out)
    torch.cuda.synchronize()
    check_projection(got, want, f"linear M={M} N={N} K={K} resid={resid} strided={strided}",
                     f64(a), f64(w), None if r is None else f64(r))
    if strided:
        assert bool((out_full[:, N:] == 7.0).all()), "wrote outside the output view"


def test_linear_in_place_residual():
    M, N, K = 200, 256, 128
    a, w, r = _bf((M, K), 11), _bf((N, K), 12, K ** -0.5), _bf((M, N), 13)
    want = oc.project(f64(a), f64(w), f64(r))
    h = r.to(DEV)
    rc.linear(a.to(DEV), w.to(DEV), residual=h, out=h)
    torch.cuda.synchronize()
    check_projection(h, want, "linear in place", f64(a), f64(w), f64(r))


@pytest.mark.parametrize("N", [384, 512])   # 128-wide and 256-wide output tiles
def test_linear_rows_do_not_depend_on_batch(N):
    """A row's result is the same bits whatever rows surround it."""
    M, K = 1000, 256
    a = _bf((M, K), 21).to(DEV)
    w = _bf((N, K), 22, K ** -0.5).to(DEV)
    whole = rc.linear(a, w)
    for lo, hi in ((0, 1), (77, 300), (129, 1000), (999, 1000)):
        part = rc.linear(a[lo:hi], w)
        torch.cuda.synchronize()
        assert torch.equal(part, whole[lo:hi]), (lo, hi)


@pytest.mark.parametrize("N,resid", [(9216, False), (3072, True)])
def test_linear_headline_shapes_sampled_rows(N, resid):
    """The projections of the 5-reference workload's live rows (4608 x 3072
    hidden, 24 heads of 128): fused QKV and output projection + residual, on
    64 sampled rows (every output row is an independent dot-product set)."""
    M, K = 4608, 3072
    a = _bf((M, K), 31)
    w = _bf((N, K), 32, K ** -0.5)
    r = _bf((M, N), 33) if resid else None
    got = rc.linear(a.to(DEV), w.to(DEV), residual=None if r is None else r.to(DEV))
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(N).choice(M, 64, replace=False))
    want = oc.project(f64(a[rows]), f64(w), None if r is None else f64(r[rows]))
    check_projection(got[rows], want, f"linear headline N={N} resid={resid} (64 rows)",
                     f64(a[rows]), f64(w), None if r is None else f64(r[rows]))


# ------------------------------------------------------------- chained layers
def _wl(name, B, H, D, lens_st_lt_x, refs, seed=42):
    st, lt, x = lens_st_lt_x
    segs = ((ANCHOR, st), (TEXT, lt), (TARGET, x)) + tuple((REF, n) for n in refs)
    return Workload(name, B, H, D, segs, seed=seed)


def seq_index(wl, static: bool):
    """Sequence positions of the static (ST, R) or live (LT, X) rows."""
    idx, pos = [], 0
    for k, n in wl.segments:
        if (k in (ANCHOR, REF)) == static:
            idx.extend(range(pos, pos + n))
        pos += n
    return torch.tensor(idx, dtype=torch.long)


def assemble(wl, h_static, h_live):
    B, _, C = h_static.shape
    N = h_static.shape[1] + h_live.shape[1]
    h = torch.empty((B, N, C), dtype=h_static.dtype, device=h_static.device)
    h[:, seq_index(wl, True).to(h.device)] = h_static
    h[:, seq_index(wl, False).to(h.device)] = h_live
    return h


def make_chain(wl, layers, preset):
    w_qkv, w_o = draw_chain_weights(wl.H, wl.D, layers, wl.seed)
    layout = rc.Layout(list(wl.segments), preset)
    ch = rc.Chain(layout, [w.to(DEV) for w in w_qkv], [w.to(DEV) for w in w_o], wl.H, wl.D)
    return ch, [f64(w) for w in w_qkv], [f64(w) for w in w_o]


CHAIN_CASES = {
    # the tiny workload's ragged 8 / 16 / 64 / 64 segments, head_dim 64
    "tiny": (workload("tiny"), 3, "perref"),
    # ragged lengths off the tile grid, two batch rows, two references
    "ragged": (_wl("ragged", 2, 2, 128, (24, 40, 200), [136, 72]), 3, "paper"),
    "ragged_perref": (_wl("ragged_perref", 1, 4, 64, (8, 56, 130), [70, 64, 9]), 2, "perref"),
}


@pytest.mark.parametrize("case", sorted(CHAIN_CASES))
def test_chain_matches_oracle(case):
    wl, layers, preset = CHAIN_CASES[case]
    ch, Wq, Wo = make_chain(wl, layers, preset)
    vis = om.PRESETS[preset](wl.kinds)
    kinds, lens, H, D, scale = wl.kinds, wl.lens, wl.H, wl.D, wl.scale
    h_s, _ = draw_hidden(wl, 0)
    print(f"[case] chain {case}: B={wl.B} H={H} D={D} segments={wl.segments} layers={layers}", flush=True)
    hs_pre = []
    caches = ch.prefill(h_s.to(DEV), collect=hs_pre)
    torch.cuda.synchronize()
    want_pre, want_caches = oc.chain_prefill(kinds, lens, vis, f64(h_s), Wq, Wo, H, D, scale)
    for l in range(layers):
        check_chain(hs_pre[l], want_pre[l], f"{case} prefill layer {l} hidden", l)
        check_chain(caches[l][0], want_caches[l][0], f"{case} layer {l} K cache", l)
        check_chain(caches[l][1], want_caches[l][1], f"{case} layer {l} V cache", l)
    for step in (0, 1):
        _, h_l = draw_hidden(wl, step)
        hs = []
        ch.step(h_l.to(DEV), caches, collect=hs)
        hs_full = []
        ch.full(assemble(wl, h_s, h_l).to(DEV), collect=hs_full)
        torch.cuda.synchronize()
        want = oc.chain_step(kinds, lens, vis, f64(h_l), want_caches, Wq, Wo, H, D, scale)
        h0 = f64(assemble(wl, h_s, h_l))
        want_full, _ = oc.chain_full(kinds, lens, vis, h0, Wq, Wo, H, D, scale)
        for l in range(layers):
            check_chain(hs[l], want[l], f"{case} step {step} layer {l} live hidden", l)
            check_chain(hs_full[l], want_full[l], f"{case} full step {step} layer {l} hidden", l)


@pytest.mark.parametrize("case", ["tiny", "ragged"])
def test_chain_fp8_cache_matches_oracle(case):
    """The chain over the FP8 reference cache: each layer's live rows against
    the fp64 chain whose step reads the oracle's own quantised-then-dequantised
    caches (Sec. 3.1, Eq. 2: a layer's cached K/V are its static rows'
    projections).  The GPU quantises its bf16 K/V, which can differ from the
    oracle's by one bf16 ulp, so a code may sit one e4m3 step away: the bound
    is the chain's."""
    wl, layers, preset = CHAIN_CASES[case]
    w_qkv, w_o = draw_chain_weights(wl.H, wl.D, layers, wl.seed)
    layout = rc.Layout(list(wl.segments), preset)
    ch = rc.Chain(layout, [w.to(DEV) for w in w_qkv], [w.to(DEV) for w in w_o], wl.H, wl.D, cache="fp8")
    Wq, Wo = [f64(w) for w in w_qkv], [f64(w) for w in w_o]
    vis = om.PRESETS[preset](wl.kinds)
    kinds, lens, H, D, scale = wl.kinds, wl.lens, wl.H, wl.D, wl.scale
    print(f"[case] chain fp8 {case}: B={wl.B} H={H} D={D} segments={wl.segments} layers={layers}", flush=True)
    h_s, h_l = draw_hidden(wl, 0)
    caches = ch.prefill(h_s.to(DEV))
    hs = []
    ch.step(h_l.to(DEV), caches, collect=hs)
    torch.cuda.synchronize()
    _, want_caches = oc.chain_prefill(kinds, lens, vis, f64(h_s), Wq, Wo, H, D, scale)
    deq = []
    for kc, vc in want_caches:
        kq, ks = of.quantize_cache(kc)
        vq, vs = of.quantize_cache(vc)
        deq.append((of.dequantize(kq, ks), of.dequantize(vq, vs)))
    want = oc.chain_step(kinds, lens, vis, f64(h_l), deq, Wq, Wo, H, D, scale)
    for l in range(layers):
        check_chain(hs[l], want[l], f"{case} fp8 step layer {l} live hidden", l)


ALIGNED = {
    "aligned": (_wl("aligned", 2, 2, 128, (64, 128, 512), [512, 256]), 3),
    # the 5-reference workload at full size (24 heads of 128, 25152 tokens)
    "ref5": (workload("ref5"), 2),
}


@pytest.mark.parametrize("case", sorted(ALIGNED))
def test_chain_cached_path_equals_full_recompute_bitwise(case):
    wl, layers = ALIGNED[case]
    ch, _, _ = make_chain(wl, layers, "perref")
    H, D, C = wl.H, wl.D, wl.H * wl.D
    print(f"[case] chain exactness {case}: B={wl.B} H={H} D={D} segments={wl.segments} layers={layers}",
          flush=True)
    h_s, h_l = draw_hidden(wl, 3)
    h_s, h_l = h_s.to(DEV), h_l.to(DEV)
    caches = ch.prefill(h_s)
    hs_step, hs_full = [], []
    ch.step(h_l, caches, splits=1, collect=hs_step)
    h0 = assemble(wl, h_s, h_l)
    ch.full(h0, collect=hs_full, last_round_split=False)
    torch.cuda.synchronize()
    live = seq_index(wl, False).to(DEV)
    cached_segs = om.cached_segments(wl.kinds, om.perref_mask(wl.kinds))
    off = np.cumsum([0] + wl.lens)
    cached = torch.tensor(np.concatenate([np.arange(off[s], off[s + 1]) for s in cached_segs]), device=DEV)
    prev = h0
    for l in range(layers):
        assert torch.equal(hs_step[l], hs_full[l][:, live]), f"layer {l}: live rows differ"
        qkv = rc.linear(prev.reshape(-1, C), ch.w_qkv[l]).view(wl.B, -1, 3, H, D)
        k_full = qkv[:, cached, 1].permute(0, 2, 1, 3)
        v_full = qkv[:, cached, 2].permute(0, 2, 1, 3)
        torch.cuda.synchronize()
        assert torch.equal(caches[l][0], k_full) and torch.equal(caches[l][1], v_full), f"layer {l}: cache differs"
        prev = hs_full[l]
    # a different step's live input leaves every cache untouched
    before = [(k.clone(), v.clone()) for k, v in caches]
    _, h_l2 = draw_hidden(wl, 4)
    ch.step(h_l2.to(DEV), caches)
    torch.cuda.synchronize()
    assert all(torch.equal(a, c) and torch.equal(b, d) for (a, b), (c, d) in zip(before, caches))
