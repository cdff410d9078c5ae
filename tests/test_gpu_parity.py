"""GPU parity: the HIP path through the C ABI against the fp64 oracle on the
same seeded bf16 inputs.  Tolerance (bf16 in, fp32 accumulate): max-abs
<= 2e-2 and relative L2 <= 5e-3 on O; LSE within 1e-3; the cache bit-exact.

Small cases are compared element by element; the full-size workloads on
sampled rows (the oracle evaluates rows independently)."""
import numpy as np
import pytest
import torch

import paper_2608_21229_amd as rc
from oracle import attention as oa
from oracle import masks as om
from synthgen import workload, SCALING_KS
from tests.parity_util import (Inputs, check, check_lse, draw_inputs, f64, full_sequence, sample_rows)

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def oracle_mask(inp, preset):
    return om.PRESETS[preset](inp.kinds)


def run_prefill(L, inp, scale, want_lse=True):
    q, k, v = (t.to(DEV) for t in inp.static)
    o, lse, kc, vc = rc.ref_kv_prefill(L, q, k, v, scale=scale, want_lse=want_lse)
    return o, lse, kc, vc


def run_step(L, inp, kc, vc, scale, splits=0, want_lse=True):
    q, k, v = (t.to(DEV) for t in inp.live)
    return rc.step_masked_attention(L, q, k, v, kc, vc, scale=scale, splits=splits, want_lse=want_lse)


def oracle_prefill(inp, vis, scale, rows=None):
    qs, ks, vs = (f64(t) for t in inp.static)
    return oa.reference_prefill(inp.kinds, inp.lens, vis, qs, ks, vs, scale, rows=rows)


def oracle_step(inp, vis, kc, vc, scale, rows=None):
    ql, kl, vl = (f64(t) for t in inp.live)
    return oa.denoise_step(inp.kinds, inp.lens, vis, ql, kl, vl, kc, vc, scale, rows=rows)


def layout_for(inp, preset):
    return rc.Layout(list(zip(inp.kinds, inp.lens)), preset)


def check_request(wl, preset, every=None, splits=0, layer=0, steps=(0,)):
    """Prefill + steps for one layer; compare prefill O/LSE, cache bits, step O/LSE."""
    print(f"[case] {wl.name}/{preset} B={wl.B} H={wl.H} D={wl.D} layer={layer} splits={splits} steps={steps}",
          flush=True)
    inp0 = draw_inputs(wl, layer=layer, step=steps[0])
    L = layout_for(inp0, preset)
    vis = oracle_mask(inp0, preset)
    scale = wl.scale
    o, lse, kc, vc = run_prefill(L, inp0, scale)
    torch.cuda.synchronize()
    ns = o.shape[1]
    rows = None if every is None else sample_rows(ns, every, seed=layer)
    Os, lses, _, kc_ref, vc_ref = oracle_prefill(inp0, vis, scale, rows)
    tag = f"{wl.name}/{preset}/layer{layer}"
    check(o, Os, f"{tag} prefill O", rows)
    check_lse(lse, lses, f"{tag} prefill", rows)
    assert np.array_equal(f64(kc), kc_ref) and np.array_equal(f64(vc), vc_ref), "cache is not a bit copy"
    for s in steps:
        inp = draw_inputs(wl, layer=layer, step=s)
        ol, lsel = run_step(L, inp, kc, vc, scale, splits=splits)
        torch.cuda.synchronize()
        nl = ol.shape[1]
        rws = None if every is None else sample_rows(nl, every, seed=s + 1)
        Ol, lsl, _ = oracle_step(inp, vis, kc_ref, vc_ref, scale, rws)
        check(ol, Ol, f"{tag} step{s} splits={splits} O", rws)
        check_lse(lsel, lsl, f"{tag} step{s}", rws)


@pytest.mark.parametrize("preset", ["perref", "paper", "isolated"])
def test_tiny_prefill_step_full(preset):
    wl = workload("tiny")
    check_request(wl, preset)
    inp = draw_inputs(wl)
    q, k, v = (full_sequence(inp, i).to(DEV) for i in range(3))
    for mask in (preset, "dense"):
        L = layout_for(inp, mask)
        o, lse = rc.full_attention(L, q, k, v, scale=wl.scale, want_lse=True)
        torch.cuda.synchronize()
        O, ls, _ = oa.full_attention(inp.kinds, inp.lens, om.PRESETS[mask](inp.kinds),
                                     *(f64(t) for t in (q, k, v)), wl.scale)
        check(o, O, f"tiny full {mask}")
        check_lse(lse, ls, f"tiny full {mask}")


RAGGED = [
    ("r1", [(0, 5), (1, 33), (2, 129), (3, 1), (3, 65), (3, 127)]),
    ("r2", [(1, 7), (2, 64), (0, 3), (3, 200), (3, 63)]),
    ("r3", [(3, 130), (0, 1), (2, 1), (1, 2), (3, 64)]),
]


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("preset", ["perref", "paper", "isolated"])
@pytest.mark.parametrize("name,segs", RAGGED)
def test_ragged_segments(name, segs, preset, D):
    from synthgen import Workload
    wl = Workload(f"{name}_D{D}", 2, 3, D, tuple(segs), std=1.0, seed=11)
    for splits in (1, 3, 0, rc.SPLITS_TAIL, rc.SPLITS_BALANCED):
        check_request(wl, preset, splits=splits)


# The prefill's bf16 cache store in each of its three forms: copy work-groups
# at the end of the attention grid take every cached row ("tail"), the rows
# that fit while the store kernel copies the rest ("split"), or none
# ("store": the attention grid fills whole rounds).  Ragged segments, several
# batch entries, one launch per batch entry (B = 2, H = 64), the paper mask,
# the largest segment table.
RAGGED5 = [(0, 50), (1, 64), (2, 256), (3, 300), (3, 77)]
# 32 segments, 30 of them cached (29 references of 39-300 tokens and the anchors)
MANY = [(0, 40), (1, 32), (2, 128)] + [(3, n) for n in (
    154, 99, 222, 275, 66, 39, 273, 165, 152, 131, 273, 276, 236, 110, 151, 110, 300, 232, 40, 65, 114, 54,
    187, 48, 170, 275, 231, 251, 235)]
CACHE_STORE = [
    ("tail_only", RAGGED5, "perref", 1, 8, 128, "tail"),
    ("split_ragged", RAGGED5, "perref", 3, 29, 128, "split"),
    ("split_per_batch", RAGGED5, "perref", 2, 64, 64, "split"),
    ("split_paper", RAGGED5, "paper", 1, 72, 64, "split"),
    # 256 equal work-groups (under the paper mask every static tile reads all static keys)
    ("store_only", [(0, 64), (1, 64), (2, 256), (3, 256), (3, 256), (3, 256)], "paper", 2, 32, 64, "store"),
    # the same layout under the per-reference mask: the one-key-tile anchor work-groups free their CUs
    ("split_anchor_cus", [(0, 64), (1, 64), (2, 256), (3, 256), (3, 256), (3, 256)], "perref", 2, 32, 64,
     "split"),
    ("split_32_segments", MANY, "perref", 1, 13, 128, "split"),
]


@pytest.mark.parametrize("name,segs,preset,B,H,D,regime", CACHE_STORE)
def test_prefill_cache_store_forms(name, segs, preset, B, H, D, regime):
    from synthgen import Workload
    wl = Workload(f"store_{name}", B, H, D, tuple(segs), std=1.0, seed=5)
    L = rc.Layout(list(segs), preset)
    _, copy_wgs, copy_rows = L.prefill_plan(B, H, D)
    total = B * H * L.rows(rc.ROWS_CACHED)
    got = "store" if copy_wgs == 0 else ("tail" if copy_rows == total else "split")
    assert got == regime, (copy_wgs, copy_rows, total)
    check_request(wl, preset)
    # every cache row is written: a poisoned cache comes back equal to the oracle's
    inp = draw_inputs(wl)
    q, k, v = (t.to(DEV) for t in inp.static)
    nc = L.rows(rc.ROWS_CACHED)
    kc = torch.full((B, H, nc, D), float("nan"), dtype=torch.bfloat16, device=DEV)
    vc = torch.full_like(kc, float("-inf"))
    rc.ref_kv_prefill(L, q, k, v, k_cache=kc, v_cache=vc, scale=wl.scale)
    torch.cuda.synchronize()
    _, _, _, kc_ref, vc_ref = oracle_prefill(inp, oracle_mask(inp, preset), wl.scale, rows=np.array([0]))
    assert np.array_equal(f64(kc), kc_ref) and np.array_equal(f64(vc), vc_ref), "cache is not a bit copy"


def last_round_rows(lens, B, H, bm=512, cus=256):
    """[B, N, H] bool: the (batch, row, head) cells of the query tiles the
    full recompute's last-round split runs as two pieces -- the last
    (B H tiles) mod 256 tiles in (batch, head, tile) order, tiles of bm rows
    inside each segment."""
    tiles, r0 = [], 0
    for n in lens:
        tiles += [(r0 + s, min(bm, n - s)) for s in range(0, n, bm)]
        r0 += n
    nt, A = len(tiles), B * H * len(tiles)
    m = torch.zeros((B, r0, H), dtype=torch.bool, device=DEV)
    for w in range(A - A % cus, A):
        b, h, t = w // (H * nt), (w // nt) % H, w % nt
        m[b, tiles[t][0]:tiles[t][0] + tiles[t][1], h] = True
    return m


# The full recompute's last-round split (rc_full_attention_ws): grids of whole
# query tiles whose partial last round leaves CUs idle; ragged last tiles,
# several query segments with different key counts, B = 2 and 3.
LAST_ROUND = [
    ("dense_D64", [(1, 100), (2, 1000), (3, 1500)], "dense", 1, 48, 64),
    ("paper_B2", [(1, 100), (2, 1000), (3, 1500), (3, 777)], "paper", 2, 24, 128),
    ("dense_B3", [(1, 100), (2, 1000), (3, 1500), (3, 777)], "dense", 3, 16, 64),
]


@pytest.mark.parametrize("name,segs,preset,B,H,D", LAST_ROUND)
def test_full_recompute_last_round_split(name, segs, preset, B, H, D):
    from synthgen import Workload
    wl = Workload(f"lastround_{name}", B, H, D, tuple(segs), std=1.0, seed=9)
    print(f"[case] last-round split {name}: B={B} H={H} D={D} segments={segs} mask={preset}", flush=True)
    L = rc.Layout(list(segs), preset)
    assert L.full_workspace_bytes(B, H, D) > 0
    inp = draw_inputs(wl)
    q, k, v = (full_sequence(inp, i).to(DEV) for i in range(3))
    o, lse = rc.full_attention(L, q, k, v, scale=wl.scale, want_lse=True)
    o2, lse2 = rc.full_attention(L, q, k, v, scale=wl.scale, want_lse=True)
    ou, lseu = rc.full_attention(L, q, k, v, scale=wl.scale, want_lse=True, last_round_split=False)
    torch.cuda.synchronize()
    assert torch.equal(o, o2) and torch.equal(lse, lse2), "split recompute is not deterministic"
    N = q.shape[1]
    rows = sample_rows(N, 5, seed=1)
    O, ls, _ = oa.full_attention(inp.kinds, inp.lens, om.PRESETS[preset](inp.kinds), *(f64(t) for t in (q, k, v)),
                                 wl.scale, rows=rows)
    check(o, O, f"{name} split O", rows)
    check_lse(lse, ls, f"{name} split", rows)
    split = last_round_rows(list(inp.lens), B, H)
    assert split.any() and not split.all()
    assert torch.equal(o[~split], ou[~split]), "tiles outside the last round differ from the unsplit call"
    assert torch.equal(lse.permute(0, 2, 1)[~split], lseu.permute(0, 2, 1)[~split])
    # the split tiles: every row of them against the oracle
    srows = np.nonzero(split.any(dim=2).any(dim=0).cpu().numpy())[0]
    O2, ls2, _ = oa.full_attention(inp.kinds, inp.lens, om.PRESETS[preset](inp.kinds),
                                   *(f64(t) for t in (q, k, v)), wl.scale, rows=srows)
    check(o, O2, f"{name} split rows O", srows)
    check_lse(lse, ls2, f"{name} split rows", srows)


# The step's last-round split (the automatic choice when the query tiles
# outnumber the CUs): the 5-reference shape at 32 and 40 heads on sampled rows
# (prefill and steps 0 and 39), a ragged layout element by element, B = 3.
@pytest.mark.parametrize("H", [32, 40])
def test_step_last_round_split_ref5_heads(H):
    from synthgen import Workload
    base = workload("ref5")
    wl = Workload(f"ref5_h{H}", 1, H, base.D, base.segments, std=base.std, seed=13)
    L = rc.Layout(list(wl.segments), "perref")
    assert L.auto_splits(1, H, wl.D) == rc.SPLITS_LAST_ROUND
    check_request(wl, "perref", every=67, splits=0, steps=(0, 39))
    # the tiles outside the last round are computed whole: bit-equal to the unsplit step
    inp = draw_inputs(wl)
    _, _, kc, vc = run_prefill(L, inp, wl.scale, want_lse=False)
    o_lr, _ = run_step(L, inp, kc, vc, wl.scale, splits=rc.SPLITS_LAST_ROUND, want_lse=False)
    o_1, _ = run_step(L, inp, kc, vc, wl.scale, splits=1, want_lse=False)
    torch.cuda.synchronize()
    live_lens = [n for kd, n in wl.segments if kd in (1, 2)]
    keep = ~last_round_rows(live_lens, 1, H)
    assert torch.equal(o_lr[keep], o_1[keep])


@pytest.mark.parametrize("B,H,D", [(1, 96, 64), (3, 32, 128)])
def test_step_last_round_split_ragged(B, H, D):
    from synthgen import Workload
    segs = ((0, 40), (1, 100), (2, 900), (3, 700), (3, 333))
    wl = Workload(f"lastround_step_B{B}_H{H}_D{D}", B, H, D, segs, std=1.0, seed=21)
    L = rc.Layout(list(segs), "perref")
    assert L.auto_splits(B, H, D) == rc.SPLITS_LAST_ROUND
    check_request(wl, "perref", every=3, splits=rc.SPLITS_LAST_ROUND)


def test_ref1_request_40_steps():
    """Single-reference 1024^2 shape: 1 prefill + 40 steps with fresh live
    Q/K/V each step, all run over the one cache.  Steps 0, 19 and 39 are
    compared on every 11th live row, every other step on every 37th."""
    wl = workload("ref1")
    inp0 = draw_inputs(wl)
    L = layout_for(inp0, "perref")
    vis = oracle_mask(inp0, "perref")
    o, lse, kc, vc = run_prefill(L, inp0, wl.scale)
    torch.cuda.synchronize()
    rows = sample_rows(o.shape[1], 13)
    Os, lses, _, kc_ref, vc_ref = oracle_prefill(inp0, vis, wl.scale, rows)
    check(o, Os, "ref1 prefill", rows)
    assert np.array_equal(f64(kc), kc_ref) and np.array_equal(f64(vc), vc_ref)
    full_rows = (0, wl.steps // 2 - 1, wl.steps - 1)
    for s in range(wl.steps):
        inp = draw_inputs(wl, step=s)
        ol, lsel = run_step(L, inp, kc, vc, wl.scale)
        torch.cuda.synchronize()
        if s in full_rows:
            rws = sample_rows(ol.shape[1], 11, seed=s)
        elif s % 2 == 0:
            rws = sample_rows(ol.shape[1], 37, seed=s)
        else:
            continue
        Ol, lsl, _ = oracle_step(inp, vis, kc_ref, vc_ref, wl.scale, rws)
        check(ol, Ol, f"ref1 step{s}", rws)
        check_lse(lsel, lsl, f"ref1 step{s}", rws)


@pytest.mark.parametrize("preset", ["perref", "paper"])
def test_ref5_headline(preset):
    """The 5-reference workload: first, middle and last of the 40 steps."""
    check_request(workload("ref5"), preset, every=37, steps=(0, 19, 39))


def test_ref1_paper_mask():
    """The figure's mask (references see only their own block and the
    anchors) at the single-reference shape, steps 0, 19 and 39."""
    check_request(workload("ref1"), "paper", every=13, steps=(0, 19, 39))


def test_ref5_isolated_cache():
    """The prior-work isolated cache (anchors detached) at the headline shape,
    the denominator of the anchor-overhead measurement."""
    check_request(workload("ref5"), "isolated", every=97)


def test_ref5_cfg_two_branch_batch():
    """Classifier-free guidance: both branches in one batch (B = 2), each with
    its own anchors, references and cache, at the headline shape."""
    from synthgen import Workload
    wl = workload("ref5")
    wl = Workload("ref5_cfg", 2, wl.H, wl.D, wl.segments, std=wl.std, seed=7)
    check_request(wl, "perref", every=113)


def test_batch_entries_equal_single_calls():
    """Two guidance branches at the headline shape: each batch entry of the
    B = 2 prefill, step (its grids fill the chip per entry, so the entries run
    as consecutive launches) and full recompute, with LSE, equals the B = 1
    call on that entry's slice bit for bit."""
    from synthgen import Workload
    wl = workload("ref5")
    wl = Workload("ref5_cfg", 2, wl.H, wl.D, wl.segments, std=wl.std, seed=7)
    inp = draw_inputs(wl)
    L = layout_for(inp, "perref")
    qs, ks, vs = (t.to(DEV) for t in inp.static)
    ql, kl, vl = (t.to(DEV) for t in inp.live)
    qa, ka, va = (full_sequence(inp, i).to(DEV) for i in range(3))
    o2, l2, kc2, vc2 = rc.ref_kv_prefill(L, qs, ks, vs, scale=wl.scale, want_lse=True)
    s2, sl2 = rc.step_masked_attention(L, ql, kl, vl, kc2, vc2, scale=wl.scale, splits=1, want_lse=True)
    f2, fl2 = rc.full_attention(L, qa, ka, va, scale=wl.scale, want_lse=True, last_round_split=False)
    for b in range(2):
        sl = slice(b, b + 1)
        o1, l1, kc1, vc1 = rc.ref_kv_prefill(L, qs[sl].contiguous(), ks[sl].contiguous(), vs[sl].contiguous(),
                                             scale=wl.scale, want_lse=True)
        s1, sl1 = rc.step_masked_attention(L, ql[sl].contiguous(), kl[sl].contiguous(), vl[sl].contiguous(),
                                           kc1, vc1, scale=wl.scale, splits=1, want_lse=True)
        f1, fl1 = rc.full_attention(L, qa[sl].contiguous(), ka[sl].contiguous(), va[sl].contiguous(),
                                    scale=wl.scale, want_lse=True, last_round_split=False)
        torch.cuda.synchronize()
        for name, x2, x1 in (("prefill O", o2, o1), ("prefill LSE", l2, l1), ("K cache", kc2, kc1),
                             ("V cache", vc2, vc1), ("step O", s2, s1), ("step LSE", sl2, sl1),
                             ("full O", f2, f1), ("full LSE", fl2, fl1)):
            assert torch.equal(x2[sl], x1), f"batch entry {b}: {name} differs from the single call"


def test_ref5_full_recompute_and_step_rows():
    """Full recompute (dense Base over [LT, X, R], and the same cacheable mask)
    on sampled rows; the step's rows equal the same-mask full recompute's
    LT/X rows bit for bit (same key tiles in the same order)."""
    wl = workload("ref5")
    inp = draw_inputs(wl)
    q, k, v = (full_sequence(inp, i).to(DEV) for i in range(3))
    L = layout_for(inp, "perref")
    of, _ = rc.full_attention(L, q, k, v, scale=wl.scale, last_round_split=False)
    o, _, kc, vc = run_prefill(L, inp, wl.scale, want_lse=False)
    ol, _ = run_step(L, inp, kc, vc, wl.scale, splits=1, want_lse=False)
    torch.cuda.synchronize()
    live_idx = np.concatenate([np.arange(64, 64 + 4608)])
    assert torch.equal(of[:, live_idx], ol), "step rows differ from same-mask full recompute"
    rows = sample_rows(q.shape[1], 97)
    O, _, _ = oa.full_attention(inp.kinds, inp.lens, om.perref_mask(inp.kinds), *(f64(t) for t in (q, k, v)),
                                wl.scale, rows=rows)
    check(of, O, "ref5 full perref", rows)
    # dense Base over [LT, X, R] (no anchors)
    kinds, lens = inp.kinds[1:], inp.lens[1:]
    LB = rc.Layout(list(zip(kinds, lens)), "dense")
    qb, kb, vb = q[:, 64:].contiguous(), k[:, 64:].contiguous(), v[:, 64:].contiguous()
    assert LB.full_workspace_bytes(1, wl.H, wl.D) > 0   # the Base runs with the last-round split
    ob, _ = rc.full_attention(LB, qb, kb, vb, scale=wl.scale)
    obu, _ = rc.full_attention(LB, qb, kb, vb, scale=wl.scale, last_round_split=False)
    torch.cuda.synchronize()
    rows = sample_rows(qb.shape[1], 101)
    O, _, _ = oa.full_attention(kinds, lens, om.dense_mask(kinds), *(f64(t) for t in (qb, kb, vb)), wl.scale,
                                rows=rows)
    check(ob, O, "ref5 full dense base", rows)
    check(obu, O, "ref5 full dense base, unsplit", rows)
    keep = ~last_round_rows(lens, 1, wl.H)
    assert torch.equal(ob[keep], obu[keep]), "tiles outside the last round differ from the unsplit call"


@pytest.mark.parametrize("preset", ["perref", "paper"])
@pytest.mark.parametrize("k", SCALING_KS)
def test_reference_scaling(k, preset):
    """k references of 4096 tokens under both masks (the figure's mask makes
    the prefill quadratic in k: the largest prefill the library runs)."""
    check_request(workload(f"scaling_k{k}"), preset, every=61)


def test_reference_scaling_paper_mask_k10_last_step():
    """Ten references under the figure's mask, steps 0 and 39."""
    check_request(workload("scaling_k10"), "paper", every=61, steps=(0, 39))


@pytest.mark.parametrize("layer", [0, 23, 47])
def test_mixed48_layers(layer):
    check_request(workload("mixed48"), "perref", every=53, layer=layer, steps=(0, 19, 39))


@pytest.mark.parametrize("layer", [0, 47])
def test_mixed48_layers_paper_mask(layer):
    check_request(workload("mixed48"), "paper", every=53, layer=layer, steps=(0, 19, 39))


@pytest.mark.parametrize("splits", [1, 2, 4, 7, 0, rc.SPLITS_TAIL, rc.SPLITS_BALANCED])
def test_split_kv_one_gpu_share(splits):
    """Headline shape at one GPU's share of heads (3 of 24): few query tiles,
    so split-KV carries the occupancy."""
    from synthgen import Workload
    wl = workload("ref5")
    wl = Workload("ref5_h3", 1, 3, 128, wl.segments, seed=5)
    check_request(wl, "perref", every=7, splits=splits)


def test_determinism_and_nan_poison():
    wl = workload("ref1")
    inp = draw_inputs(wl)
    L = layout_for(inp, "perref")
    q, k, v = (t.to(DEV) for t in inp.static)
    nc = L.rows(rc.ROWS_CACHED)
    B, N, H, D = q.shape
    # outputs poisoned with NaN and surrounded by guard elements (B = 1)
    guard = 16 * H * D
    nan = float("nan")
    obuf = torch.full((N * H * D + 2 * guard,), nan, dtype=torch.bfloat16, device=DEV)
    kcb = torch.full((B * H * nc * D + guard,), nan, dtype=torch.bfloat16, device=DEV)
    vcb = torch.full((B * H * nc * D + guard,), nan, dtype=torch.bfloat16, device=DEV)
    kc = kcb[:B * H * nc * D].view(B, H, nc, D)
    vc = vcb[:B * H * nc * D].view(B, H, nc, D)
    o = obuf[guard:guard + N * H * D].view(B, N, H, D)
    rc.ref_kv_prefill(L, q, k, v, o=o, k_cache=kc, v_cache=vc, scale=wl.scale)
    torch.cuda.synchronize()
    assert not torch.isnan(o).any() and not torch.isnan(kc).any() and not torch.isnan(vc).any()
    assert torch.isnan(obuf[:guard]).all() and torch.isnan(obuf[guard + N * H * D:]).all()
    assert torch.isnan(kcb[B * H * nc * D:]).all() and torch.isnan(vcb[B * H * nc * D:]).all()
    kc_c, vc_c = kc, vc
    ql, kl, vl = (t.to(DEV) for t in inp.live)
    runs = []
    for splits in (1, 1, 3, 3, -1, -1):
        ol = torch.full_like(ql, float("nan"))
        lse = torch.full((B, H, ql.shape[1]), float("nan"), device=DEV)
        rc.step_masked_attention(L, ql, kl, vl, kc_c, vc_c, o=ol, lse=lse, splits=splits, scale=wl.scale)
        runs.append((ol, lse))
    torch.cuda.synchronize()
    for ol, lse in runs:
        assert not torch.isnan(ol).any() and not torch.isnan(lse).any()
    assert torch.equal(runs[0][0], runs[1][0]) and torch.equal(runs[0][1], runs[1][1])
    assert torch.equal(runs[2][0], runs[3][0]) and torch.equal(runs[2][1], runs[3][1])
    assert torch.equal(runs[4][0], runs[5][0]) and torch.equal(runs[4][1], runs[5][1])


def test_fused_qkv_views_and_batch():
    """Q/K/V as views into one fused [B, N, 3, H, D] buffer (token stride 3*H*D), B = 2."""
    from synthgen import Workload, bf16_normal
    segs = ((0, 16), (1, 40), (2, 200), (3, 150), (3, 70))
    wl = Workload("fused", 2, 4, 128, segs, seed=3)
    inp = draw_inputs(wl)
    L = layout_for(inp, "paper")
    vis = oracle_mask(inp, "paper")
    fused = torch.stack(inp.static, dim=2).to(DEV)   # [B, N, 3, H, D]
    q, k, v = fused[:, :, 0], fused[:, :, 1], fused[:, :, 2]
    assert q.stride(1) == 3 * 4 * 128
    o, lse, kc, vc = rc.ref_kv_prefill(L, q, k, v, scale=wl.scale, want_lse=True)
    fl = torch.stack(inp.live, dim=2).to(DEV)
    ol, lsel = rc.step_masked_attention(L, fl[:, :, 0], fl[:, :, 1], fl[:, :, 2], kc, vc, scale=wl.scale,
                                        want_lse=True)
    torch.cuda.synchronize()
    Os, lses, _, kcr, vcr = oracle_prefill(inp, vis, wl.scale)
    check(o, Os, "fused prefill")
    check_lse(lse, lses, "fused prefill")
    Ol, lsl, _ = oracle_step(inp, vis, kcr, vcr, wl.scale)
    check(ol, Ol, "fused step")
    check_lse(lsel, lsl, "fused step")


@pytest.mark.parametrize("preset", ["perref", "paper", "isolated"])
def test_tiny_balanced_schedule(preset):
    """Balanced schedule on the tiny workload: 16 key-tile units over 256
    work-groups, so every query tile is cut into one-tile pieces and merged."""
    check_request(workload("tiny"), preset, splits=rc.SPLITS_BALANCED, steps=(0, 1))


def test_ref5_balanced_schedule():
    """Headline shape under the balanced schedule (432 query tiles of 393 key
    tiles dealt over 256 work-groups), sampled rows, two steps."""
    check_request(workload("ref5"), "perref", every=89, splits=rc.SPLITS_BALANCED, steps=(0, 1))


def test_ref5_cfg_batch_balanced():
    from synthgen import Workload
    wl = workload("ref5")
    wl = Workload("ref5_cfg_bal", 2, wl.H, wl.D, wl.segments, seed=9)
    check_request(wl, "perref", every=131, splits=rc.SPLITS_BALANCED)


@pytest.mark.parametrize("splits", [1, 3, -1])
def test_step_query_segment_without_keys(splits):
    """A live segment that reads no key: O = 0 and LSE = -inf on its rows
    (written by the merge under the balanced schedule), next to segments that
    read many."""
    from synthgen import Workload
    segs = ((0, 40), (1, 300), (2, 520), (3, 200), (3, 77))
    wl = Workload("nokeys", 2, 2, 128, segs, seed=13)
    n = len(segs)
    vis = om.perref_mask(wl.kinds)
    vis = [list(r) for r in vis]
    vis[1] = [False] * n          # LT reads nothing
    inp = draw_inputs(wl)
    L = rc.Layout(list(segs), vis)
    scale = wl.scale
    o, lse, kc, vc = run_prefill(L, inp, scale)
    ol, lsel = run_step(L, inp, kc, vc, scale, splits=splits)
    torch.cuda.synchronize()
    _, _, _, Kc, Vc = oracle_prefill(inp, vis, scale)
    Ol, Ll, _ = oracle_step(inp, vis, Kc, Vc, scale)
    check(ol, Ol, f"no-key segment step splits={splits} O")
    check_lse(lsel, Ll, f"no-key segment step splits={splits}")
    assert bool((ol[:, :300] == 0).all()) and bool(torch.isinf(lsel[:, :, :300]).all())
