"""Host-only checks of the C ABI: the library loads, exports every function
include/refcache.h declares, computes presets / pair counts / row counts that
agree with the oracle's independent statement, and rejects bad arguments with
the documented status before any HIP call (so no GPU is needed)."""
import ctypes
import os
import random
import re
import subprocess

import pytest

import paper_2608_21229_amd as rc
from paper_2608_21229_amd import binding
from oracle import cost as oc
from oracle import masks as om

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "refcache.h")
FAKE = 0x7f0000000000   # 16-byte aligned, never dereferenced: every call below fails validation first


def header_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\**\s+\**(rc_\w+)\s*\(", text, re.M)))


def test_library_exports_every_declared_function():
    names = header_functions()
    assert len(names) >= 10
    out = subprocess.run(["nm", "-D", "--defined-only", binding.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\sT\s(rc_\w+)", out))
    missing = [n for n in names if n not in exported]
    assert not missing, missing
    assert set(names) == set(binding.SIGNATURES), "binding signatures out of sync with the header"
    L = rc.lib()
    for n in names:
        assert getattr(L, n) is not None


def random_layout(rng):
    n = rng.randint(1, 10)
    kinds = [rng.choice([0, 1, 2, 3]) for _ in range(n)]
    lens = [rng.choice([1, 2, 7, 64, 65, 100, 4096]) for _ in range(n)]
    return kinds, lens


@pytest.mark.parametrize("preset", ["paper", "perref", "isolated", "dense"])
def test_presets_and_counts_match_oracle(preset):
    rng = random.Random(7)
    for _ in range(200):
        kinds, lens = random_layout(rng)
        L = rc.Layout(list(zip(kinds, lens)), preset)
        vis = om.PRESETS[preset](kinds)
        assert L.visible == vis
        assert L.pairs(rc.ENTRY_FULL) == oc.visible_pairs(kinds, lens, vis, "all")
        cacheable = om.is_cacheable(kinds, vis)
        for entry, rows in ((rc.ENTRY_PREFILL, "static"), (rc.ENTRY_STEP, "live")):
            if cacheable:
                assert L.pairs(entry) == oc.visible_pairs(kinds, lens, vis, rows)
            else:
                assert L.validate(entry) == rc.RC_ERR_MASK_NOT_CACHEABLE
        assert L.rows(rc.ROWS_STATIC) == sum(n for k, n in zip(kinds, lens) if k in (0, 3))
        assert L.rows(rc.ROWS_LIVE) == sum(n for k, n in zip(kinds, lens) if k in (1, 2))
        assert L.rows(rc.ROWS_ALL) == sum(lens)
        assert L.rows(rc.ROWS_CACHED) == sum(lens[i] for i in om.cached_segments(kinds, vis))


def test_headline_counts():
    segs = [(0, 64), (1, 512), (2, 4096)] + [(3, 4096)] * 5
    L = rc.Layout(segs, "perref")
    assert L.pairs(rc.ENTRY_STEP) == 115_900_416
    assert L.pairs(rc.ENTRY_PREFILL) == 85_200_896
    assert L.rows(rc.ROWS_CACHED) == 20_544
    P = rc.Layout(segs, "paper")
    n_r, n_st, s = 20480, 64, 4608
    assert P.pairs(rc.ENTRY_PREFILL) == oc.c_pre(n_r, n_st)
    assert P.pairs(rc.ENTRY_STEP) == oc.c_step(n_r, s)
    D = rc.Layout(segs[1:], "dense")
    assert D.pairs(rc.ENTRY_FULL) * 40 == oc.c_full(n_r, s, 40)


def test_live_text_mask_rejected_for_cached_entries():
    kinds = [0, 1, 2, 3]
    L = rc.Layout(list(zip(kinds, [4, 4, 4, 4])), om.live_text_mask(kinds))
    assert L.validate(rc.ENTRY_PREFILL) == rc.RC_ERR_MASK_NOT_CACHEABLE
    assert L.validate(rc.ENTRY_STEP) == rc.RC_ERR_MASK_NOT_CACHEABLE
    assert L.validate(rc.ENTRY_FULL) == rc.RC_OK
    with pytest.raises(rc.RcError) as e:
        L.pairs(rc.ENTRY_STEP)
    assert e.value.status == rc.RC_ERR_MASK_NOT_CACHEABLE
    assert "not exactly cacheable" in rc.lib().rc_last_error().decode()


def _prefill(L, B=1, H=2, D=128, scale=0.1, q=FAKE, k=FAKE, v=FAKE, ts=None, o=FAKE, lse=None, kc=FAKE, vc=FAKE):
    ts = H * D if ts is None else ts
    return rc.lib().rc_ref_kv_prefill(ctypes.byref(L.c), B, H, D, scale, q, k, v, ts, o, lse, kc, vc, None)


def _step(L, B=1, H=2, D=128, scale=0.1, q=FAKE, k=FAKE, v=FAKE, ts=None, kc=FAKE, vc=FAKE, o=FAKE, lse=None,
          splits=1, ws=None, wsb=0):
    ts = H * D if ts is None else ts
    return rc.lib().rc_step_masked_attention(ctypes.byref(L.c), B, H, D, scale, q, k, v, ts, kc, vc, o, lse,
                                             splits, ws, wsb, None)


def _full(L, B=1, H=2, D=128, scale=0.1, q=FAKE, k=FAKE, v=FAKE, ts=None, o=FAKE, lse=None):
    ts = H * D if ts is None else ts
    return rc.lib().rc_full_attention(ctypes.byref(L.c), B, H, D, scale, q, k, v, ts, o, lse, None)


def _full_ws(L, B=1, H=2, D=128, scale=0.1, q=FAKE, k=FAKE, v=FAKE, ts=None, o=FAKE, lse=None, ws=None, wsb=0):
    ts = H * D if ts is None else ts
    return rc.lib().rc_full_attention_ws(ctypes.byref(L.c), B, H, D, scale, q, k, v, ts, o, lse, ws, wsb, None)


SEGS = [(0, 8), (1, 16), (2, 64), (3, 64)]


def test_argument_errors_launch_nothing():
    L = rc.Layout(SEGS, "perref")
    A, U, W = rc.RC_ERR_ARG, rc.RC_ERR_UNSUPPORTED, rc.RC_ERR_WORKSPACE
    for fn in (_prefill, _step, _full):
        assert fn(L, q=None) == A
        assert fn(L, q=FAKE + 8) == A                  # misaligned
        assert fn(L, o=None) == A
        assert fn(L, D=96) == U
        assert fn(L, D=256) == U
        assert fn(L, B=0) == A
        assert fn(L, H=0) == A
        assert fn(L, scale=0.0) == A
        assert fn(L, scale=float("nan")) == A
        assert fn(L, ts=2 * 128 - 8) == A              # token stride below H*D
        assert fn(L, ts=2 * 128 + 4) == A              # not a multiple of 8
        assert fn(L, ts=(1 << 24) + 8) == A            # a tile's byte record count would pass 2^31
        assert "tok_stride" in rc.lib().rc_last_error().decode()
        # the largest stride passes its check (64 tokens x 2^25 bytes = 2^31
        # fits the unsigned 32-bit record count); the call then fails on q
        assert fn(L, ts=1 << 24, q=None) == A
        assert "null" in rc.lib().rc_last_error().decode()
        assert fn(L, lse=FAKE + 2) == A                # misaligned LSE
        assert rc.lib().rc_last_error().decode() != ""
    assert _prefill(L, kc=None) == A
    assert _step(L, vc=None) == A
    assert _step(L, splits=-4) == A
    assert _step(L, splits=33) == A
    assert _step(L, splits=-2) == W                    # tail split, no workspace
    assert L.workspace_bytes(1, 2, 128, -2) == L.workspace_bytes(1, 2, 128, 2)
    assert _step(L, splits=-1) == W                    # balanced schedule, no workspace
    need_bal = L.workspace_bytes(1, 2, 128, -1)
    assert need_bal == 2 * 256 * 256 * 130 * 4         # fixed: two partial tiles per work-group
    assert L.workspace_bytes(1, 2, 64, -1) == 2 * 256 * 256 * 66 * 4
    assert _step(L, splits=-1, ws=FAKE, wsb=need_bal - 1) == W
    assert _step(L, splits=2) == W                     # no workspace
    need = L.workspace_bytes(1, 2, 128, 2)
    assert need == 2 * 1 * 2 * 80 * 130 * 4
    assert _step(L, splits=2, ws=FAKE, wsb=need - 1) == W
    assert _step(L, splits=2, ws=FAKE + 4, wsb=need) == W
    # grid overflow: 65535 x 65535 x tiles work-groups
    assert _full(L, B=65535, H=65535, ts=65535 * 128) == A
    # the cache store's grid (one thread per 16-byte granule) overflows before
    # the prefill attention's: 2^28 (b, h) pairs x 2 query tiles, 160 cached rows
    Lc = rc.Layout([(0, 32), (1, 8), (2, 8), (3, 128)], "perref")
    assert _prefill(Lc, B=16384, H=16384, ts=16384 * 128) == A
    assert "cache store" in rc.lib().rc_last_error().decode()
    # the split-KV combine's grid overflows before the step's: 2^26 (b, h)
    # pairs x 8 query tiles x 2 splits, 2048 live rows
    Ls = rc.Layout([(0, 64), (1, 256), (2, 1792), (3, 64)], "perref")
    need = Ls.workspace_bytes(8192, 8192, 128, 2)
    assert _step(Ls, B=8192, H=8192, ts=8192 * 128, splits=2, ws=FAKE, wsb=need) == A
    assert "combine" in rc.lib().rc_last_error().decode()
    need = Ls.workspace_bytes(8192, 8192, 128, -1)
    assert _step(Ls, B=8192, H=8192, ts=8192 * 128, splits=-1, ws=FAKE, wsb=need) == A
    assert "balanced merge" in rc.lib().rc_last_error().decode()


def test_layout_errors():
    c = binding.rc_layout()
    c.n_seg = 0
    lb = rc.lib()
    assert lb.rc_layout_preset(ctypes.byref(c), 0) == rc.RC_ERR_ARG
    assert lb.rc_pairs(ctypes.byref(c), 2) == rc.RC_ERR_ARG
    c.n_seg = 33
    assert lb.rc_layout_validate(ctypes.byref(c), 2) == rc.RC_ERR_ARG
    c.n_seg = 2
    c.seg[0].kind, c.seg[0].len = 0, 4
    c.seg[1].kind, c.seg[1].len = 3, 0
    assert lb.rc_layout_validate(ctypes.byref(c), 2) == rc.RC_ERR_ARG      # zero-length segment
    c.seg[1].len = 4
    c.seg[1].kind = 9
    assert lb.rc_layout_validate(ctypes.byref(c), 2) == rc.RC_ERR_ARG      # unknown kind
    c.seg[1].kind = 3
    assert lb.rc_layout_preset(ctypes.byref(c), 7) == rc.RC_ERR_ARG       # unknown preset
    assert lb.rc_layout_preset(ctypes.byref(c), 1) == rc.RC_OK
    c.visible[0] |= 1 << 5                                                 # bit beyond n_seg
    assert lb.rc_layout_validate(ctypes.byref(c), 2) == rc.RC_ERR_ARG
    assert lb.rc_layout_validate(ctypes.byref(c), 5) == rc.RC_ERR_ARG      # unknown entry
    assert lb.rc_status_string(rc.RC_ERR_MASK_NOT_CACHEABLE).decode() == "mask is not cacheable"


def test_no_rows_is_a_no_op():
    # a layout without live segments has nothing to step; without static ones nothing to prefill
    only_static = rc.Layout([(0, 4), (3, 8)], "perref")
    assert _step(only_static, q=None, k=None, v=None, o=None) == rc.RC_OK
    only_live = rc.Layout([(1, 4), (2, 8)], "perref")
    assert _prefill(only_live, q=None, k=None, v=None, o=None, kc=None, vc=None) == rc.RC_OK


def test_fragmented_schedule_is_refused():
    # 32 one-token segments; every query reads the even segments (16 separate
    # runs) and odd queries also read themselves: 16 distinct lists of 15
    # runs plus one shared list of 16 -> 256 merged ranges, above the limit
    segs = [(1, 1)] * 32
    vis = [[k % 2 == 0 or (q % 2 == 1 and k == q) for k in range(32)] for q in range(32)]
    L = rc.Layout(segs, vis)
    assert _full(L) == rc.RC_ERR_UNSUPPORTED
    assert "merged key ranges" in rc.lib().rc_last_error().decode()


def test_auto_splits_and_workspace():
    # 512-row query tiles: LT 512 is one tile, X 4096 eight, so 9 per head;
    # the splits fill at most one round of 256 work-groups
    L = rc.Layout([(0, 64), (1, 512), (2, 4096)] + [(3, 4096)] * 5, "perref")
    # 216 query tiles leave 40 CUs: their short pieces would take 6 rounds, no split
    assert L.auto_splits(1, 24, 128) == 1
    assert L.workspace_bytes(1, 24, 128, 0) == 0
    assert L.auto_splits(1, 22, 128) == 1            # 198 tiles: 4 rounds on 58 CUs
    assert L.auto_splits(1, 21, 128) == rc.SPLITS_TAIL   # 189 tiles: 3 rounds on 67 CUs
    assert L.workspace_bytes(1, 21, 128, 0) == 2 * 21 * 4608 * 130 * 4
    # more query tiles than CUs: the last round's tiles split on the idle CUs
    assert L.auto_splits(1, 29, 128) == rc.SPLITS_LAST_ROUND   # 261 tiles: the last 5 over 251 idle CUs
    assert L.workspace_bytes(1, 29, 128, 0) == 2 * 5 * 512 * 130 * 4
    assert L.auto_splits(1, 56, 128) == 1            # 504 tiles: the last 248 on 8 idle CUs, not split
    assert L.auto_splits(1, 15, 128) == rc.SPLITS_TAIL   # 135 query tiles: more than half
    assert L.auto_splits(1, 14, 128) == 2            # 126 query tiles: two even splits keep one round
    # one GPU's share of 24 heads over 8: 27 query tiles, 9 splits keep one round
    assert L.auto_splits(1, 3, 128) == 9
    assert L.workspace_bytes(1, 3, 128, 0) == 9 * 3 * 4608 * 130 * 4
    assert L.auto_splits(1, 7, 128) == 4             # 63 query tiles
    assert L.auto_splits(1, 1, 128) == 28            # 9 query tiles (393 key tiles allow up to 49)
    # few key tiles cap the splits at one per 8 key tiles
    L2 = rc.Layout([(1, 64), (2, 64)], "perref")
    assert L2.auto_splits(1, 1, 128) == 1


def test_step_launch_shape():
    # the headline step: 9 query tiles of 512 rows per head (LT 512 + X 4096)
    L = rc.Layout([(0, 64), (1, 512), (2, 4096)] + [(3, 4096)] * 5, "perref")
    assert L.launch_shape(1, 24, 128) == (216, 512, 1)
    assert L.launch_shape(1, 24, 128, rc.SPLITS_TAIL) == (432, 512, 2)
    assert L.launch_shape(1, 24, 128, rc.SPLITS_BALANCED) == (256, 256, rc.SPLITS_BALANCED)
    assert L.launch_shape(1, 24, 128, 3) == (648, 512, 3)
    assert L.launch_shape(2, 24, 128, 1) == (432, 512, 1)
    # more query tiles than CUs: the last-round split (B = 2: 432 tiles, the
    # last 176 as two pieces each; 32 heads: 288 tiles, the last 32 split);
    # where it does not apply (one round) the step runs unsplit
    assert L.launch_shape(2, 24, 128) == (432 + 176, 512, rc.SPLITS_LAST_ROUND)
    assert L.launch_shape(1, 32, 128) == (288 + 32, 512, rc.SPLITS_LAST_ROUND)
    assert L.launch_shape(1, 32, 128, rc.SPLITS_LAST_ROUND, fp8=True) == (320, 512, rc.SPLITS_LAST_ROUND)
    assert L.launch_shape(1, 24, 128, rc.SPLITS_LAST_ROUND) == (216, 512, 1)
    assert L.workspace_bytes(1, 32, 128, rc.SPLITS_LAST_ROUND) == 2 * 32 * 512 * 130 * 4
    assert L.workspace_bytes(1, 24, 128, rc.SPLITS_LAST_ROUND) == 0
    # the FP8 step tiles its queries as the bf16 step does, and splits the same way
    assert L.launch_shape(1, 24, 128, 0, fp8=True) == (216, 512, 1)
    assert L.launch_shape(1, 24, 128, rc.SPLITS_TAIL, fp8=True) == (432, 512, 2)
    # 15 heads: 135 tiles take the tail split
    assert L.launch_shape(1, 15, 128) == (270, 512, 2)
    assert L.launch_shape(1, 15, 128, 0, fp8=True) == (270, 512, 2)
    # 7 heads: 63 tiles under the automatic choice of 4 even splits
    assert L.launch_shape(1, 7, 128, 0, fp8=True) == L.launch_shape(1, 7, 128) == (4 * 7 * 9, 512, 4)
    for kw, status in ((dict(D=96), rc.RC_ERR_UNSUPPORTED), (dict(splits=-4), rc.RC_ERR_ARG),
                       (dict(splits=33), rc.RC_ERR_ARG), (dict(B=0), rc.RC_ERR_ARG),
                       (dict(splits=rc.SPLITS_BALANCED, fp8=True), rc.RC_ERR_UNSUPPORTED)):
        args = dict(B=1, H=2, D=128, splits=0, fp8=False)
        args.update(kw)
        with pytest.raises(rc.RcError) as e:
            L.launch_shape(args["B"], args["H"], args["D"], args["splits"], args["fp8"])
        assert e.value.status == status
    wg, bm, sp = ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int32()
    assert rc.lib().rc_step_launch_shape(ctypes.byref(L.c), 1, 2, 128, 0, 0, None, ctypes.byref(bm),
                                         ctypes.byref(sp)) == rc.RC_ERR_ARG


def test_full_last_round_split_workspace():
    """rc_full_workspace_bytes: 2 T 512 (D + 2) 4 bytes for the T query tiles
    of the grid's partial last round, when the idle CUs run at most three
    rounds of short pieces and every split tile has >= 16 key tiles."""
    # the dense Base over [LT, X, R] at five references: 49 tiles x 24 heads =
    # 1176 work-groups, T = 152 on 104 idle CUs (two rounds of short pieces)
    Lb = rc.Layout([(1, 512), (2, 4096)] + [(3, 4096)] * 5, "dense")
    assert Lb.full_workspace_bytes(1, 24, 128) == 2 * 152 * 512 * 130 * 4
    # B = 2: 2352 work-groups, T = 48
    assert Lb.full_workspace_bytes(2, 24, 128) == 2 * 48 * 512 * 130 * 4
    # one round or whole rounds: nothing to split
    assert Lb.full_workspace_bytes(1, 4, 128) == 0          # 196 work-groups
    L2 = rc.Layout([(1, 512), (2, 3584)], "dense")           # 8 tiles per head
    assert L2.full_workspace_bytes(1, 64, 64) == 0           # 512 work-groups
    # 36 heads: 1764 work-groups, 228 tiles in the last round on 28 idle CUs
    # (nine rounds of short pieces): not split
    assert Lb.full_workspace_bytes(1, 36, 128) == 0
    # the per-reference mask's anchor tiles (one key tile) in the last round: not split
    Lp = rc.Layout([(0, 64), (1, 512), (2, 4096)] + [(3, 4096)] * 5, "perref")
    assert Lp.full_workspace_bytes(1, 24, 128) == 0
    for kw in (dict(D=96), dict(B=0), dict(H=0)):
        args = dict(B=1, H=24, D=128)
        args.update(kw)
        assert Lb.full_workspace_bytes(args["B"], args["H"], args["D"]) == 0
    # a workspace that is too small or misaligned is refused before any launch;
    # none at all runs the unsplit recompute
    need = Lb.full_workspace_bytes(1, 24, 128)
    W = rc.RC_ERR_WORKSPACE
    assert _full_ws(Lb, H=24, ws=FAKE, wsb=need - 1) == W
    assert _full_ws(Lb, H=24, ws=FAKE + 4, wsb=need) == W


def test_prefill_launch_plan():
    """The bf16 prefill's cache store split: copy work-groups appended to the
    attention grid (at most one per CU its partial last round leaves free)
    take the first rows, the store kernel the rest."""
    head = [(0, 64), (1, 512), (2, 4096)]
    # five references, per-reference mask: 41 query tiles x 24 heads = 984
    # work-groups, 24 of them one-key-tile anchor rows; the 960 reference
    # tiles leave 64 CUs idle in the last round, where the model fits 53% of
    # the 24 x 20 544 cache rows
    L5 = rc.Layout(head + [(3, 4096)] * 5, "perref")
    assert L5.prefill_plan(1, 24, 128) == (984, 64, 262144)
    # one reference: a single partial round; every row goes with the attention,
    # on as few of the 64 idle CUs as can take them (24: 4 160 rows each)
    L1 = rc.Layout(head + [(3, 4096)], "perref")
    assert L1.prefill_plan(1, 24, 128) == (216, 24, 24 * 4160)
    # the paper mask's references read each other: long work-groups, the whole cache fits
    Lp = rc.Layout(head + [(3, 4096)] * 5, "paper")
    a, c, r = Lp.prefill_plan(1, 24, 128)
    assert (a, c, r) == (984, 24, 24 * Lp.rows(rc.ROWS_CACHED))
    # 256 equal work-groups fill whole rounds: no copy work-groups
    Ls = rc.Layout([(0, 64), (1, 64), (2, 256), (3, 256), (3, 256), (3, 256)], "paper")
    assert Ls.prefill_plan(2, 32, 64) == (256, 0, 0)
    rng = random.Random(5)
    for _ in range(300):
        kinds, lens = random_layout(rng)
        L = rc.Layout(list(zip(kinds, lens)), "perref")
        B, H = rng.choice([1, 2, 3]), rng.choice([1, 2, 5, 24, 64])
        try:
            a, c, r = L.prefill_plan(B, H, 128)
        except rc.RcError as e:
            assert e.status == rc.RC_ERR_MASK_NOT_CACHEABLE
            continue
        total = B * H * L.rows(rc.ROWS_CACHED)
        assert 0 <= c <= 256 and 0 <= r <= total
        assert (c == 0) == (r == 0)
        if c:
            assert r >= c * 64
    for kw in (dict(D=96), dict(B=0), dict(H=0)):
        args = dict(B=1, H=2, D=128)
        args.update(kw)
        with pytest.raises(rc.RcError):
            L5.prefill_plan(args["B"], args["H"], args["D"])
    a, c = ctypes.c_int64(), ctypes.c_int32()
    assert rc.lib().rc_prefill_launch_plan(ctypes.byref(L5.c), 1, 2, 128, ctypes.byref(a), ctypes.byref(c),
                                           None) == rc.RC_ERR_ARG


def _tiles(kinds, lens, vis, rows, keys, bm=512):
    """Key tiles of each query tile, in the kernel's per-head tile order:
    query segments `rows` in sequence order, tiles of bm rows inside each; a
    segment's visible key segments merged into runs that are adjacent in the
    key buffer (the segments `keys`, in sequence order), 64 keys per tile."""
    pos, p = {}, 0
    for i in keys:
        pos[i] = p
        p += lens[i]
    out = []
    for q in rows:
        runs = []
        for k in range(len(kinds)):
            if not vis[q][k]:
                continue
            if runs and runs[-1][0] + runs[-1][1] == pos[k]:
                runs[-1][1] += lens[k]
            else:
                runs.append([pos[k], lens[k]])
        out += [sum(-(-n // 64) for _, n in runs)] * (-(-lens[q] // bm))
    return out


def _model_copy_plan(kinds, lens, vis, B, H):
    """The prefill's copy plan as the header documents it, written out: a
    dispatch model of the attention grid (work-group i to XCD i mod 8, there
    to the first of 32 CUs to free; key tiles + 2 tile times each), up to 256
    copy work-groups after it, the first c with the largest c x (shortest
    window), at least 64 rows each, 64 rows per tile time, and the fewest that
    take every row when they can."""
    import heapq
    static = [i for i, k in enumerate(kinds) if k in (0, 3)]
    tiles = _tiles(kinds, lens, vis, static, static)
    nt = len(tiles)
    R = B * H * sum(lens[i] for i in om.cached_segments(kinds, vis))
    A = H * nt if (B > 1 and 2 * H * nt > 256) else B * H * nt
    if R <= 0 or R >= 2 ** 31 or A <= 0 or A > 65536:
        return 0, 0
    heaps = [[0] * 32 for _ in range(8)]
    per, rem, end = A >> 3, A & 7, 0
    for bid in range(A):
        x, kx = bid & 7, bid >> 3
        w = x * (per + 1) + kx if x < rem else rem * (per + 1) + (x - rem) * per + kx
        fin = heapq.heappop(heaps[x]) + tiles[w % nt] + 2
        heapq.heappush(heaps[x], fin)
        end = max(end, fin)
    win, window, best = [], end, 0
    for j in range(256):
        window = min(window, end - heapq.heappop(heaps[(A + j) & 7]))
        win.append(window)
        if (j + 1) * window > (best * win[best - 1] if best else 0):
            best = j + 1
    c = min(best, R // 64)
    if c <= 0:
        return 0, 0
    if c * 64 * win[c - 1] >= R:
        c = next(m for m in range(1, c + 1) if m * 64 * win[m - 1] >= R)
    return c, min(R, c * 64 * win[c - 1])


def _model_last_round(kinds, lens, vis, B, H):
    """The full recompute's last-round split as documented: T = A mod 256 of
    A > 256 whole tiles, R = ceil(T / (256 - T)) <= 3 rounds of short pieces,
    every split tile >= 16 key tiles."""
    every = list(range(len(kinds)))
    tiles = _tiles(kinds, lens, vis, every, every)
    nt = len(tiles)
    A = B * H * nt
    T = A % 256
    if A <= 256 or T == 0 or -(-T // (256 - T)) > 3:
        return 0
    if any(tiles[w % nt] < 16 for w in range(A - T, A)):
        return 0
    return T


def test_launch_plans_match_their_documented_models():
    """The prefill's copy plan and the full recompute's last-round split
    against their models written out in Python, over random layouts, mask
    presets, batch sizes and head counts (grids from one work-group to many
    rounds)."""
    rng = random.Random(23)
    n_copy = n_split = 0
    for _ in range(150):
        kinds, lens = random_layout(rng)
        preset = rng.choice(["paper", "perref", "isolated", "dense"])
        L = rc.Layout(list(zip(kinds, lens)), preset)
        vis = L.visible
        B, H = rng.choice([1, 2, 3]), rng.choice([1, 2, 5, 24, 40, 96])
        T = _model_last_round(kinds, lens, vis, B, H)
        assert L.full_workspace_bytes(B, H, 128) == 2 * T * 512 * 130 * 4, (kinds, lens, preset, B, H)
        n_split += T > 0
        if not om.is_cacheable(kinds, om.PRESETS[preset](kinds)) or L.rows(rc.ROWS_STATIC) == 0:
            continue
        _, c, r = L.prefill_plan(B, H, 128)
        assert (c, r) == _model_copy_plan(kinds, lens, vis, B, H), (kinds, lens, preset, B, H)
        n_copy += c > 0
    assert n_copy > 20 and n_split > 5, (n_copy, n_split)


def test_binding_checks_row_counts():
    """Every read and write is sized from the layout's row count, so the
    binding refuses Q with another token count before anything else (no GPU
    needed: the check comes before the device check)."""
    import torch
    L = rc.Layout([(0, 8), (1, 16), (2, 64), (3, 64)], "perref")   # 72 static, 80 live, 152 rows
    cases = ((rc.ref_kv_prefill, 72), (rc.step_masked_attention, 80), (rc.full_attention, 152),
             (rc.ref_kv_prefill_fp8, 72), (rc.step_masked_attention_fp8, 80))
    for fn, n in cases:
        for bad in (n - 1, n + 1):
            q = torch.zeros(1, bad, 2, 64, dtype=torch.bfloat16)
            args = (L, q, q, q) + ((None, None) if fn is rc.step_masked_attention else
                                   (None, None, None) if fn is rc.step_masked_attention_fp8 else ())
            with pytest.raises(ValueError, match=f"\\[B, {n}, H, D\\]"):
                fn(*args)


def test_binding_rejects_host_tensors():
    """The library takes raw device pointers: the binding refuses host tensors
    (and mismatched shapes) before any call into it."""
    import pytest
    import torch
    L = rc.Layout([(0, 8), (1, 16), (2, 64), (3, 64)], "perref")
    qs, ql, qa = (torch.zeros(1, n, 2, 64, dtype=torch.bfloat16) for n in (72, 80, 152))
    for fn in (lambda: rc.ref_kv_prefill(L, qs, qs, qs),
               lambda: rc.full_attention(L, qa, qa, qa),
               lambda: rc.step_masked_attention(L, ql, ql, ql, None, None)):
        with pytest.raises(ValueError, match="GPU tensor"):
            fn()


def _lin(M=300, N=256, K=192, a=FAKE, lda=None, w=FAKE, r=None, ldr=0, out=FAKE, ldo=None):
    lda = K if lda is None else lda
    ldo = N if ldo is None else ldo
    return rc.lib().rc_linear(M, N, K, a, lda, w, r, ldr, out, ldo, None)


def test_linear_argument_errors_launch_nothing():
    A, U = rc.RC_ERR_ARG, rc.RC_ERR_UNSUPPORTED
    assert _lin(M=-1) == A
    assert _lin(M=2 ** 40 + 1) == A
    assert _lin(M=2 ** 40) == A                     # grid of 2^34 work-groups
    assert _lin(N=0) == A and _lin(K=0) == A
    assert _lin(N=192) == U and _lin(K=96) == U     # off the 128 / 64 tile multiples
    assert _lin(K=2 ** 22 + 64, lda=2 ** 22 + 64) == U
    assert _lin(lda=128) == A                       # lda < K
    assert _lin(lda=196) == A                       # not a multiple of 8
    assert _lin(lda=2 ** 22 + 8) == A
    assert _lin(ldo=248) == A
    assert _lin(r=FAKE, ldr=128) == A               # ldr < N
    assert _lin(a=FAKE + 8) == A                    # misaligned
    assert _lin(r=FAKE + 2, ldr=256) == A
    assert _lin(w=None) == A and _lin(out=None) == A
    assert _lin(lda=128) == A
    assert "linear" in rc.lib().rc_last_error().decode()
    assert _lin(M=0, a=None, w=None, out=None) == rc.RC_OK   # nothing to do


def test_linear_binding_rejects_host_tensors():
    import torch
    a = torch.zeros(4, 64, dtype=torch.bfloat16)
    w = torch.zeros(128, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="GPU tensor"):
        rc.linear(a, w)


def test_fp8_cache_rows_and_errors():
    # the FP8 cache holds the bf16 cache's rows: ST 5 + R 33 + R 7
    L = rc.Layout([(0, 5), (1, 8), (2, 16), (3, 33), (3, 7)], "perref")
    assert L.rows(rc.ROWS_CACHED) == 45
    assert rc.fp8_cache_shapes(L, 2, 3, 64) == ((2, 3, 45, 64), (2, 3, 45, 64), (2, 3, 2))
    lb = rc.lib()
    A, U = rc.RC_ERR_ARG, rc.RC_ERR_UNSUPPORTED
    args = lambda **kw: dict(dict(q=FAKE, k=FAKE, v=FAKE, o=FAKE, kc=FAKE, vc=FAKE, sc=FAKE, splits=1), **kw)

    def step8(**kw):
        a = args(**kw)
        return lb.rc_step_masked_attention_fp8(ctypes.byref(L.c), 1, 2, 64, 0.125, a["q"], a["k"], a["v"], 128,
                                               a["kc"], a["vc"], a["sc"], a["o"], None, a["splits"], None, 0, None)

    def pre8(**kw):
        a = args(**kw)
        return lb.rc_ref_kv_prefill_fp8(ctypes.byref(L.c), 1, 2, 64, 0.125, a["q"], a["k"], a["v"], 128, a["o"],
                                        None, a["kc"], a["vc"], a["sc"], None)

    assert step8(sc=None) == A and pre8(sc=None) == A
    assert step8(sc=FAKE + 2) == A and pre8(sc=FAKE + 2) == A   # scales need 4-byte alignment
    assert step8(kc=FAKE + 8) == A and pre8(vc=FAKE + 8) == A    # caches need 16-byte alignment
    assert step8(splits=-1) == U
    assert "balanced" in lb.rc_last_error().decode()


def test_fp8_cache_key_limit():
    """The amax pass runs one grid row per 256 cached keys: at most 65535 x 256."""
    lb = rc.lib()
    lim = 65535 * 256
    for n_ref, ok in ((lim - 16, True), (lim - 15, False)):
        L = rc.Layout([(0, 16), (1, 16), (2, 64), (3, n_ref)], "perref")
        n_cached = L.rows(rc.ROWS_CACHED)
        assert (n_cached <= lim) == ok
        if ok:
            continue
        st = lb.rc_step_masked_attention_fp8(ctypes.byref(L.c), 1, 2, 64, 0.125, FAKE, FAKE, FAKE, 128, FAKE,
                                             FAKE, FAKE, FAKE, None, 1, None, 0, None)
        assert st == rc.RC_ERR_ARG and "exceeds" in lb.rc_last_error().decode()
        st = lb.rc_ref_kv_prefill_fp8(ctypes.byref(L.c), 1, 2, 64, 0.125, FAKE, FAKE, FAKE, 128, FAKE, None,
                                      FAKE, FAKE, FAKE, None)
        assert st == rc.RC_ERR_ARG and "exceeds" in lb.rc_last_error().decode()
