"""Seeded random layouts through every entry on the GPU against the fp64
oracle, on sampled rows: 2-7 segments of ragged, one-token and tile-aligned
lengths, all four mask presets, B from 1 to 3 and 1 to 96 heads, so that the
grids range from a few work-groups to several rounds (the prefill's copy
work-groups, the automatic split choices of the step and the full
recompute's last-round split all come up)."""
import math
import random

import pytest
import torch

import paper_2608_21229_amd as rc
from oracle import attention as oa
from oracle import masks as om
from synthgen import Workload
from tests.parity_util import check, check_lse, draw_inputs, f64, full_sequence, sample_rows
from tests.test_gpu_parity import check_request

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _case(seed):
    rng = random.Random(seed)
    n = rng.randint(2, 7)
    kinds = [rng.choice([0, 1, 2, 3]) for _ in range(n)]
    kinds[rng.randrange(n)] = rng.choice([1, 2])           # at least one live segment
    if not any(k in (0, 3) for k in kinds):
        kinds[rng.randrange(n)] = rng.choice([0, 3])       # and one static, where it fits
    lens = [rng.choice([1, 3, 31, 64, 65, 127, 200, 513, 900]) for _ in range(n)]
    preset = rng.choice(["paper", "perref", "isolated", "dense"])
    return kinds, lens, preset, rng.choice([1, 2, 3]), rng.choice([1, 3, 24, 40, 96]), rng.choice([64, 128])


def _every(B, N, H, D):
    # sample rows so that each oracle call stays near 10 GFLOP
    return max(3, math.ceil(4.0 * B * N * N * H * D / 1e10))


@pytest.mark.parametrize("seed", range(24))
def test_random_layout_every_entry(seed):
    kinds, lens, preset, B, H, D = _case(seed)
    segs = tuple(zip(kinds, lens))
    wl = Workload(f"random{seed}", B, H, D, segs, std=1.0, seed=100 + seed)
    L = rc.Layout(list(segs), preset)
    vis = om.PRESETS[preset](kinds)
    N = sum(lens)
    every = _every(B, N, H, D)
    print(f"[case] random {seed}: B={B} H={H} D={D} {list(segs)} {preset} every={every} "
          f"full_ws={L.full_workspace_bytes(B, H, D)}", flush=True)
    inp = draw_inputs(wl)
    q, k, v = (full_sequence(inp, i).to(DEV) for i in range(3))
    o, lse = rc.full_attention(L, q, k, v, scale=wl.scale, want_lse=True)
    torch.cuda.synchronize()
    rows = sample_rows(N, every, seed=seed)
    O, ls, _ = oa.full_attention(kinds, lens, vis, *(f64(t) for t in (q, k, v)), wl.scale, rows=rows)
    check(o, O, f"random{seed} full", rows)
    check_lse(lse, ls, f"random{seed} full", rows)
    if om.is_cacheable(kinds, vis) and L.rows(rc.ROWS_STATIC) > 0:
        print(f"  prefill plan {L.prefill_plan(B, H, D)}, step launch {L.launch_shape(B, H, D)}", flush=True)
        check_request(wl, preset, every=every, splits=0)
