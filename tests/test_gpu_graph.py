"""The entry points under HIP graph capture: a request (prefill and steps,
bf16 and FP8 cache) is captured once into a torch.cuda.CUDAGraph and replayed
several times, with eager work and synchronisations between the replays; every
replay equals the eager calls bit for bit (the kernels are deterministic and
the library neither allocates nor synchronises inside a call)."""
import pytest
import torch

import paper_2608_21229_amd as rc
from synthgen import Workload, workload
from tests.parity_util import draw_inputs

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _request(L, st, lives, bufs, scale, fp8, splits=1):
    """Prefill then one step per live set, into the preallocated buffers."""
    q, k, v = st
    if fp8:
        rc.ref_kv_prefill_fp8(L, q, k, v, o=bufs["o_s"], k_cache8=bufs["kc"], v_cache8=bufs["vc"],
                              kv_scale=bufs["sc"], scale=scale)
    else:
        rc.ref_kv_prefill(L, q, k, v, o=bufs["o_s"], k_cache=bufs["kc"], v_cache=bufs["vc"], scale=scale)
    for i, (ql, kl, vl) in enumerate(lives):
        if fp8:
            rc.step_masked_attention_fp8(L, ql, kl, vl, bufs["kc"], bufs["vc"], bufs["sc"], o=bufs["o_l"][i],
                                         lse=bufs["lse"][i], splits=splits, workspace=bufs.get("ws"), scale=scale)
        else:
            rc.step_masked_attention(L, ql, kl, vl, bufs["kc"], bufs["vc"], o=bufs["o_l"][i], lse=bufs["lse"][i],
                                     splits=splits, workspace=bufs.get("ws"), scale=scale)


@pytest.mark.parametrize("fp8", [False, True])
@pytest.mark.parametrize("name", ["tiny", "ragged", "wide"])
def test_request_graph_replays_equal_eager(name, fp8):
    # "wide": 96 heads, so the prefill carries copy work-groups and the step
    # runs the last-round split (288 query tiles) with a preallocated workspace
    splits = 1
    if name == "tiny":
        wl = workload("tiny")
    elif name == "ragged":
        wl = Workload("graph_ragged", 2, 3, 128, ((0, 5), (1, 33), (2, 129), (3, 65), (3, 127)), seed=13)
    else:
        wl = Workload("graph_wide", 1, 96, 64, ((0, 40), (1, 100), (2, 900), (3, 700), (3, 333)), seed=15)
        splits = rc.SPLITS_LAST_ROUND
    print(f"[case] graph {wl.name} fp8={fp8} splits={splits}", flush=True)
    inp = draw_inputs(wl)
    L = rc.Layout(list(zip(inp.kinds, inp.lens)), "perref")
    st = tuple(t.to(DEV) for t in inp.static)
    lives = [tuple(t.to(DEV) for t in draw_inputs(wl, step=s).live) for s in range(3)]
    B, H, D = wl.B, wl.H, wl.D
    ns, nl, nc = L.rows(rc.ROWS_STATIC), L.rows(rc.ROWS_LIVE), L.rows(rc.ROWS_CACHED)
    cache_dtype = torch.uint8 if fp8 else torch.bfloat16
    bufs = {"o_s": torch.empty((B, ns, H, D), dtype=torch.bfloat16, device=DEV),
            "kc": torch.empty((B, H, nc, D), dtype=cache_dtype, device=DEV),
            "vc": torch.empty((B, H, nc, D), dtype=cache_dtype, device=DEV),
            "sc": torch.empty((B, H, 2), dtype=torch.float32, device=DEV),
            "o_l": [torch.empty((B, nl, H, D), dtype=torch.bfloat16, device=DEV) for _ in lives],
            "lse": [torch.empty((B, H, nl), dtype=torch.float32, device=DEV) for _ in lives]}
    need = L.workspace_bytes(B, H, D, splits)
    if splits != 1:
        assert need > 0 and L.prefill_plan(B, H, D)[1] > 0
        bufs["ws"] = torch.empty(need, dtype=torch.uint8, device=DEV)
    # eager reference
    _request(L, st, lives, bufs, wl.scale, fp8, splits)
    torch.cuda.synchronize()
    want = [t.clone() for t in [bufs["o_s"], bufs["kc"], bufs["vc"], bufs["sc"]] + bufs["o_l"] + bufs["lse"]]
    if not fp8:
        want[3] = None
    # capture on a side stream (warmed up above), then replay
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            _request(L, st, lives, bufs, wl.scale, fp8, splits)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for rep in range(3):
        # clobber the outputs eagerly between replays
        for t in [bufs["o_s"], bufs["kc"], bufs["vc"], bufs["sc"]] + bufs["o_l"] + bufs["lse"]:
            t.fill_(7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = [bufs["o_s"], bufs["kc"], bufs["vc"], bufs["sc"]] + bufs["o_l"] + bufs["lse"]
        for i, (a, b) in enumerate(zip(got, want)):
            if b is None:
                continue
            assert torch.equal(a, b), f"replay {rep}: output {i} differs from the eager calls"
