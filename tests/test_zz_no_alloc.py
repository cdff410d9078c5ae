"""The no-allocation step entry (static scratch array) against the step entry
with a caller workspace: same kernels, so the outputs and LSE must agree bit
for bit.  Two calls in a row, the second on a smaller input, so the second
runs over the first call's leftovers in the array."""
import pytest
import torch

import paper_2608_21229_amd as rc
from synthgen import Workload, workload
from tests.parity_util import draw_inputs

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _prepare(wl, preset="perref"):
    inp = draw_inputs(wl)
    L = rc.Layout(list(zip(inp.kinds, inp.lens)), preset)
    q, k, v = (t.to(DEV) for t in inp.static)
    _, _, kc, vc = rc.ref_kv_prefill(L, q, k, v, scale=wl.scale)
    ql, kl, vl = (t.to(DEV) for t in inp.live)
    return L, (ql, kl, vl), kc, vc


def _compare(wl, L, live, kc, vc, splits):
    ql, kl, vl = live
    print(f"[case] noalloc {wl.name} B={wl.B} H={wl.H} D={wl.D} splits={splits}", flush=True)
    o_ref, lse_ref = rc.step_masked_attention(L, ql, kl, vl, kc, vc, splits=splits, scale=wl.scale, want_lse=True)
    o = torch.full_like(o_ref, float("nan"))
    lse = torch.full_like(lse_ref, float("nan"))
    rc.step_masked_attention_noalloc(L, ql, kl, vl, kc, vc, o, lse, splits=splits, scale=wl.scale)
    torch.cuda.synchronize()
    assert torch.equal(o, o_ref), f"{wl.name} splits={splits}: O differs from the workspace entry"
    assert torch.equal(lse, lse_ref), f"{wl.name} splits={splits}: LSE differs from the workspace entry"


@pytest.mark.parametrize("splits", [0, 2, rc.SPLITS_TAIL, rc.SPLITS_BALANCED])
def test_noalloc_two_calls_second_smaller(splits):
    big = Workload("ref5_h3", 1, 3, 128, workload("ref5").segments, seed=5)
    assert 0 < rc.Layout(list(big.segments), "perref").workspace_bytes(1, 3, 128, splits) <= rc.NOALLOC_SCRATCH_BYTES
    small = Workload("ragged_small", 2, 3, 64, ((1, 7), (2, 64), (0, 3), (3, 200), (3, 63)), seed=17)
    for wl in (big, small):
        L, live, kc, vc = _prepare(wl)
        _compare(wl, L, live, kc, vc, splits)


def test_noalloc_without_splits_and_over_limit():
    wl = workload("ref5")
    L, live, kc, vc = _prepare(wl)
    _compare(wl, L, live, kc, vc, 1)
    # four even splits over 24 heads need 230 MB: refused before any launch
    need = L.workspace_bytes(wl.B, wl.H, wl.D, 4)
    assert need > rc.NOALLOC_SCRATCH_BYTES
    ql, kl, vl = live
    o = torch.empty_like(ql)
    with pytest.raises(rc.RcError) as e:
        rc.step_masked_attention_noalloc(L, ql, kl, vl, kc, vc, o, splits=4, scale=wl.scale)
    assert e.value.status == rc.RC_ERR_WORKSPACE
    assert "scratch" in str(e.value)


def test_noalloc_last_round_split():
    """The last-round split through the static scratch: 32 heads at the
    5-reference shape, then a smaller ragged grid that also splits."""
    big = Workload("ref5_h32", 1, 32, 128, workload("ref5").segments, seed=25)
    small = Workload("ragged_h96", 1, 96, 64, ((0, 40), (1, 100), (2, 900), (3, 700), (3, 333)), seed=27)
    sizes = []
    for wl in (big, small):
        L, live, kc, vc = _prepare(wl)
        need = L.workspace_bytes(wl.B, wl.H, wl.D, rc.SPLITS_LAST_ROUND)
        assert 0 < need <= rc.NOALLOC_SCRATCH_BYTES
        sizes.append(need)
        _compare(wl, L, live, kc, vc, rc.SPLITS_LAST_ROUND)
    assert sizes[1] < sizes[0]
