"""GPU checks of the FP8 reference cache against the oracle on the same seeded
inputs.

* The prefill writes, at every cached position (the rows of the bf16 cache),
  the e4m3fn code of the oracle's quantisation (bit-exact) and the oracle's
  power-of-two scales (exact); its O and LSE are those of the bf16 prefill, bit
  for bit (the same kernel).
* The step's output equals attention over the dequantised cache within the
  standard tolerance (max-abs 2e-2, rel-L2 5e-3; LSE 1e-3): the quantisation is
  part of the definition, so only the usual accumulation-order differences
  remain.
* The FP8 approximation itself, against the bf16 cache: relative L2 of O at
  most 0.1 -- one e4m3 rounding (at most 2^-4 relative, about 3.6% RMS) on each
  cached K and V value perturbs the scores by a few percent of their spread and
  the outputs by a few percent (measured values are printed)."""
import numpy as np
import pytest
import torch

import paper_2608_21229_amd as rc
from oracle import attention as oa
from oracle import fp8 as of
from oracle import masks as om
from synthgen import Workload, workload
from tests.parity_util import check, check_lse, draw_inputs, f64, sample_rows

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
FP8_REL_L2 = 0.1


def decode(u8: torch.Tensor) -> np.ndarray:
    return u8.cpu().view(torch.float8_e4m3fn).float().numpy().astype(np.float64)


def check_fp8_request(wl, preset, every=None, splits=0, steps=(0,)):
    inp0 = draw_inputs(wl, step=steps[0])
    L = rc.Layout(list(zip(inp0.kinds, inp0.lens)), preset)
    vis = om.PRESETS[preset](inp0.kinds)
    scale = wl.scale
    q, k, v = (t.to(DEV) for t in inp0.static)
    print(f"[case] fp8 {wl.name}/{preset} B={wl.B} H={wl.H} D={wl.D} splits={splits}", flush=True)
    o, lse, k8, v8, sc = rc.ref_kv_prefill_fp8(L, q, k, v, scale=scale, want_lse=True)
    o_b, lse_b, kc_b, vc_b = rc.ref_kv_prefill(L, q, k, v, scale=scale, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(o, o_b) and torch.equal(lse, lse_b), "FP8 prefill O/LSE differ from the bf16 prefill"
    # oracle cache (only the cache is needed: one prefill row evaluated)
    qs, ks, vs = (f64(t) for t in inp0.static)
    _, _, _, kc_ref, vc_ref = oa.reference_prefill(inp0.kinds, inp0.lens, vis, qs, ks, vs, scale, rows=[0])
    kq, ksc = of.quantize_cache(kc_ref)
    vq, vsc = of.quantize_cache(vc_ref)
    assert tuple(k8.shape) == tuple(v8.shape) == kq.shape
    assert np.array_equal(decode(k8), kq), "K codes differ from the oracle's quantisation"
    assert np.array_equal(decode(v8), vq), "V codes differ from the oracle's quantisation"
    scg = sc.cpu().numpy().astype(np.float64)
    assert np.array_equal(scg[..., 0], ksc) and np.array_equal(scg[..., 1], vsc), "scales differ"
    kdq, vdq = of.dequantize(kq, ksc), of.dequantize(vq, vsc)
    for s in steps:
        inp = draw_inputs(wl, step=s)
        ql, kl, vl = (t.to(DEV) for t in inp.live)
        ol, lsel = rc.step_masked_attention_fp8(L, ql, kl, vl, k8, v8, sc, splits=splits, scale=scale, want_lse=True)
        ob, _ = rc.step_masked_attention(L, ql, kl, vl, kc_b, vc_b, splits=splits, scale=scale)
        torch.cuda.synchronize()
        nl = ol.shape[1]
        rws = None if every is None else sample_rows(nl, every, seed=s + 1)
        Ol, lsl, _ = oa.denoise_step(inp.kinds, inp.lens, vis, *(f64(t) for t in inp.live), kdq, vdq, scale, rws)
        tag = f"fp8 {wl.name}/{preset} step{s} splits={splits}"
        check(ol, Ol, tag + " O", rws)
        check_lse(lsel, lsl, tag, rws)
        d = (ol.float() - ob.float()).norm().item() / ob.float().norm().item()
        print(f"[fp8] {tag}: rel-L2 of the FP8 output against the bf16 cache's = {d:.3e}", flush=True)
        assert d <= FP8_REL_L2


@pytest.mark.parametrize("preset", ["perref", "paper", "isolated"])
def test_fp8_tiny(preset):
    check_fp8_request(workload("tiny"), preset, steps=(0, 1))


RAGGED = [
    ("r1", [(0, 5), (1, 33), (2, 129), (3, 1), (3, 65), (3, 127)]),
    ("r2", [(1, 7), (2, 64), (0, 3), (3, 200), (3, 63)]),
]


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("name,segs", RAGGED)
def test_fp8_ragged(name, segs, D):
    wl = Workload(f"{name}_D{D}", 2, 3, D, tuple(segs), seed=17)
    for splits in (1, 3, 0):
        check_fp8_request(wl, "perref", splits=splits)
    check_fp8_request(wl, "paper")


def test_fp8_every_range_length_mod_16():
    """One cached range of every length 1..17 (and 31, 33, 63): ragged 8-bit
    tiles (rows past the range end load as zeros) at every alignment."""
    lens = list(range(1, 18)) + [31, 33, 63]
    segs = [(0, 16), (1, 16), (2, 64)] + [(3, n) for n in lens]
    wl = Workload("fp8_lengths", 1, 2, 64, tuple(segs), seed=23)
    check_fp8_request(wl, "perref", splits=1)
    check_fp8_request(wl, "isolated", splits=0)


def test_fp8_headline():
    """The 5-reference workload at full size (24 heads, 20 544 cached keys),
    sampled rows of steps 0, 19 and 39 over the one quantised cache."""
    check_fp8_request(workload("ref5"), "perref", every=97, steps=(0, 19, 39))


def test_fp8_cfg_two_branch_batch():
    """Both guidance branches in one batch at the headline shape: the step's
    entries run as consecutive launches, each with its own scales."""
    wl = workload("ref5")
    wl = Workload("ref5_cfg_fp8", 2, wl.H, wl.D, wl.segments, seed=7)
    check_fp8_request(wl, "perref", every=113, splits=1)


def test_fp8_last_round_split():
    """More query tiles than CUs (32 heads: 288 tiles): the last round's tiles
    as long and short pieces over the FP8 cache."""
    wl = workload("ref5")
    wl = Workload("ref5_h32_fp8", 1, 32, 128, wl.segments, seed=23)
    assert rc.Layout(list(wl.segments), "perref").auto_splits(1, 32, 128) == rc.SPLITS_LAST_ROUND
    check_fp8_request(wl, "perref", every=71, splits=0)


def test_fp8_three_head_share_split_kv():
    wl = workload("ref5")
    wl = Workload("ref5_h3_fp8", 1, 3, 128, wl.segments, seed=19)
    check_fp8_request(wl, "perref", every=29, splits=0)


def test_fp8_refuses_balanced_schedule():
    wl = workload("tiny")
    inp = draw_inputs(wl)
    L = rc.Layout(list(zip(inp.kinds, inp.lens)), "perref")
    q, k, v = (t.to(DEV) for t in inp.static)
    _, _, k8, v8, sc = rc.ref_kv_prefill_fp8(L, q, k, v)
    ql, kl, vl = (t.to(DEV) for t in inp.live)
    with pytest.raises(rc.RcError) as e:
        rc.step_masked_attention_fp8(L, ql, kl, vl, k8, v8, sc, splits=rc.SPLITS_BALANCED)
    assert e.value.status == rc.RC_ERR_UNSUPPORTED
