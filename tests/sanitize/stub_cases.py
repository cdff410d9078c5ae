"""Planner cases for the sanitizer build (run by test_host_sanitized.py, with
REFCACHE_LIB naming a library whose kernel launchers are the checking stubs of
stub_launchers.cpp; skipped otherwise).  Every successful call hands its
schedule to a stub that aborts on a broken invariant; pointers are fake and
never dereferenced."""
import ctypes
import os
import random

import pytest

import paper_2608_21229_amd as rc
from oracle import masks as om
from tests.test_capi_host import FAKE, _full, _full_ws, _prefill, _step, random_layout

pytestmark = pytest.mark.skipif(not os.environ.get("REFCACHE_STUB"), reason="needs the stub-launcher build")


def launches():
    f = rc.lib().rc_stub_launches
    f.restype = ctypes.c_long
    return f()


@pytest.mark.parametrize("preset", ["paper", "perref", "isolated", "dense"])
def test_random_layouts_through_every_entry(preset):
    rng = random.Random(11)
    for _ in range(200):
        kinds, lens = random_layout(rng)
        L = rc.Layout(list(zip(kinds, lens)), preset)
        vis = om.PRESETS[preset](kinds)
        B, H = rng.choice([1, 2, 3]), rng.choice([1, 2, 5, 24, 64])
        D = rng.choice([64, 128])
        ts = H * D
        n0 = launches()
        assert _full(L, B=B, H=H, D=D, ts=ts, lse=FAKE) == rc.RC_OK
        assert launches() == n0 + (1 if sum(lens) else 0)
        # with the last-round split's workspace: the attention launch, plus the
        # merge when it splits
        need = L.full_workspace_bytes(B, H, D)
        n0 = launches()
        assert _full_ws(L, B=B, H=H, D=D, ts=ts, lse=FAKE, ws=FAKE, wsb=need) == rc.RC_OK
        assert launches() == n0 + (1 if sum(lens) else 0) + (1 if need else 0)
        if not om.is_cacheable(kinds, vis):
            assert _prefill(L, B=B, H=H, D=D, ts=ts) == rc.RC_ERR_MASK_NOT_CACHEABLE
            continue
        assert _prefill(L, B=B, H=H, D=D, ts=ts, lse=FAKE) == rc.RC_OK
        for splits in (1, 2, 5, 0, rc.SPLITS_TAIL, rc.SPLITS_BALANCED, rc.SPLITS_LAST_ROUND):
            need = L.workspace_bytes(B, H, D, splits)
            st = _step(L, B=B, H=H, D=D, ts=ts, splits=splits, ws=FAKE if need else None, wsb=need, lse=FAKE)
            assert st == rc.RC_OK, (kinds, lens, splits, rc.lib().rc_last_error().decode())
