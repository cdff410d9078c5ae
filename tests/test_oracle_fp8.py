"""Pins for the FP8 cache oracle (oracle/fp8.py): torch's float32 ->
float8_e4m3fn conversion (a library routine), worked cases of the e4m3fn grid
(ties, subnormals, the largest value), the scale rule by search, and the
quantisation error bound."""
import numpy as np
import pytest
import torch

from oracle import chain as oc
from oracle import fp8 as of


def e4m3_values():
    v = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).float().numpy().astype(np.float64)
    return v[np.isfinite(v)]


def test_round_e4m3_matches_torch():
    vals = e4m3_values()
    pos = np.unique(np.abs(vals))
    mids = (pos[1:] + pos[:-1]) / 2                       # exact ties
    rng = np.random.default_rng(1)
    rand = rng.uniform(-448, 448, 50_000)
    small = rng.uniform(-0.05, 0.05, 50_000)
    x = np.concatenate([vals, mids, -mids, mids * (1 + 2 ** -20), mids * (1 - 2 ** -20), rand, small])
    x32 = x.astype(np.float32)                          # torch converts from float32
    want = torch.from_numpy(x32).to(torch.float8_e4m3fn).float().numpy().astype(np.float64)
    got = of.round_e4m3(x32.astype(np.float64))
    assert np.array_equal(got, want)


@pytest.mark.parametrize("x,want", [
    (1.0625, 1.0),            # tie between 1 and 1.125: even mantissa 000
    (1.1875, 1.25),           # tie between 1.125 and 1.25: even mantissa 010
    (3 * 2 ** -10, 2 ** -8),  # subnormal tie between 2^-9 (001) and 2^-8 (010)
    (2 ** -10, 0.0),          # half the smallest subnormal: ties to even zero
    (448.0, 448.0), (-448.0, -448.0), (0.0, 0.0),
    (464.0, 448.0),           # saturates
    (2.0 ** -6, 2.0 ** -6),   # smallest normal
])
def test_round_e4m3_worked_cases(x, want):
    assert of.round_e4m3(np.float64(x)) == want


def test_scale_exponent_is_minimal():
    rng = np.random.default_rng(2)
    amaxes = np.concatenate([np.exp(rng.uniform(-30, 30, 3000)), [448.0, 449.0, 224.0, 896.0, 1.0, 2.0 ** -20]])
    for a in amaxes:
        e = of.scale_exponent(a)
        assert a * 2.0 ** -e <= 448.0 and a * 2.0 ** -(e - 1) > 448.0, (a, e)
    assert of.scale_exponent(0.0) == 0


def test_quantize_cache_error_and_exactness():
    rng = np.random.default_rng(3)
    c = oc.round_bf16(rng.standard_normal((2, 3, 50, 16)) * np.array([1.0, 30.0, 0.01])[None, :, None, None])
    codes, scales = of.quantize_cache(c)
    deq = of.dequantize(codes, scales)
    # every code is an e4m3fn value, every scale a power of two, every
    # dequantised value exact in bf16
    assert np.isin(codes, e4m3_values()).all()
    assert np.array_equal(np.log2(scales), np.round(np.log2(scales)))
    assert np.array_equal(oc.round_bf16(deq), deq)
    # the largest magnitude uses the top binade: amax / s in (224, 448]
    for b in range(2):
        for h in range(3):
            r = np.abs(c[b, h]).max() / scales[b, h]
            assert 224.0 < r <= 448.0
    # error: half an e4m3 step (1/16 relative) for normals, 2^-10 s below
    err = np.abs(deq - c)
    bound = np.maximum(np.abs(c) * 2.0 ** -4, scales[:, :, None, None] * 2.0 ** -10)
    assert (err <= bound * (1 + 1e-12)).all()
