"""FP8 (e4m3fn) reference cache in float64 -- TEST INFRASTRUCTURE ONLY.

The paper treats caching as complementary to other accelerations (Sec. 1,
Sec. 4.2).  Storing the reference K/V cache in 8-bit floating point is one such
combination: the library's FP8 cache keeps, for each (batch, head) and each of
K and V, one power-of-two scale and the e4m3fn code of every cached value.

e4m3fn (the OCP 8-bit format with 4 exponent bits, bias 7, 3 mantissa bits and
no infinities): finite values are 0, the subnormals k 2^-9 (k = 1..7) and the
normals (1 + f/8) 2^E for E = -6..8, the largest being 448 = 1.75 * 2^8.

Quantisation of a tensor X (one (b, h) slice of the cache):
    amax = max |x|
    s    = 2^e, e the smallest integer with amax / s <= 448 (s = 1 when amax = 0)
    code = nearest e4m3fn value of x / s, ties to even (x / s is exact)
and the value the attention reads is code * s.  With these definitions the
quantised cache is a deterministic function of the bf16 cache, so the FP8 step
is compared with plain attention over the dequantised cache.

Pins: ``tests/test_oracle_fp8.py`` (torch's float32 -> float8_e4m3fn
conversion, worked ties and subnormals, the scale's minimality by search).
"""
from __future__ import annotations

import numpy as np

E4M3_MAX = 448.0


def round_e4m3(x) -> np.ndarray:
    """Nearest e4m3fn value of float64 x (ties to even), saturating at +-448."""
    x = np.asarray(x, dtype=np.float64)
    ax = np.abs(x)
    m, e = np.frexp(ax)                    # ax = m 2^e, 0.5 <= m < 1
    # normal range (>= 2^-6): 4 significant bits; below it the grid is 2^-9
    normal = np.ldexp(np.rint(m * 16.0), e - 4)
    sub = np.rint(ax * 2.0 ** 9) * 2.0 ** -9
    r = np.where(ax >= 2.0 ** -6, normal, sub)
    r = np.minimum(r, E4M3_MAX)
    return np.copysign(r, x)


def scale_exponent(amax: float) -> int:
    """The smallest integer e with amax * 2^-e <= 448 (0 for amax = 0)."""
    if not amax > 0:
        return 0
    m, k = np.frexp(np.float64(amax))      # amax = m 2^k, 0.5 <= m < 1; 448 = 0.875 * 2^9
    return int(k - 9) if m <= 0.875 else int(k - 8)


def quantize_cache(c: np.ndarray):
    """c: a cache [B, H, N, D] (float64 of bf16 values).  Returns (codes, scales):
    codes [B, H, N, D] as e4m3fn values (float64) and scales [B, H] with
    code * scale the value the step reads."""
    B, H = c.shape[:2]
    codes = np.zeros_like(c, dtype=np.float64)
    scales = np.ones((B, H))
    for b in range(B):
        for h in range(H):
            s = 2.0 ** scale_exponent(float(np.abs(c[b, h]).max()) if c[b, h].size else 0.0)
            codes[b, h] = round_e4m3(c[b, h] / s)
            scales[b, h] = s
    return codes, scales


def dequantize(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    return codes * scales[:, :, None, None]
