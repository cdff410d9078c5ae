"""Chained synthetic DiT layers in float64 -- TEST INFRASTRUCTURE ONLY.

The masked attention of Sec. 3.3 sits inside a stack of transformer layers.
Eq. 2 makes each layer's K and V of a token a projection of that token's
hidden state at the layer's input, and a layer's output is the next layer's
input.  The smallest layer with that dependency structure (normalisation, MLP
and timestep modulation are per-token maps as well and change nothing about
which rows read which) is, per token and per head:

    [Q | K | V] = h W_qkv^T          fused projection, W_qkv [3 C, C], C = H D;
                                     its rows are the Q heads, then the K
                                     heads, then the V heads (D each)
    O           = masked softmax attention of Q over the visible K, V
    h'          = h + O W_o^T        output projection plus residual

Storage precision.  Every tensor that crosses the library boundary is bf16:
the hidden state, the fused projection and O.  The chain therefore rounds
each of them to the nearest bf16 value (ties to even) where it is stored and
does all arithmetic in between in float64.  Rounding at the same points as
the GPU path keeps the two comparable over several layers; the remaining
difference is only the accumulation order inside each stage.

Caching (Sec. 3.1, Eq. 2; App. A): under a structurally cacheable mask the
static rows (ST, R) never read a live row, at any layer, so their hidden
states -- and with them every layer's cached K/V -- do not depend on the live
inputs.  A prefill that carries only the static rows through all layers and
stores each layer's cached K/V, followed by steps that carry only the live
rows (LT, X) through all layers over those caches, yields the full
recompute's live rows.

Pins (``tests/test_oracle_chain.py``): ``round_bf16`` against torch's
float32 -> bfloat16 conversion and worked double-rounding cases; the whole
chain against a pure-Python brute force on tiny inputs; a closed form for
uniform attention with permutation weights; the identity W_o = 0; the cached
path against the full recompute.
"""
from __future__ import annotations

from typing import List, Optional, Sequence, Tuple

import numpy as np

from . import attention as oa
from .masks import Mask


def round_bf16(x) -> np.ndarray:
    """Nearest bfloat16 value of float64 ``x`` (8 significant bits, ties to
    even), as float64.  Valid in bf16's normal range (|x| >= 2^-126) and at 0;
    one rounding straight from float64, never through float32."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                    # x = m 2^e with 0.5 <= |m| < 1
    return np.ldexp(np.rint(m * 256.0), e - 8)


def project(a: np.ndarray, w: np.ndarray, residual: Optional[np.ndarray] = None) -> np.ndarray:
    """bf16(a W^T (+ residual)) for a [..., K], w [N, K], residual [..., N]."""
    y = a @ w.T
    if residual is not None:
        y = y + residual
    return round_bf16(y)


def split_qkv(qkv: np.ndarray, H: int, D: int):
    """[B, N, 3 H D] -> Q, K, V as [B, N, H, D] (Q heads first, then K, then V)."""
    B, N, _ = qkv.shape
    t = qkv.reshape(B, N, 3, H, D)
    return t[:, :, 0], t[:, :, 1], t[:, :, 2]


def _out(o: np.ndarray, h: np.ndarray, w_o: np.ndarray) -> np.ndarray:
    """h + bf16(O) W_o^T, rounded; O [B, n, H, D] -> [B, n, H D]."""
    B, n, H, D = o.shape
    return project(round_bf16(o).reshape(B, n, H * D), w_o, h)


def chain_full(kinds, lens, vis: Mask, h0: np.ndarray, w_qkv: Sequence[np.ndarray],
               w_o: Sequence[np.ndarray], H: int, D: int, scale: float):
    """Full recompute: every row of the sequence through every layer.

    h0 [B, N, C] in sequence order.  Returns (hs, kvs): hs[l] is the hidden
    state after layer l, kvs[l] the (K, V) [B, N, H, D] layer l attended over."""
    h = np.asarray(h0, dtype=np.float64)
    hs: List[np.ndarray] = []
    kvs: List[Tuple[np.ndarray, np.ndarray]] = []
    for wq, wo in zip(w_qkv, w_o):
        q, k, v = split_qkv(project(h, wq), H, D)
        o, _, _ = oa.full_attention(kinds, lens, vis, q, k, v, scale)
        h = _out(o, h, wo)
        hs.append(h)
        kvs.append((k, v))
    return hs, kvs


def chain_prefill(kinds, lens, vis: Mask, h_static: np.ndarray, w_qkv: Sequence[np.ndarray],
                  w_o: Sequence[np.ndarray], H: int, D: int, scale: float):
    """The static rows (ST and R tokens in sequence order) through every layer.

    Returns (hs, caches): hs[l] the static rows' hidden state after layer l,
    caches[l] = (K_cache, V_cache) [B, H, N_cached, D] of layer l."""
    h = np.asarray(h_static, dtype=np.float64)
    hs, caches = [], []
    for wq, wo in zip(w_qkv, w_o):
        q, k, v = split_qkv(project(h, wq), H, D)
        o, _, _, kc, vc = oa.reference_prefill(kinds, lens, vis, q, k, v, scale)
        h = _out(o, h, wo)
        hs.append(h)
        caches.append((kc, vc))
    return hs, caches


def chain_step(kinds, lens, vis: Mask, h_live: np.ndarray, caches, w_qkv: Sequence[np.ndarray],
               w_o: Sequence[np.ndarray], H: int, D: int, scale: float):
    """The live rows (LT and X tokens in sequence order) of one denoising step
    through every layer, reading layer l's cached K/V.  Returns hs[l], the
    live rows' hidden state after layer l."""
    h = np.asarray(h_live, dtype=np.float64)
    hs = []
    for (kc, vc), wq, wo in zip(caches, w_qkv, w_o):
        q, k, v = split_qkv(project(h, wq), H, D)
        o, _, _ = oa.denoise_step(kinds, lens, vis, q, k, v, kc, vc, scale)
        h = _out(o, h, wo)
        hs.append(h)
    return hs
