"""Shared helpers for the GPU parity tests: seeded inputs for a workload,
buffer assembly by segment, and the benchmark spec's tolerance check
(max-abs <= 2e-2 and relative L2 <= 5e-3 against the fp64 oracle)."""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

import numpy as np
import torch

from synthgen import ANCHOR, REF, TEXT, TARGET, Workload, bf16_normal, derive_seed

MAX_ABS = 2e-2
REL_L2 = 5e-3
# LSE: fp32 logits from exact bf16 products (relative error ~D 2^-24) and one
# log of an fp32 row sum of the unrounded weights, so the expected error is
# ~1e-5; 1e-3 leaves two orders of margin.
LSE_ABS = 1e-3


def is_static(kind):
    return kind in (ANCHOR, REF)


@dataclasses.dataclass
class Inputs:
    kinds: List[int]
    lens: List[int]
    static: tuple   # (q, k, v) [B, N_static, H, D] bf16 CPU
    live: tuple     # (q, k, v) [B, N_live, H, D] bf16 CPU


def draw_inputs(wl: Workload, layer: int = 0, step: int = 0, std: Optional[float] = None) -> Inputs:
    std = wl.std if std is None else std
    ns = sum(n for k, n in wl.segments if is_static(k))
    nl = sum(n for k, n in wl.segments if not is_static(k))
    st = tuple(bf16_normal((wl.B, ns, wl.H, wl.D), derive_seed(wl.seed, layer, 0, t), std) for t in range(3))
    lv = tuple(bf16_normal((wl.B, nl, wl.H, wl.D), derive_seed(wl.seed, layer, step + 1, 3 + t), std)
               for t in range(3))
    return Inputs(wl.kinds, wl.lens, st, lv)


def full_sequence(inp: Inputs, which: int) -> torch.Tensor:
    """Interleave the static and live buffers back into sequence order."""
    parts, si, li = [], 0, 0
    for k, n in zip(inp.kinds, inp.lens):
        if is_static(k):
            parts.append(inp.static[which][:, si:si + n])
            si += n
        else:
            parts.append(inp.live[which][:, li:li + n])
            li += n
    return torch.cat(parts, dim=1).contiguous()


def f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def check(gpu: torch.Tensor, ref: np.ndarray, what: str, rows=None):
    g = f64(gpu if rows is None else gpu[:, rows])
    assert g.shape == ref.shape, (what, g.shape, ref.shape)
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    err = g - ref
    max_abs = float(np.abs(err).max()) if err.size else 0.0
    nref = float(np.linalg.norm(ref))
    rel = float(np.linalg.norm(err) / nref) if nref > 0 else float(np.linalg.norm(err))
    print(f"[parity] {what}: max_abs={max_abs:.3e} rel_l2={rel:.3e} n={ref.size}", flush=True)
    assert max_abs <= MAX_ABS, f"{what}: max_abs {max_abs:.3e} > {MAX_ABS}"
    assert rel <= REL_L2, f"{what}: rel_l2 {rel:.3e} > {REL_L2}"
    return max_abs, rel


def check_lse(gpu: torch.Tensor, ref: np.ndarray, what: str, rows=None):
    g = f64(gpu if rows is None else gpu[:, :, rows])
    fin = np.isfinite(ref)
    assert np.array_equal(fin, np.isfinite(g)), f"{what}: -inf pattern differs"
    d = float(np.abs(g[fin] - ref[fin]).max()) if fin.any() else 0.0
    print(f"[parity] {what} lse: max_abs={d:.3e}", flush=True)
    assert d <= LSE_ABS


def sample_rows(n: int, every: int, seed: int = 0) -> np.ndarray:
    """Every `every`-th row from a seeded offset, plus the first and last row."""
    off = seed % every
    rows = set(range(off, n, every)) | {0, n - 1}
    return np.array(sorted(rows), dtype=np.int64)
