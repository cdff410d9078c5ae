"""Workload shapes and the seeded bf16 draw.

Segment kinds follow the paper's sequence notation (Sec. 3.1, Eq. 1 and
Sec. 3.3): ST = static text anchors, LT = live text, X = denoising target,
R = reference image tokens.  A workload is a list of (kind, length)
segments in sequence order plus the attention-head shape.

The shapes stand in for the paper's Qwen-Image-Edit setting (1024^2 images:
about 4096 target tokens and 4096 tokens per reference, S = N_X + N_LT =
4608, App. C); no benchmark items or trained weights are involved.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Sequence, Tuple

import torch

ANCHOR, TEXT, TARGET, REF = 0, 1, 2, 3
KIND_NAMES = {ANCHOR: "ST", TEXT: "LT", TARGET: "X", REF: "R"}


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    D: int
    segments: Tuple[Tuple[int, int], ...]   # (kind, length) in sequence order
    std: float = 1.0                        # every Q/K/V draw is N(0,1) * std
    seed: int = 42
    steps: int = 40                         # denoising steps per request
    layers: int = 1

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.D)

    @property
    def kinds(self) -> List[int]:
        return [k for k, _ in self.segments]

    @property
    def lens(self) -> List[int]:
        return [n for _, n in self.segments]

    def with_refs(self, ref_lens: Sequence[int]) -> "Workload":
        head = tuple(s for s in self.segments if s[0] != REF)
        return dataclasses.replace(self, segments=head + tuple((REF, n) for n in ref_lens),
                                   name=f"{self.name}_k{len(ref_lens)}")


def _wl(name, B, H, D, st, lt, x, refs, **kw) -> Workload:
    segs = ((ANCHOR, st), (TEXT, lt), (TARGET, x)) + tuple((REF, n) for n in refs)
    return Workload(name, B, H, D, segs, **kw)


WORKLOADS = {
    # tiny oracle-checkable case: ragged 8/16/64/64 segments, head_dim 64
    "tiny": _wl("tiny", 1, 2, 64, 8, 16, 64, [64], steps=1),
    # single reference at 1024^2: per-head value scale 0.5
    "ref1": _wl("ref1", 1, 24, 128, 64, 512, 4096, [4096], std=0.5),
    # headline: five references of 4096 tokens (20480 cached reference keys)
    "ref5": _wl("ref5", 1, 24, 128, 64, 512, 4096, [4096] * 5),
    # reference-count scaling base (k set by with_refs)
    "scaling": _wl("scaling", 1, 24, 128, 64, 512, 4096, [4096], std=0.5),
    # 48-layer schedule with mixed-resolution references
    "mixed48": _wl("mixed48", 1, 24, 128, 64, 512, 4096, [4096] * 3 + [1024] * 3, layers=48),
}
SCALING_KS = (1, 2, 5, 8, 10)


def workload(name: str) -> Workload:
    if name.startswith("scaling_k"):
        k = int(name[len("scaling_k"):])
        return WORKLOADS["scaling"].with_refs([4096] * k)
    return WORKLOADS[name]


def derive_seed(base: int, layer: int = 0, step: int = 0, tensor: int = 0) -> int:
    """Deterministic per-(layer, step, tensor) seed; tensor 0/1/2 = Q/K/V."""
    return (base * 1_000_003 + layer * 7919 + step * 104_729 + tensor * 15_485_863) % (2 ** 62)


def bf16_normal(shape, seed: int, std: float = 1.0) -> torch.Tensor:
    """N(0,1)*std drawn in float32 on the CPU, rounded to bfloat16 (RNE)."""
    g = torch.Generator(device="cpu")
    g.manual_seed(int(seed))
    x = torch.randn(tuple(shape), generator=g, dtype=torch.float32)
    if std != 1.0:
        x = x * std
    return x.to(torch.bfloat16)


def draw_qkv(B: int, N: int, H: int, D: int, seed: int, std: float = 1.0,
             layer: int = 0, step: int = 0):
    """Q, K, V as [B, N, H, D] bf16 CPU tensors."""
    return tuple(bf16_normal((B, N, H, D), derive_seed(seed, layer, step, t), std) for t in range(3))


# ------------------------------------------------- chained synthetic layers
# Seed slots of the chained-layer draws (the `tensor` argument of derive_seed);
# 0..5 are the per-layer Q/K/V draws of the attention-only workloads.
_SLOT_H_STATIC, _SLOT_H_LIVE, _SLOT_W_QKV, _SLOT_W_O = 6, 7, 8, 9


def draw_chain_weights(H: int, D: int, layers: int, seed: int):
    """Per-layer projection weights of a chained synthetic layer, bf16 CPU:
    w_qkv [3 H D, H D] (rows: Q heads, then K heads, then V heads) and
    w_o [H D, H D], each N(0, 1 / (H D)) so that projections of an N(0,1)
    hidden state have unit variance."""
    C = H * D
    std = 1.0 / math.sqrt(C)
    w_qkv = [bf16_normal((3 * C, C), derive_seed(seed, l, 0, _SLOT_W_QKV), std) for l in range(layers)]
    w_o = [bf16_normal((C, C), derive_seed(seed, l, 0, _SLOT_W_O), std) for l in range(layers)]
    return w_qkv, w_o


def draw_hidden(wl: Workload, step: int = 0):
    """Layer-0 hidden states [B, N, H D] bf16 N(0,1): the static rows (ST and
    R tokens in sequence order, fixed for the request) and the live rows (LT
    and X tokens, fresh at each denoising step)."""
    C = wl.H * wl.D
    ns = sum(n for k, n in wl.segments if k in (ANCHOR, REF))
    nl = sum(n for k, n in wl.segments if k in (TEXT, TARGET))
    h_static = bf16_normal((wl.B, ns, C), derive_seed(wl.seed, 0, 0, _SLOT_H_STATIC))
    h_live = bf16_normal((wl.B, nl, C), derive_seed(wl.seed, 0, step + 1, _SLOT_H_LIVE))
    return h_static, h_live
