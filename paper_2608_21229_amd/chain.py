"""Chained synthetic DiT layers on the library's kernels.

Each layer projects its input hidden state to Q, K and V (Sec. 3.1, Eq. 2:
a layer's K and V are projections of that layer's input), runs the masked
attention, and adds the output projection to the residual:

    qkv = h W_qkv^T            rc_linear; W_qkv rows are the Q heads, then the
                               K heads, then the V heads (D each)
    O   = attention(Q, K, V)   Q/K/V are strided views of qkv (token stride 3 H D)
    h'  = h + O W_o^T          rc_linear with the residual

Three ways through the stack:
    prefill  the static rows (ST and R) through every layer; each layer's
             attention stores that layer's reference K/V cache
    step     the live rows (LT and X) through every layer over those caches
    full     every row through every layer: the recompute baseline, in which
             every token is re-projected and attended at each step

With ``cache="fp8"`` each layer's reference cache is stored as e4m3 codes
with per-(batch, head) scales (``ref_kv_prefill_fp8`` /
``step_masked_attention_fp8``); the computation stays bf16.

Marshalling only: every multiply-add runs in librefcache.  Work buffers come
from torch's allocator; ``collect`` (a list) receives a copy of the hidden
state after each layer.
"""
from __future__ import annotations

import math
from typing import List, Optional, Sequence, Tuple

from . import binding as rcb


class Chain:
    """A stack of synthetic layers with fixed weights and block mask.

    w_qkv[l]: [3 H D, H D] bf16, w_o[l]: [H D, H D] bf16, on one GPU."""

    def __init__(self, layout: rcb.Layout, w_qkv: Sequence, w_o: Sequence, H: int, D: int,
                 scale: Optional[float] = None, cache: str = "bf16"):
        if len(w_qkv) != len(w_o) or not w_qkv:
            raise ValueError("need one W_qkv and one W_o per layer")
        if cache not in ("bf16", "fp8"):
            raise ValueError(f"cache must be 'bf16' or 'fp8', got {cache!r}")
        self.cache = cache
        C = H * D
        for l, (wq, wo) in enumerate(zip(w_qkv, w_o)):
            if tuple(wq.shape) != (3 * C, C) or tuple(wo.shape) != (C, C):
                raise ValueError(f"layer {l}: W_qkv must be [{3 * C}, {C}] and W_o [{C}, {C}], "
                                 f"got {tuple(wq.shape)} and {tuple(wo.shape)}")
        self.layout, self.w_qkv, self.w_o = layout, list(w_qkv), list(w_o)
        self.H, self.D, self.C = H, D, C
        self.scale = 1.0 / math.sqrt(D) if scale is None else scale

    @property
    def layers(self) -> int:
        return len(self.w_qkv)

    def _buffers(self, h, rows_kind: int):
        torch = rcb._torch()
        if h.dim() != 3 or h.shape[2] != self.C:
            raise ValueError(f"hidden state must be [B, N, {self.C}], got {tuple(h.shape)}")
        B, N, _ = h.shape
        want = self.layout.rows(rows_kind)
        if N != want:
            raise ValueError(f"hidden state has {N} rows, the layout {want}")
        qkv = torch.empty((B * N, 3 * self.C), dtype=torch.bfloat16, device=h.device)
        o = torch.empty((B, N, self.H, self.D), dtype=torch.bfloat16, device=h.device)
        work = torch.empty((B * N, self.C), dtype=torch.bfloat16, device=h.device)
        return B, N, qkv, o, work

    def _qkv_views(self, qkv, B, N):
        t = qkv.view(B, N, 3, self.H, self.D)
        return t[:, :, 0], t[:, :, 1], t[:, :, 2]

    def _run(self, h, rows_kind, attend, collect: Optional[List], last_out: bool = True, stream=None):
        B, N, qkv, o, work = self._buffers(h, rows_kind)
        src = h.reshape(B * N, self.C)
        for l in range(self.layers):
            rcb.linear(src, self.w_qkv[l], out=qkv, stream=stream)
            q, k, v = self._qkv_views(qkv, B, N)
            attend(l, q, k, v, o)
            if l + 1 < self.layers or last_out or collect is not None:
                rcb.linear(o.view(B * N, self.C), self.w_o[l], residual=src, out=work, stream=stream)
                src = work
                if collect is not None:
                    collect.append(work.view(B, N, self.C).clone())
        return src.view(B, N, self.C)

    def new_caches(self, B: int, device) -> List[Tuple]:
        """Per layer (K_cache, V_cache) bf16, or (K8, V8, scales) for the FP8 cache."""
        torch = rcb._torch()
        if self.cache == "fp8":
            ks, vs, ss = rcb.fp8_cache_shapes(self.layout, B, self.H, self.D)
            return [(torch.empty(ks, dtype=torch.uint8, device=device),
                     torch.empty(vs, dtype=torch.uint8, device=device),
                     torch.empty(ss, dtype=torch.float32, device=device)) for _ in range(self.layers)]
        nc = self.layout.rows(rcb.ROWS_CACHED)
        shape = (B, self.H, nc, self.D)
        return [(torch.empty(shape, dtype=torch.bfloat16, device=device),
                 torch.empty(shape, dtype=torch.bfloat16, device=device)) for _ in range(self.layers)]

    def prefill(self, h_static, caches=None, collect: Optional[List] = None, stream=None):
        """h_static [B, N_static, H D]: the ST and R rows in sequence order.
        Fills and returns one cache entry per layer (see ``new_caches``).  The static
        rows' output projection of the last layer is skipped (nobody reads
        it) unless ``collect`` asks for the hidden states."""
        caches = self.new_caches(h_static.shape[0], h_static.device) if caches is None else caches
        if len(caches) != self.layers:
            raise ValueError(f"need {self.layers} cache entries, got {len(caches)}")

        def attend(l, q, k, v, o):
            if self.cache == "fp8":
                rcb.ref_kv_prefill_fp8(self.layout, q, k, v, o=o, k_cache8=caches[l][0], v_cache8=caches[l][1],
                                       kv_scale=caches[l][2], scale=self.scale, stream=stream)
            else:
                rcb.ref_kv_prefill(self.layout, q, k, v, o=o, k_cache=caches[l][0], v_cache=caches[l][1],
                                   scale=self.scale, stream=stream)

        self._run(h_static, rcb.ROWS_STATIC, attend, collect, last_out=False, stream=stream)
        return caches

    def step(self, h_live, caches, splits: int = 0, collect: Optional[List] = None, stream=None):
        """h_live [B, N_live, H D]: the LT and X rows of one denoising step.
        Returns the live rows' hidden state after the last layer."""
        if len(caches) != self.layers:
            raise ValueError(f"need {self.layers} cache entries, got {len(caches)}")
        torch = rcb._torch()
        B = h_live.shape[0]
        need = self.layout.workspace_bytes(B, self.H, self.D, splits)
        ws = torch.empty(need, dtype=torch.uint8, device=h_live.device) if need else None

        def attend(l, q, k, v, o):
            if self.cache == "fp8":
                rcb.step_masked_attention_fp8(self.layout, q, k, v, *caches[l], o=o, splits=splits, workspace=ws,
                                              scale=self.scale, stream=stream)
            else:
                rcb.step_masked_attention(self.layout, q, k, v, caches[l][0], caches[l][1], o=o, splits=splits,
                                          workspace=ws, scale=self.scale, stream=stream)

        return self._run(h_live, rcb.ROWS_LIVE, attend, collect, stream=stream)

    def full(self, h, collect: Optional[List] = None, stream=None, last_round_split: bool = True):
        """h [B, N, H D]: every row in sequence order.  Returns the hidden state
        after the last layer.  last_round_split=False computes every query tile
        whole (bit-comparable with the cached path)."""
        def attend(l, q, k, v, o):
            rcb.full_attention(self.layout, q, k, v, o=o, scale=self.scale, last_round_split=last_round_split,
                               stream=stream)

        return self._run(h, rcb.ROWS_ALL, attend, collect, stream=stream)
