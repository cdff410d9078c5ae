"""ctypes binding of librefcache (include/refcache.h).

Argument marshalling only: tensors are passed as device pointers and the
current torch stream as a hipStream_t; every step of the computation runs in
the library's HIP kernels.  torch supplies device memory and streams.

Loading fails loudly if the library has not been built
(``python -m paper_2608_21229_amd.build``): there is no fallback path.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Iterable, Optional, Sequence, Tuple

RC_MAX_SEGMENTS = 32
SPLITS_BALANCED = -1   # rc_step_masked_attention: one round of 256 work-groups sharing all key tiles evenly
NOALLOC_SCRATCH_BYTES = 128 << 20   # rc_step_masked_attention_noalloc's static scratch per GPU
SPLITS_TAIL = -2       # rc_step_masked_attention: a long and a short key split per query tile (idle CUs take the short)
SPLITS_LAST_ROUND = -3  # rc_step_masked_attention: the tail split for the query tiles of a grid's partial last round
RC_OK, RC_ERR_ARG, RC_ERR_UNSUPPORTED, RC_ERR_MASK_NOT_CACHEABLE, RC_ERR_WORKSPACE, RC_ERR_HIP = 0, -1, -2, -3, -4, -5
SEG_ANCHOR, SEG_TEXT, SEG_TARGET, SEG_REF = 0, 1, 2, 3
MASK_PAPER, MASK_PERREF, MASK_ISOLATED, MASK_DENSE = 0, 1, 2, 3
ENTRY_PREFILL, ENTRY_STEP, ENTRY_FULL = 0, 1, 2
ROWS_STATIC, ROWS_LIVE, ROWS_CACHED, ROWS_ALL = 0, 1, 2, 3
MASKS = {"paper": MASK_PAPER, "perref": MASK_PERREF, "isolated": MASK_ISOLATED, "dense": MASK_DENSE}

# REFCACHE_LIB names another build of the same ABI (the host tests load a
# sanitizer build of the planner through it); by default the in-tree library.
LIB_PATH = os.environ.get("REFCACHE_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                                          "librefcache.so")


class RcError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"librefcache status {status}: {message}")
        self.status = status


class _Segment(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("len", ctypes.c_int32)]


class rc_layout(ctypes.Structure):
    _fields_ = [("n_seg", ctypes.c_int32),
                ("seg", _Segment * RC_MAX_SEGMENTS),
                ("visible", ctypes.c_uint32 * RC_MAX_SEGMENTS)]


_LIB = None
_vp, _i32, _i64, _f32, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
_PL = ctypes.POINTER(rc_layout)
SIGNATURES = {
    "rc_layout_preset": (_i32, [_PL, _i32]),
    "rc_layout_validate": (_i32, [_PL, _i32]),
    "rc_pairs": (_i64, [_PL, _i32]),
    "rc_rows": (_i64, [_PL, _i32]),
    "rc_step_workspace_bytes": (_sz, [_PL, _i32, _i32, _i32, _i32]),
    "rc_step_auto_splits": (_i32, [_PL, _i32, _i32, _i32]),
    "rc_ref_kv_prefill": (_i32, [_PL, _i32, _i32, _i32, _f32, _vp, _vp, _vp, _i64, _vp, _vp, _vp, _vp, _vp]),
    "rc_step_masked_attention": (_i32, [_PL, _i32, _i32, _i32, _f32, _vp, _vp, _vp, _i64, _vp, _vp, _vp, _vp,
                                        _i32, _vp, _sz, _vp]),
    "rc_full_attention": (_i32, [_PL, _i32, _i32, _i32, _f32, _vp, _vp, _vp, _i64, _vp, _vp, _vp]),
    "rc_linear": (_i32, [_i64, _i32, _i32, _vp, _i64, _vp, _vp, _i64, _vp, _i64, _vp]),
    "rc_ref_kv_prefill_fp8": (_i32, [_PL, _i32, _i32, _i32, _f32, _vp, _vp, _vp, _i64, _vp, _vp, _vp, _vp, _vp,
                                     _vp]),
    "rc_step_masked_attention_fp8": (_i32, [_PL, _i32, _i32, _i32, _f32, _vp, _vp, _vp, _i64, _vp, _vp, _vp, _vp,
                                            _vp, _i32, _vp, _sz, _vp]),
    "rc_step_masked_attention_noalloc": (_i32, [_PL, _i32, _i32, _i32, _f32, _vp, _vp, _vp, _i64, _vp, _vp, _vp,
                                                _vp, _i32, _vp]),
    "rc_step_launch_shape": (_i32, [_PL, _i32, _i32, _i32, _i32, _i32, ctypes.POINTER(_i64),
                                    ctypes.POINTER(_i32), ctypes.POINTER(_i32)]),
    "rc_full_attention_ws": (_i32, [_PL, _i32, _i32, _i32, _f32, _vp, _vp, _vp, _i64, _vp, _vp, _vp, _sz, _vp]),
    "rc_full_workspace_bytes": (_sz, [_PL, _i32, _i32, _i32]),
    "rc_prefill_launch_plan": (_i32, [_PL, _i32, _i32, _i32, ctypes.POINTER(_i64), ctypes.POINTER(_i32),
                                      ctypes.POINTER(_i64)]),
    "rc_status_string": (ctypes.c_char_p, [_i32]),
    "rc_last_error": (ctypes.c_char_p, []),
}


def lib():
    """The loaded library; raises if it was not built."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_21229_amd.build` "
                               "(there is no CPU fallback)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = L
    return _LIB


def _check(status: int):
    if status != RC_OK:
        raise RcError(status, lib().rc_last_error().decode())


class Layout:
    """Segment table + block mask (rc_layout).

    segments: (kind, length) pairs in sequence order, kinds SEG_*.
    mask: a preset name ('paper', 'perref', 'isolated', 'dense'), a MASK_*
    id, or an explicit query-first boolean matrix over segments.
    """

    def __init__(self, segments: Sequence[Tuple[int, int]], mask="perref"):
        if not 1 <= len(segments) <= RC_MAX_SEGMENTS:
            raise ValueError(f"need 1..{RC_MAX_SEGMENTS} segments")
        self.c = rc_layout()
        self.c.n_seg = len(segments)
        for i, (k, n) in enumerate(segments):
            self.c.seg[i].kind = int(k)
            self.c.seg[i].len = int(n)
        self.segments = [(int(k), int(n)) for k, n in segments]
        if isinstance(mask, str) or isinstance(mask, int):
            preset = MASKS[mask] if isinstance(mask, str) else mask
            _check(lib().rc_layout_preset(ctypes.byref(self.c), preset))
        else:
            for q, row in enumerate(mask):
                self.c.visible[q] = sum(1 << k for k, v in enumerate(row) if v)

    @property
    def visible(self):
        n = self.c.n_seg
        return [[bool(self.c.visible[q] >> k & 1) for k in range(n)] for q in range(n)]

    def validate(self, entry: int) -> int:
        return lib().rc_layout_validate(ctypes.byref(self.c), entry)

    def pairs(self, entry: int) -> int:
        v = lib().rc_pairs(ctypes.byref(self.c), entry)
        if v < 0:
            _check(int(v))
        return int(v)

    def rows(self, which: int) -> int:
        v = lib().rc_rows(ctypes.byref(self.c), which)
        if v < 0:
            _check(int(v))
        return int(v)

    def workspace_bytes(self, B: int, H: int, D: int, splits: int = 0) -> int:
        return int(lib().rc_step_workspace_bytes(ctypes.byref(self.c), B, H, D, splits))

    def launch_shape(self, B: int, H: int, D: int, splits: int = 0, fp8: bool = False):
        """(work-groups, query rows per work-group, resolved splits) of the
        step's attention kernel."""
        wg, bm, sp = ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int32()
        _check(lib().rc_step_launch_shape(ctypes.byref(self.c), B, H, D, splits, int(fp8), ctypes.byref(wg),
                                          ctypes.byref(bm), ctypes.byref(sp)))
        return wg.value, bm.value, sp.value

    def full_workspace_bytes(self, B: int, H: int, D: int) -> int:
        """Workspace of the full recompute's last-round split (0: no split)."""
        return int(lib().rc_full_workspace_bytes(ctypes.byref(self.c), B, H, D))

    def prefill_plan(self, B: int, H: int, D: int):
        """(attention work-groups, copy work-groups, cache rows they copy) of
        the bf16 prefill; the store kernel copies the remaining rows."""
        a, c, r = ctypes.c_int64(), ctypes.c_int32(), ctypes.c_int64()
        _check(lib().rc_prefill_launch_plan(ctypes.byref(self.c), B, H, D, ctypes.byref(a), ctypes.byref(c),
                                            ctypes.byref(r)))
        return a.value, c.value, r.value

    def auto_splits(self, B: int, H: int, D: int) -> int:
        return int(lib().rc_step_auto_splits(ctypes.byref(self.c), B, H, D))


# ---------------------------------------------------------------- tensor entry points
def _torch():
    import torch
    return torch


def _tok_stride(*ts) -> int:
    strides = set()
    for t in ts:
        B, N, H, D = t.shape
        if t.stride(3) != 1 or t.stride(2) != D or (B > 1 and t.stride(0) != N * t.stride(1)):
            raise ValueError("Q/K/V must be [B, N, H, D] with D contiguous, head stride D and batch stride N*tok_stride")
        strides.add(t.stride(1))
    if len(strides) != 1:
        raise ValueError("Q, K and V must share one token stride")
    return strides.pop()


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _expect(t, shape, dtype_name, what):
    """Outputs and the cache use the library's contiguous layouts."""
    if t is None:
        return
    if tuple(t.shape) != tuple(shape) or not t.is_contiguous() or str(t.dtype) != dtype_name:
        raise ValueError(f"{what} must be a contiguous {dtype_name} tensor of shape {tuple(shape)}, "
                         f"got {str(t.dtype)} {tuple(t.shape)} contiguous={t.is_contiguous()}")


def _stream(stream, dev) -> Optional[int]:
    torch = _torch()
    s = torch.cuda.current_stream(dev) if stream is None else stream
    return s.cuda_stream


def _inputs(q, k, v):
    """Q/K/V: bf16 tensors of one shape on one GPU; returns that device.  The
    library takes raw device pointers, so a host tensor must never reach it."""
    dev = q.device
    if dev.type != "cuda":
        raise ValueError(f"q must be a GPU tensor, got device {dev}")
    for name, t in (("q", q), ("k", k), ("v", v)):
        if t.device != dev or str(t.dtype) != "torch.bfloat16" or tuple(t.shape) != tuple(q.shape):
            raise ValueError(f"{name} must be a bf16 tensor of shape {tuple(q.shape)} on {dev}, "
                             f"got {str(t.dtype)} {tuple(t.shape)} on {t.device}")
    return dev


def _rows_of(layout: "Layout", q, which: int, what: str):
    """The library sizes every read and write from the layout's row count, so
    Q must hold exactly that many tokens (checked before anything else)."""
    n = layout.rows(which)
    if q.dim() != 4 or q.shape[1] != n:
        raise ValueError(f"{what}: q must be [B, {n}, H, D] (the layout's row count), got {tuple(q.shape)}")


def _same_device(dev, **tensors):
    for name, t in tensors.items():
        if t is not None and t.device != dev:
            raise ValueError(f"{name} is on {t.device}, the inputs on {dev}")


def ref_kv_prefill(layout: Layout, q, k, v, o=None, lse=None, k_cache=None, v_cache=None,
                   scale: Optional[float] = None, want_lse: bool = False, stream=None):
    """Static-subgraph prefill.  q/k/v: [B, N_static, H, D] bf16 (ST and R
    tokens in sequence order).  Returns (o, lse or None, k_cache, v_cache)."""
    torch = _torch()
    _rows_of(layout, q, ROWS_STATIC, "ref_kv_prefill")
    dev = _inputs(q, k, v)
    B, N, H, D = q.shape
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    ts = _tok_stride(q, k, v)
    nc = layout.rows(ROWS_CACHED)
    if o is None:
        o = torch.empty((B, N, H, D), dtype=torch.bfloat16, device=q.device)
    if lse is None and want_lse:
        lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    if k_cache is None:
        k_cache = torch.empty((B, H, nc, D), dtype=torch.bfloat16, device=q.device)
    if v_cache is None:
        v_cache = torch.empty((B, H, nc, D), dtype=torch.bfloat16, device=q.device)
    _expect(o, (B, N, H, D), "torch.bfloat16", "o")
    _expect(lse, (B, H, N), "torch.float32", "lse")
    _expect(k_cache, (B, H, nc, D), "torch.bfloat16", "k_cache")
    _expect(v_cache, (B, H, nc, D), "torch.bfloat16", "v_cache")
    _same_device(dev, o=o, lse=lse, k_cache=k_cache, v_cache=v_cache)
    with torch.cuda.device(dev):
        _check(lib().rc_ref_kv_prefill(ctypes.byref(layout.c), B, H, D, scale, q.data_ptr(), k.data_ptr(),
                                       v.data_ptr(), ts, o.data_ptr(), _ptr(lse), k_cache.data_ptr(),
                                       v_cache.data_ptr(), _stream(stream, dev)))
    return o, lse, k_cache, v_cache


def step_masked_attention(layout: Layout, q, k, v, k_cache, v_cache, o=None, lse=None, splits: int = 0,
                          workspace=None, scale: Optional[float] = None, want_lse: bool = False, stream=None):
    """Per-step attention.  q/k/v: [B, N_live, H, D] bf16 (LT and X tokens);
    k_cache/v_cache: [B, H, N_cached, D].  splits: 0 automatic, 1 none, > 1
    even split-KV, SPLITS_TAIL the tail split, SPLITS_LAST_ROUND the tail split
    of the last round's tiles, SPLITS_BALANCED the balanced schedule.  Returns
    (o, lse or None)."""
    torch = _torch()
    _rows_of(layout, q, ROWS_LIVE, "step_masked_attention")
    dev = _inputs(q, k, v)
    B, N, H, D = q.shape
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    ts = _tok_stride(q, k, v)
    if o is None:
        o = torch.empty((B, N, H, D), dtype=torch.bfloat16, device=q.device)
    if lse is None and want_lse:
        lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    nc = layout.rows(ROWS_CACHED)
    _expect(o, (B, N, H, D), "torch.bfloat16", "o")
    _expect(lse, (B, H, N), "torch.float32", "lse")
    _expect(k_cache, (B, H, nc, D), "torch.bfloat16", "k_cache")
    _expect(v_cache, (B, H, nc, D), "torch.bfloat16", "v_cache")
    need = layout.workspace_bytes(B, H, D, splits)
    if need and (workspace is None or workspace.numel() * workspace.element_size() < need):
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    _same_device(dev, o=o, lse=lse, k_cache=k_cache, v_cache=v_cache, workspace=workspace if need else None)
    with torch.cuda.device(dev):
        _check(lib().rc_step_masked_attention(ctypes.byref(layout.c), B, H, D, scale, q.data_ptr(),
                                              k.data_ptr(), v.data_ptr(), ts, _ptr(k_cache), _ptr(v_cache),
                                              o.data_ptr(), _ptr(lse), splits,
                                              _ptr(workspace) if need else None, need, _stream(stream, dev)))
    return o, lse


def step_masked_attention_noalloc(layout: Layout, q, k, v, k_cache, v_cache, o, lse=None, splits: int = 0,
                                  scale: Optional[float] = None, stream=None):
    """step_masked_attention without any device allocation: the caller passes
    the output `o` (and `lse`, or None), and split partials go to the
    library's static scratch array (NOALLOC_SCRATCH_BYTES per GPU; a larger
    split choice raises RcError with RC_ERR_WORKSPACE).  Calls that overlap on
    one GPU share that array and race.  Returns (o, lse)."""
    if o is None:
        raise ValueError("step_masked_attention_noalloc: pass the output o (it allocates nothing)")
    _rows_of(layout, q, ROWS_LIVE, "step_masked_attention_noalloc")
    dev = _inputs(q, k, v)
    B, N, H, D = q.shape
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    ts = _tok_stride(q, k, v)
    nc = layout.rows(ROWS_CACHED)
    _expect(o, (B, N, H, D), "torch.bfloat16", "o")
    _expect(lse, (B, H, N), "torch.float32", "lse")
    _expect(k_cache, (B, H, nc, D), "torch.bfloat16", "k_cache")
    _expect(v_cache, (B, H, nc, D), "torch.bfloat16", "v_cache")
    _same_device(dev, o=o, lse=lse, k_cache=k_cache, v_cache=v_cache)
    with _torch().cuda.device(dev):
        _check(lib().rc_step_masked_attention_noalloc(ctypes.byref(layout.c), B, H, D, scale, q.data_ptr(),
                                                      k.data_ptr(), v.data_ptr(), ts, _ptr(k_cache),
                                                      _ptr(v_cache), o.data_ptr(), _ptr(lse), splits,
                                                      _stream(stream, dev)))
    return o, lse


def full_attention(layout: Layout, q, k, v, o=None, lse=None, scale: Optional[float] = None,
                   want_lse: bool = False, last_round_split: bool = True, stream=None):
    """Full recompute over all rows.  q/k/v: [B, N, H, D] bf16.  Returns (o, lse or None).
    last_round_split: give the library the workspace it asks for to split the
    grid's partial last round (rc_full_attention_ws); False computes every
    query tile whole (rc_full_attention)."""
    torch = _torch()
    _rows_of(layout, q, ROWS_ALL, "full_attention")
    dev = _inputs(q, k, v)
    B, N, H, D = q.shape
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    ts = _tok_stride(q, k, v)
    if o is None:
        o = torch.empty((B, N, H, D), dtype=torch.bfloat16, device=q.device)
    if lse is None and want_lse:
        lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    _expect(o, (B, N, H, D), "torch.bfloat16", "o")
    _expect(lse, (B, H, N), "torch.float32", "lse")
    _same_device(dev, o=o, lse=lse)
    need = layout.full_workspace_bytes(B, H, D) if last_round_split else 0
    with torch.cuda.device(dev):
        ws = torch.empty(need, dtype=torch.uint8, device=q.device) if need else None
        _check(lib().rc_full_attention_ws(ctypes.byref(layout.c), B, H, D, scale, q.data_ptr(), k.data_ptr(),
                                          v.data_ptr(), ts, o.data_ptr(), _ptr(lse), _ptr(ws), need,
                                          _stream(stream, dev)))
    return o, lse


def _rows_view(t, what):
    """A [M, n] bf16 GPU view with unit column stride; returns its row stride."""
    if t.dim() != 2 or str(t.dtype) != "torch.bfloat16" or t.device.type != "cuda":
        raise ValueError(f"{what} must be a 2-D bf16 GPU tensor, got {str(t.dtype)} {tuple(t.shape)} on {t.device}")
    if t.shape[1] > 1 and t.stride(1) != 1:
        raise ValueError(f"{what} must have unit column stride")
    return t.stride(0) if t.shape[0] > 1 else t.shape[1]


def linear(a, w, residual=None, out=None, stream=None):
    """out = a @ w.T (+ residual), bf16 in and out, fp32 accumulation.
    a: [M, K] (any row stride); w: [N, K] contiguous; residual, out: [M, N]
    (any row stride; out may be residual).  Returns out."""
    torch = _torch()
    lda = _rows_view(a, "a")
    dev = a.device
    M, K = a.shape
    if w.dim() != 2 or w.shape[1] != K or not w.is_contiguous() or str(w.dtype) != "torch.bfloat16":
        raise ValueError(f"w must be a contiguous bf16 [N, {K}] tensor, got {str(w.dtype)} {tuple(w.shape)}")
    N = w.shape[0]
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    for name, t in (("out", out), ("residual", residual)):
        if t is not None and tuple(t.shape) != (M, N):
            raise ValueError(f"{name} must have shape {(M, N)}, got {tuple(t.shape)}")
    ldo = _rows_view(out, "out")
    ldr = _rows_view(residual, "residual") if residual is not None else 0
    _same_device(dev, w=w, out=out, residual=residual)
    with torch.cuda.device(dev):
        _check(lib().rc_linear(M, N, K, a.data_ptr(), lda, w.data_ptr(), _ptr(residual), ldr, out.data_ptr(), ldo,
                               _stream(stream, dev)))
    return out


# ---------------------------------------------------------------- FP8 reference cache
def fp8_cache_shapes(layout: Layout, B: int, H: int, D: int):
    """Shapes of the FP8 cache: K8 and V8 [B, H, N_cached, D] (uint8 e4m3fn
    codes, the rows of the bf16 cache) and the scales [B, H, 2] (fp32)."""
    n = layout.rows(ROWS_CACHED)
    return (B, H, n, D), (B, H, n, D), (B, H, 2)


def ref_kv_prefill_fp8(layout: Layout, q, k, v, o=None, lse=None, k_cache8=None, v_cache8=None, kv_scale=None,
                       scale: Optional[float] = None, want_lse: bool = False, stream=None):
    """Static-subgraph prefill writing the FP8 cache.  Returns
    (o, lse or None, k_cache8, v_cache8, kv_scale)."""
    torch = _torch()
    _rows_of(layout, q, ROWS_STATIC, "ref_kv_prefill_fp8")
    dev = _inputs(q, k, v)
    B, N, H, D = q.shape
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    ts = _tok_stride(q, k, v)
    ks, vs, ss = fp8_cache_shapes(layout, B, H, D)
    if o is None:
        o = torch.empty((B, N, H, D), dtype=torch.bfloat16, device=dev)
    if lse is None and want_lse:
        lse = torch.empty((B, H, N), dtype=torch.float32, device=dev)
    if k_cache8 is None:
        k_cache8 = torch.empty(ks, dtype=torch.uint8, device=dev)
    if v_cache8 is None:
        v_cache8 = torch.empty(vs, dtype=torch.uint8, device=dev)
    if kv_scale is None:
        kv_scale = torch.empty(ss, dtype=torch.float32, device=dev)
    _expect(o, (B, N, H, D), "torch.bfloat16", "o")
    _expect(lse, (B, H, N), "torch.float32", "lse")
    _expect(k_cache8, ks, "torch.uint8", "k_cache8")
    _expect(v_cache8, vs, "torch.uint8", "v_cache8")
    _expect(kv_scale, ss, "torch.float32", "kv_scale")
    _same_device(dev, o=o, lse=lse, k_cache8=k_cache8, v_cache8=v_cache8, kv_scale=kv_scale)
    with torch.cuda.device(dev):
        _check(lib().rc_ref_kv_prefill_fp8(ctypes.byref(layout.c), B, H, D, scale, q.data_ptr(), k.data_ptr(),
                                           v.data_ptr(), ts, o.data_ptr(), _ptr(lse), k_cache8.data_ptr(),
                                           v_cache8.data_ptr(), kv_scale.data_ptr(), _stream(stream, dev)))
    return o, lse, k_cache8, v_cache8, kv_scale


def step_masked_attention_fp8(layout: Layout, q, k, v, k_cache8, v_cache8, kv_scale, o=None, lse=None,
                              splits: int = 0, workspace=None, scale: Optional[float] = None, want_lse: bool = False,
                              stream=None):
    """Per-step attention reading the FP8 cache (fresh LT/X K/V stay bf16).
    Returns (o, lse or None)."""
    torch = _torch()
    _rows_of(layout, q, ROWS_LIVE, "step_masked_attention_fp8")
    dev = _inputs(q, k, v)
    B, N, H, D = q.shape
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    ts = _tok_stride(q, k, v)
    ks, vs, ss = fp8_cache_shapes(layout, B, H, D)
    if o is None:
        o = torch.empty((B, N, H, D), dtype=torch.bfloat16, device=dev)
    if lse is None and want_lse:
        lse = torch.empty((B, H, N), dtype=torch.float32, device=dev)
    _expect(o, (B, N, H, D), "torch.bfloat16", "o")
    _expect(lse, (B, H, N), "torch.float32", "lse")
    _expect(k_cache8, ks, "torch.uint8", "k_cache8")
    _expect(v_cache8, vs, "torch.uint8", "v_cache8")
    _expect(kv_scale, ss, "torch.float32", "kv_scale")
    need = layout.workspace_bytes(B, H, D, splits) if splits != SPLITS_BALANCED else 0
    if need and (workspace is None or workspace.numel() * workspace.element_size() < need):
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    _same_device(dev, o=o, lse=lse, k_cache8=k_cache8, v_cache8=v_cache8, kv_scale=kv_scale,
                 workspace=workspace if need else None)
    with torch.cuda.device(dev):
        _check(lib().rc_step_masked_attention_fp8(ctypes.byref(layout.c), B, H, D, scale, q.data_ptr(), k.data_ptr(),
                                                  v.data_ptr(), ts, k_cache8.data_ptr(), v_cache8.data_ptr(),
                                                  kv_scale.data_ptr(), o.data_ptr(), _ptr(lse), splits,
                                                  _ptr(workspace) if need else None, need, _stream(stream, dev)))
    return o, lse
