"""bd_attn: block-diffusion masked attention for MI355X (gfx950).

Thin Python binding over the C-ABI library libbd_attn.so: the functions here
carry the names of the C entry points and only marshal arguments (shape and
dtype checks, output/workspace allocation through torch, the current HIP
stream).  Every step of the computation runs in the library's HIP kernels.

Attention over the packed sequence [x_t | x_0] of 2L tokens with the
block-diffusion mask of DiRL (arXiv 2512.22234, Section 4.1; Eq. 1 and
Eq. 2): a noisy query sees noisy keys of its own block and clean keys of
earlier blocks; a clean query sees clean keys of its own and earlier blocks.
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch

from ._lib import LIB_PATH, BdAttnError, lib, status_string  # noqa: F401

BD_ATTN_BF16 = 0
BD_ATTN_FP32 = 1

__all__ = [
    "bd_attn", "BdAttnFunction", "bd_attn_fwd", "bd_attn_bwd", "bd_attn_workspace_bytes",
    "bd_attn_classify_tiles_host", "bd_attn_visit_lists_host", "bd_attn_mask_windows_host",
    "bd_attn_status_string", "bd_attn_bwd_noalloc", "BD_ATTN_NOALLOC_SCRATCH_BYTES",
    "bd_attn_version", "bd_attn_fwd_marked", "bd_attn_bwd_marked", "bd_attn_stage_names",
    "BdAttnError", "BD_ATTN_BF16", "BD_ATTN_FP32",
    "bd_attn_varlen", "BdAttnVarlenFunction", "bd_attn_varlen_fwd", "bd_attn_varlen_bwd",
    "bd_attn_varlen_workspace_bytes", "bd_attn_decode_fwd", "bd_attn_decode_workspace_bytes",
    "bd_lce_fwd", "bd_lce_bwd", "bd_lce_workspace_bytes", "bd_lce_logits_bytes", "bd_lce_objective", "LceFunction", "lm_head_logprobs",
    "BD_LCE_CE", "BD_LCE_DIPO",
]


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BD_ATTN_BF16
    if t.dtype == torch.float32:
        return BD_ATTN_FP32
    raise TypeError(f"bd_attn supports bfloat16 and float32 tensors, got {t.dtype}")


def _ptr(t) -> ctypes.c_void_p:
    return ctypes.c_void_p(t.data_ptr())


def _stream(device: torch.device, stream):
    s = torch.cuda.current_stream(device) if stream is None else stream
    return s, ctypes.c_void_p(s.cuda_stream)


def _check(name: str, t: torch.Tensor, shape, dtype, device):
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if t.device != device:
        raise ValueError(f"{name}: expected device {device}, got {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")


def _scale_arg(scale) -> float:
    return 0.0 if scale is None else float(scale)


def bd_attn_version() -> int:
    return int(lib().bd_attn_version())


def bd_attn_status_string(status: int) -> str:
    return status_string(status)


def bd_attn_workspace_bytes(B, L, S, Hq, Hkv, D, dtype, for_bwd) -> int:
    return int(lib().bd_attn_workspace_bytes(B, L, S, Hq, Hkv, D, int(dtype), int(for_bwd)))


def bd_attn_classify_tiles_host(L: int, S: int, BM: int, BN: int) -> np.ndarray:
    nq, nk = 2 * (-(-L // BM)), 2 * (-(-L // BN))
    out = np.zeros((nq, nk), dtype=np.int8)
    st = lib().bd_attn_classify_tiles_host(L, S, BM, BN, out.ctypes.data_as(ctypes.c_void_p))
    if st:
        raise BdAttnError(st, "bd_attn_classify_tiles_host")
    return out


def bd_attn_visit_lists_host(L: int, S: int, BM: int, BN: int, by_key_tile: bool, nsplit: int = 2) -> np.ndarray:
    nq, nk = 2 * (-(-L // BM)), 2 * (-(-L // BN))
    out = np.zeros((nq, nk), dtype=np.int8)
    st = lib().bd_attn_visit_lists_host(L, S, BM, BN, int(by_key_tile), nsplit, out.ctypes.data_as(ctypes.c_void_p))
    if st:
        raise BdAttnError(st, "bd_attn_visit_lists_host")
    return out


def bd_attn_mask_windows_host(L: int, S: int, by_key: bool) -> np.ndarray:
    out = np.zeros((2 * L, 2 * L), dtype=np.int8)
    st = lib().bd_attn_mask_windows_host(L, S, int(by_key), out.ctypes.data_as(ctypes.c_void_p))
    if st:
        raise BdAttnError(st, "bd_attn_mask_windows_host")
    return out


def bd_attn_group_windows_host(L: int, S: int, by_key: bool, group: int) -> np.ndarray:
    out = np.zeros((2 * L, 2 * L), dtype=np.int8)
    st = lib().bd_attn_group_windows_host(L, S, int(by_key), group, out.ctypes.data_as(ctypes.c_void_p))
    if st:
        raise BdAttnError(st, "bd_attn_group_windows_host")
    return out


def _shapes(q, k, L):
    if q.dim() != 4 or k.dim() != 4:
        raise ValueError("q [B,Hq,2L,D] and k/v [B,Hkv,2L,D] expected")
    B, Hq, N, D = q.shape
    Hkv = k.shape[1]
    if N != 2 * L:
        raise ValueError(f"packed length {N} != 2L = {2 * L}")
    return B, Hq, Hkv, D


def _marks_arg(marks):
    """ctypes array of raw HIP event handles from torch.cuda.Event objects."""
    if not marks:
        return None, 0
    for ev in marks:
        if ev.cuda_event == 0:      # torch creates the event lazily on first record
            ev.record()
    arr = (ctypes.c_void_p * len(marks))(*[ev.cuda_event for ev in marks])
    return arr, len(marks)


def bd_attn_stage_names(for_bwd: bool, dtype: int = BD_ATTN_BF16):
    return lib().bd_attn_stage_names(int(for_bwd), int(dtype)).decode().split(",")


def bd_attn_fwd_marked(q, k, v, L: int, S: int, marks, scale=None, out=None, lse=None, workspace=None,
                       stream=None):
    """bd_attn_fwd that also records marks[2i] and marks[2i + 1] as kernel i begins and ends."""
    return bd_attn_fwd(q, k, v, L, S, scale, out, lse, workspace, stream, _marks=marks)


def bd_attn_bwd_marked(do, q, k, v, o, lse, L: int, S: int, marks, scale=None, dq=None, dk=None, dv=None,
                       workspace=None, stream=None):
    """bd_attn_bwd that also records marks[2i] and marks[2i + 1] as kernel i begins and ends."""
    return bd_attn_bwd(do, q, k, v, o, lse, L, S, scale, dq, dk, dv, workspace, stream, _marks=marks)


def bd_attn_fwd(q, k, v, L: int, S: int, scale=None, out=None, lse=None, workspace=None, stream=None,
                _marks=None):
    """Forward pass; returns (O, LSE).  O has q's dtype, LSE is float32 [B,Hq,2L]."""
    B, Hq, Hkv, D = _shapes(q, k, L)
    dev, dt = q.device, q.dtype
    code = _dtype_code(q)
    _check("q", q, (B, Hq, 2 * L, D), dt, dev)
    _check("k", k, (B, Hkv, 2 * L, D), dt, dev)
    _check("v", v, (B, Hkv, 2 * L, D), dt, dev)
    o = torch.empty_like(q) if out is None else out
    l_ = torch.empty((B, Hq, 2 * L), dtype=torch.float32, device=dev) if lse is None else lse
    _check("out", o, q.shape, dt, dev)
    _check("lse", l_, (B, Hq, 2 * L), torch.float32, dev)
    nbytes = bd_attn_workspace_bytes(B, L, S, Hq, Hkv, D, code, 0)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=dev) if workspace is None else workspace
    s, sh = _stream(dev, stream)
    args = (_ptr(q), _ptr(k), _ptr(v), B, L, S, Hq, Hkv, D, _scale_arg(scale), code,
            _ptr(o), _ptr(l_), _ptr(ws), ws.numel(), sh)
    if _marks:
        st = lib().bd_attn_fwd_marked(*args, *_marks_arg(_marks))
    else:
        st = lib().bd_attn_fwd(*args)
    if st:
        raise BdAttnError(st, "bd_attn_fwd")
    if stream is not None and workspace is None:
        ws.record_stream(s)
    return o, l_


def bd_attn_bwd(do, q, k, v, o, lse, L: int, S: int, scale=None, dq=None, dk=None, dv=None,
                workspace=None, stream=None, _marks=None):
    """Backward pass; returns (dQ, dK, dV) in q's dtype."""
    B, Hq, Hkv, D = _shapes(q, k, L)
    dev, dt = q.device, q.dtype
    code = _dtype_code(q)
    for name, t, shp in (("do", do, q.shape), ("q", q, q.shape), ("k", k, (B, Hkv, 2 * L, D)),
                         ("v", v, (B, Hkv, 2 * L, D)), ("o", o, q.shape)):
        _check(name, t, shp, dt, dev)
    _check("lse", lse, (B, Hq, 2 * L), torch.float32, dev)
    dq_ = torch.empty_like(q) if dq is None else dq
    dk_ = torch.empty_like(k) if dk is None else dk
    dv_ = torch.empty_like(v) if dv is None else dv
    nbytes = bd_attn_workspace_bytes(B, L, S, Hq, Hkv, D, code, 1)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=dev) if workspace is None else workspace
    s, sh = _stream(dev, stream)
    args = (_ptr(do), _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, L, S, Hq, Hkv, D,
            _scale_arg(scale), code, _ptr(dq_), _ptr(dk_), _ptr(dv_), _ptr(ws), ws.numel(), sh)
    if _marks:
        st = lib().bd_attn_bwd_marked(*args, *_marks_arg(_marks))
    else:
        st = lib().bd_attn_bwd(*args)
    if st:
        raise BdAttnError(st, "bd_attn_bwd")
    if stream is not None and workspace is None:
        ws.record_stream(s)
    return dq_, dk_, dv_


BD_ATTN_NOALLOC_SCRATCH_BYTES = 96 << 20   # the library's scratch array for bd_attn_bwd_noalloc


def bd_attn_bwd_noalloc(do, q, k, v, o, lse, L: int, S: int, dq, dk, dv, scale=None, stream=None):
    """bd_attn_bwd with the library's own scratch array as its workspace (for
    callers that cannot allocate): writes the caller's dq, dk, dv and returns
    them.  Calls whose work overlaps in time on one GPU race on that array."""
    B, Hq, Hkv, D = _shapes(q, k, L)
    dev, dt = q.device, q.dtype
    code = _dtype_code(q)
    for name, t, shp in (("do", do, q.shape), ("q", q, q.shape), ("k", k, (B, Hkv, 2 * L, D)),
                         ("v", v, (B, Hkv, 2 * L, D)), ("o", o, q.shape), ("dq", dq, q.shape),
                         ("dk", dk, (B, Hkv, 2 * L, D)), ("dv", dv, (B, Hkv, 2 * L, D))):
        _check(name, t, shp, dt, dev)
    _check("lse", lse, (B, Hq, 2 * L), torch.float32, dev)
    _, sh = _stream(dev, stream)
    st = lib().bd_attn_bwd_noalloc(_ptr(do), _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), B, L, S, Hq, Hkv, D,
                                   _scale_arg(scale), code, _ptr(dq), _ptr(dk), _ptr(dv), sh)
    if st:
        raise BdAttnError(st, "bd_attn_bwd_noalloc")
    return dq, dk, dv


class BdAttnFunction(torch.autograd.Function):
    """Autograd wrapper: forward saves Q, K, V, O, LSE; backward returns dQ, dK, dV."""

    @staticmethod
    def forward(ctx, q, k, v, L, S, scale=None):
        o, lse = bd_attn_fwd(q, k, v, L, S, scale)
        ctx.save_for_backward(q, k, v, o, lse)
        ctx.L, ctx.S, ctx.scale = L, S, scale
        return o

    @staticmethod
    def backward(ctx, do):
        q, k, v, o, lse = ctx.saved_tensors
        dq, dk, dv = bd_attn_bwd(do.contiguous(), q, k, v, o, lse, ctx.L, ctx.S, ctx.scale)
        return dq, dk, dv, None, None, None


def bd_attn(q, k, v, L: int, S: int, scale=None):
    """Block-diffusion masked attention over [x_t | x_0]; differentiable."""
    return BdAttnFunction.apply(q, k, v, L, S, scale)


# ---------------------------------------------------------------------------
# Packed sequences: q [Hq, 2T, D], k/v [Hkv, 2T, D], cu_seqlens int32 [n+1] on
# the same device (cu_seqlens[0] = 0, cu_seqlens[n] = T); sequence i occupies
# rows [2 cu[i], 2 cu[i+1]) of every head, noisy copy first.

def bd_attn_varlen_workspace_bytes(n_seqs, total_L, max_L, S, Hq, Hkv, D, dtype, for_bwd) -> int:
    return int(lib().bd_attn_varlen_workspace_bytes(n_seqs, total_L, max_L, S, Hq, Hkv, D, int(dtype),
                                                      int(for_bwd)))


def _varlen_shapes(q, k, cu_seqlens):
    if q.dim() != 3 or k.dim() != 3:
        raise ValueError("q [Hq,2T,D] and k/v [Hkv,2T,D] expected")
    Hq, N, D = q.shape
    Hkv = k.shape[0]
    if N % 2:
        raise ValueError(f"packed length {N} is odd")
    if cu_seqlens.dtype != torch.int32 or cu_seqlens.dim() != 1 or cu_seqlens.numel() < 2:
        raise ValueError("cu_seqlens must be a 1-D int32 tensor of n_seqs + 1 entries")
    if cu_seqlens.device != q.device or not cu_seqlens.is_contiguous():
        raise ValueError("cu_seqlens must be contiguous and on q's device")
    return Hq, Hkv, D, N // 2, cu_seqlens.numel() - 1


def bd_attn_varlen_fwd(q, k, v, cu_seqlens, max_L: int, S: int, scale=None, out=None, lse=None,
                       workspace=None, stream=None):
    """Forward pass over packed sequences; returns (O, LSE [Hq, 2T] float32)."""
    Hq, Hkv, D, T, n = _varlen_shapes(q, k, cu_seqlens)
    dev, dt = q.device, q.dtype
    code = _dtype_code(q)
    _check("k", k, (Hkv, 2 * T, D), dt, dev)
    _check("v", v, (Hkv, 2 * T, D), dt, dev)
    o = torch.empty_like(q) if out is None else out
    l_ = torch.empty((Hq, 2 * T), dtype=torch.float32, device=dev) if lse is None else lse
    _check("out", o, q.shape, dt, dev)
    _check("lse", l_, (Hq, 2 * T), torch.float32, dev)
    nbytes = bd_attn_varlen_workspace_bytes(n, T, max_L, S, Hq, Hkv, D, code, 0)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=dev) if workspace is None else workspace
    s, sh = _stream(dev, stream)
    st = lib().bd_attn_varlen_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(cu_seqlens), n, T, max_L, S, Hq, Hkv, D,
                                  _scale_arg(scale), code, _ptr(o), _ptr(l_), _ptr(ws), ws.numel(), sh)
    if st:
        raise BdAttnError(st, "bd_attn_varlen_fwd")
    if stream is not None and workspace is None:
        ws.record_stream(s)
    return o, l_


def bd_attn_varlen_bwd(do, q, k, v, o, lse, cu_seqlens, max_L: int, S: int, scale=None, dq=None, dk=None,
                       dv=None, workspace=None, stream=None):
    """Backward pass over packed sequences; returns (dQ, dK, dV) in q's dtype."""
    Hq, Hkv, D, T, n = _varlen_shapes(q, k, cu_seqlens)
    dev, dt = q.device, q.dtype
    code = _dtype_code(q)
    for name, t, shp in (("do", do, q.shape), ("k", k, (Hkv, 2 * T, D)), ("v", v, (Hkv, 2 * T, D)),
                         ("o", o, q.shape)):
        _check(name, t, shp, dt, dev)
    _check("lse", lse, (Hq, 2 * T), torch.float32, dev)
    dq_ = torch.empty_like(q) if dq is None else dq
    dk_ = torch.empty_like(k) if dk is None else dk
    dv_ = torch.empty_like(v) if dv is None else dv
    nbytes = bd_attn_varlen_workspace_bytes(n, T, max_L, S, Hq, Hkv, D, code, 1)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=dev) if workspace is None else workspace
    s, sh = _stream(dev, stream)
    st = lib().bd_attn_varlen_bwd(_ptr(do), _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), _ptr(cu_seqlens), n,
                                  T, max_L, S, Hq, Hkv, D, _scale_arg(scale), code, _ptr(dq_), _ptr(dk_),
                                  _ptr(dv_), _ptr(ws), ws.numel(), sh)
    if st:
        raise BdAttnError(st, "bd_attn_varlen_bwd")
    if stream is not None and workspace is None:
        ws.record_stream(s)
    return dq_, dk_, dv_


class BdAttnVarlenFunction(torch.autograd.Function):
    """Autograd wrapper of the packed-sequence calls."""

    @staticmethod
    def forward(ctx, q, k, v, cu_seqlens, max_L, S, scale=None):
        o, lse = bd_attn_varlen_fwd(q, k, v, cu_seqlens, max_L, S, scale)
        ctx.save_for_backward(q, k, v, o, lse, cu_seqlens)
        ctx.max_L, ctx.S, ctx.scale = max_L, S, scale
        return o

    @staticmethod
    def backward(ctx, do):
        q, k, v, o, lse, cu = ctx.saved_tensors
        dq, dk, dv = bd_attn_varlen_bwd(do.contiguous(), q, k, v, o, lse, cu, ctx.max_L, ctx.S, ctx.scale)
        return dq, dk, dv, None, None, None, None


def bd_attn_varlen(q, k, v, cu_seqlens, max_L: int, S: int, scale=None):
    """Block-diffusion masked attention over packed [x_t | x_0] sequences; differentiable."""
    return BdAttnVarlenFunction.apply(q, k, v, cu_seqlens, max_L, S, scale)


def bd_attn_decode_workspace_bytes(B, S, Hq, Hkv, D, capacity, dtype=BD_ATTN_BF16) -> int:
    return int(lib().bd_attn_decode_workspace_bytes(B, S, Hq, Hkv, D, capacity, int(dtype)))


def bd_attn_decode_fwd(q, k_cache, v_cache, k_new, v_new, cache_lens, scale=None, out=None, lse=None,
                       workspace=None, stream=None):
    """One block's decoding step over a KV cache; returns (O [B,Hq,S,D], LSE [B,Hq,S] float32).

    q [B,Hq,S,D]; k_cache/v_cache [B,Hkv,C,D]; k_new/v_new [B,Hkv,S,D], all
    bfloat16; cache_lens: int32 [B] on the device (clamped to [0, C])."""
    if q.dim() != 4 or k_cache.dim() != 4:
        raise ValueError("q [B,Hq,S,D] and k_cache/v_cache [B,Hkv,C,D] expected")
    B, Hq, S, D = q.shape
    Hkv, C = k_cache.shape[1], k_cache.shape[2]
    dev = q.device
    if q.dtype != torch.bfloat16:
        raise TypeError(f"bd_attn_decode_fwd supports bfloat16 tensors, got {q.dtype}")
    for name, t, shp in (("k_cache", k_cache, (B, Hkv, C, D)), ("v_cache", v_cache, (B, Hkv, C, D)),
                         ("k_new", k_new, (B, Hkv, S, D)), ("v_new", v_new, (B, Hkv, S, D))):
        _check(name, t, shp, torch.bfloat16, dev)
    _check("cache_lens", cache_lens, (B,), torch.int32, dev)
    o = torch.empty_like(q) if out is None else out
    l_ = torch.empty((B, Hq, S), dtype=torch.float32, device=dev) if lse is None else lse
    _check("out", o, q.shape, torch.bfloat16, dev)
    _check("lse", l_, (B, Hq, S), torch.float32, dev)
    nbytes = bd_attn_decode_workspace_bytes(B, S, Hq, Hkv, D, C, BD_ATTN_BF16)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=dev) if workspace is None else workspace
    s, sh = _stream(dev, stream)
    st = lib().bd_attn_decode_fwd(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(k_new), _ptr(v_new),
                                  _ptr(cache_lens), B, S, Hq, Hkv, D, C, _scale_arg(scale), BD_ATTN_BF16,
                                  _ptr(o), _ptr(l_), _ptr(ws), ws.numel(), sh)
    if st:
        raise BdAttnError(st, "bd_attn_decode_fwd")
    if stream is not None and workspace is None:
        ws.record_stream(s)
    return o, l_


# ---------------------------------------------------------------------------
# Token log-probabilities through the LM head (Eq. 3 and Eq. 6-7 objectives).

BD_LCE_CE = 0
BD_LCE_DIPO = 1


def bd_lce_workspace_bytes(N, V, Dm, for_bwd, dtype=BD_ATTN_BF16) -> int:
    return int(lib().bd_lce_workspace_bytes(N, V, Dm, int(dtype), int(for_bwd)))


def _lce_shapes(h, w, targets):
    if h.dim() != 2 or w.dim() != 2 or h.shape[1] != w.shape[1]:
        raise ValueError("h [N, Dm] and w [V, Dm] expected")
    N, Dm = h.shape
    V = w.shape[0]
    dev = h.device
    _check("h", h, (N, Dm), torch.bfloat16, dev)
    _check("w", w, (V, Dm), torch.bfloat16, dev)
    _check("targets", targets, (N,), torch.int32, dev)
    return N, V, Dm, dev


def bd_lce_logits_bytes(N, V, Dm, dtype=BD_ATTN_BF16) -> int:
    return int(lib().bd_lce_logits_bytes(N, V, Dm, int(dtype)))


def bd_lce_fwd(h, w, targets, lse=None, logp=None, workspace=None, stream=None, logits=None):
    """Per-position LSE and log p(target) (float32 [N]) of logits h w^T.
    logits: optional float32 tensor of bd_lce_logits_bytes bytes that receives
    the logits for bd_lce_bwd."""
    N, V, Dm, dev = _lce_shapes(h, w, targets)
    if logits is not None and (logits.dtype != torch.float32 or logits.numel() * 4 < bd_lce_logits_bytes(N, V, Dm)
                               or not logits.is_contiguous() or logits.device != dev):
        raise ValueError("logits: a contiguous float32 buffer of bd_lce_logits_bytes bytes on the device expected")
    l_ = torch.empty(N, dtype=torch.float32, device=dev) if lse is None else lse
    lp = torch.empty(N, dtype=torch.float32, device=dev) if logp is None else logp
    _check("lse", l_, (N,), torch.float32, dev)
    _check("logp", lp, (N,), torch.float32, dev)
    nbytes = bd_lce_workspace_bytes(N, V, Dm, 0)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=dev) if workspace is None else workspace
    s, sh = _stream(dev, stream)
    kl = ctypes.c_void_p(None) if logits is None else _ptr(logits)
    st = lib().bd_lce_fwd(_ptr(h), _ptr(w), _ptr(targets), N, V, Dm, BD_ATTN_BF16, _ptr(l_), _ptr(lp), kl, _ptr(ws),
                          ws.numel(), sh)
    if st:
        raise BdAttnError(st, "bd_lce_fwd")
    if stream is not None and workspace is None:
        ws.record_stream(s)
    return l_, lp


def bd_lce_bwd(h, w, targets, lse, dlogp, dh=None, dw=None, workspace=None, stream=None, logits=None):
    """dH [N, Dm] and dW [V, Dm] (bf16) for dLoss/dlogp = dlogp (logits: the
    buffer bd_lce_fwd filled, to skip recomputing them)."""
    N, V, Dm, dev = _lce_shapes(h, w, targets)
    if logits is not None and (logits.dtype != torch.float32 or logits.numel() * 4 < bd_lce_logits_bytes(N, V, Dm)
                               or not logits.is_contiguous() or logits.device != dev):
        raise ValueError("logits: a contiguous float32 buffer of bd_lce_logits_bytes bytes on the device expected")
    _check("lse", lse, (N,), torch.float32, dev)
    _check("dlogp", dlogp, (N,), torch.float32, dev)
    dh_ = torch.empty_like(h) if dh is None else dh
    dw_ = torch.empty_like(w) if dw is None else dw
    _check("dh", dh_, (N, Dm), torch.bfloat16, dev)
    _check("dw", dw_, (V, Dm), torch.bfloat16, dev)
    nbytes = bd_lce_workspace_bytes(N, V, Dm, 1)
    ws = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=dev) if workspace is None else workspace
    s, sh = _stream(dev, stream)
    kl = ctypes.c_void_p(None) if logits is None else _ptr(logits)
    st = lib().bd_lce_bwd(_ptr(h), _ptr(w), _ptr(targets), _ptr(lse), _ptr(dlogp), kl, N, V, Dm, BD_ATTN_BF16,
                          _ptr(dh_), _ptr(dw_), _ptr(ws), ws.numel(), sh)
    if st:
        raise BdAttnError(st, "bd_lce_bwd")
    if stream is not None and workspace is None:
        ws.record_stream(s)
    return dh_, dw_


def bd_lce_objective(logp, weight, kind=BD_LCE_CE, logp_old=None, logp_ref=None, adv=None, eps=0.2, beta=0.0,
                     loss=None, dlogp=None, stream=None):
    """Per-position loss and dloss/dlogp (float32 [N]) of the masked CE (kind
    BD_LCE_CE) or the DiPO clipped surrogate with KL (kind BD_LCE_DIPO)."""
    N = logp.numel()
    dev = logp.device
    for name, t in (("logp", logp), ("weight", weight), ("logp_old", logp_old), ("logp_ref", logp_ref),
                    ("adv", adv)):
        if t is not None:
            _check(name, t, (N,), torch.float32, dev)
    lo = torch.empty(N, dtype=torch.float32, device=dev) if loss is None else loss
    dl = torch.empty(N, dtype=torch.float32, device=dev) if dlogp is None else dlogp
    opt = lambda t: ctypes.c_void_p(None) if t is None else _ptr(t)  # noqa: E731
    _, sh = _stream(dev, stream)
    st = lib().bd_lce_objective(_ptr(logp), opt(logp_old), opt(logp_ref), opt(adv), _ptr(weight), N, int(kind),
                                float(eps), float(beta), _ptr(lo), _ptr(dl), sh)
    if st:
        raise BdAttnError(st, "bd_lce_objective")
    return lo, dl


class LceFunction(torch.autograd.Function):
    """log p(target) through the LM head; differentiable in h and w."""

    @staticmethod
    def forward(ctx, h, w, targets, keep_logits=False):
        N, V, Dm, dev = _lce_shapes(h, w, targets)
        logits = (torch.empty(bd_lce_logits_bytes(N, V, Dm) // 4, dtype=torch.float32, device=dev)
                  if keep_logits else None)
        lse, logp = bd_lce_fwd(h, w, targets, logits=logits)
        ctx.save_for_backward(h, w, targets, lse)
        ctx.logits = logits
        return logp

    @staticmethod
    def backward(ctx, dlogp):
        h, w, targets, lse = ctx.saved_tensors
        dh, dw = bd_lce_bwd(h, w, targets, lse, dlogp.contiguous().float(), logits=ctx.logits)
        ctx.logits = None
        return dh, dw, None, None


def lm_head_logprobs(h, w, targets, keep_logits=False):
    """Differentiable per-position log p(target) [N] float32 (targets outside
    [0, V): 0).  keep_logits trades N x V float32 of memory for the
    backward's recomputation of the logits."""
    return LceFunction.apply(h, w, targets, keep_logits)
