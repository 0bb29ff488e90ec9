"""ctypes loader for libbd_attn.so (the HIP library built in-tree).

torch is imported first so that the library binds to the HIP runtime torch
already loaded (same soname), giving one runtime per process.  A missing
library is an error: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import torch  # noqa: F401  (loads the HIP runtime the library binds to)

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libbd_attn.so")

_lib = None


class BdAttnError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} (status {status})")


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing; build it with `python -m paper_2512_22234_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, ci, cf, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    L.bd_attn_fwd.restype = ci
    L.bd_attn_fwd.argtypes = [vp, vp, vp, ci, ci, ci, ci, ci, ci, cf, ci, vp, vp, vp, sz, vp]
    L.bd_attn_bwd.restype = ci
    L.bd_attn_bwd.argtypes = [vp, vp, vp, vp, vp, vp, ci, ci, ci, ci, ci, ci, cf, ci,
                              vp, vp, vp, vp, sz, vp]
    L.bd_attn_bwd_noalloc.restype = ci
    L.bd_attn_bwd_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, ci, ci, ci, ci, ci, ci, cf, ci, vp, vp, vp, vp]
    L.bd_attn_fwd_marked.restype = ci
    L.bd_attn_fwd_marked.argtypes = L.bd_attn_fwd.argtypes + [vp, ci]
    L.bd_attn_bwd_marked.restype = ci
    L.bd_attn_bwd_marked.argtypes = L.bd_attn_bwd.argtypes + [vp, ci]
    L.bd_attn_varlen_fwd.restype = ci
    L.bd_attn_varlen_fwd.argtypes = [vp, vp, vp, vp, ci, ci, ci, ci, ci, ci, ci, cf, ci, vp, vp, vp, sz, vp]
    L.bd_attn_varlen_bwd.restype = ci
    L.bd_attn_varlen_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, ci, ci, ci, ci, ci, ci, ci, cf, ci,
                                     vp, vp, vp, vp, sz, vp]
    L.bd_attn_varlen_workspace_bytes.restype = sz
    L.bd_attn_varlen_workspace_bytes.argtypes = [ci, ci, ci, ci, ci, ci, ci, ci, ci]
    L.bd_attn_decode_fwd.restype = ci
    L.bd_attn_decode_fwd.argtypes = [vp, vp, vp, vp, vp, vp, ci, ci, ci, ci, ci, ci, cf, ci, vp, vp, vp, sz, vp]
    L.bd_attn_decode_workspace_bytes.restype = sz
    L.bd_attn_decode_workspace_bytes.argtypes = [ci, ci, ci, ci, ci, ci, ci]
    L.bd_lce_fwd.restype = ci
    L.bd_lce_fwd.argtypes = [vp, vp, vp, ci, ci, ci, ci, vp, vp, vp, vp, sz, vp]
    L.bd_lce_bwd.restype = ci
    L.bd_lce_bwd.argtypes = [vp, vp, vp, vp, vp, vp, ci, ci, ci, ci, vp, vp, vp, sz, vp]
    L.bd_lce_logits_bytes.restype = sz
    L.bd_lce_logits_bytes.argtypes = [ci, ci, ci, ci]
    L.bd_lce_workspace_bytes.restype = sz
    L.bd_lce_workspace_bytes.argtypes = [ci, ci, ci, ci, ci]
    L.bd_lce_objective.restype = ci
    L.bd_lce_objective.argtypes = [vp, vp, vp, vp, vp, ci, ci, cf, cf, vp, vp, vp]
    L.bd_attn_stage_names.restype = ctypes.c_char_p
    L.bd_attn_stage_names.argtypes = [ci, ci]
    L.bd_attn_workspace_bytes.restype = sz
    L.bd_attn_workspace_bytes.argtypes = [ci, ci, ci, ci, ci, ci, ci, ci]
    L.bd_attn_classify_tiles_host.restype = ci
    L.bd_attn_classify_tiles_host.argtypes = [ci, ci, ci, ci, vp]
    L.bd_attn_visit_lists_host.restype = ci
    L.bd_attn_visit_lists_host.argtypes = [ci, ci, ci, ci, ci, ci, vp]
    L.bd_attn_mask_windows_host.restype = ci
    L.bd_attn_mask_windows_host.argtypes = [ci, ci, ci, vp]
    L.bd_attn_group_windows_host.restype = ci
    L.bd_attn_group_windows_host.argtypes = [ci, ci, ci, ci, vp]
    L.bd_attn_status_string.restype = ctypes.c_char_p
    L.bd_attn_status_string.argtypes = [ci]
    L.bd_attn_version.restype = ci
    L.bd_attn_version.argtypes = []
    _lib = L
    return L


def status_string(status: int) -> str:
    return lib().bd_attn_status_string(int(status)).decode()
