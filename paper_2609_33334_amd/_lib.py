"""ctypes loader for libdge.so: struct layout and function prototypes of include/dge.h.

The library is loaded from this package directory only.  A missing or stale
library raises immediately: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_double, c_int, c_int32, c_int64, c_size_t, c_void_p

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdge.so")

DGE_OK, DGE_ERR_INVALID, DGE_ERR_UNSUPPORTED, DGE_ERR_WORKSPACE, DGE_ERR_HIP = 0, 1, 2, 3, 4
DGE_BF16, DGE_F32 = 0, 1
ROWS_WINDOW_DRAFT, ROWS_DRAFT, ROWS_WINDOW = 0, 1, 2
OP_SCORE, OP_SELECT, OP_H2O = 0, 1, 2
ABI_VERSION = 1
NOALLOC_SCRATCH_BYTES = 16 << 20   # DGE_NOALLOC_SCRATCH_BYTES

# every entry point declared in include/dge.h
EXPORTS = ("dge_abi_version", "dge_status_string", "dge_workspace_size", "dge_score",
           "dge_score_noalloc", "dge_score_with_lse", "dge_score_lse", "dge_evicted_mass",
           "dge_select_topb", "dge_select_compact", "dge_select_compact_layers",
           "dge_select_streaming", "dge_compact", "dge_compact_inplace",
           "dge_cache_attention", "dge_rope", "dge_project_rope", "dge_project_rope_workspace", "dge_retained_runs", "dge_h2o_colsum",
           "dge_pyramid_budgets")


class Geom(ctypes.Structure):
    """dge_geom_t"""
    _fields_ = [
        ("batch", c_int32),
        ("n_q_heads", c_int32),
        ("n_kv_heads", c_int32),
        ("head_dim", c_int32),
        ("window", c_int32),
        ("k_draft", c_int32),
        ("kv_offsets", c_void_p),
        ("kv_offsets_host", c_void_p),
        ("kv_head_stride", c_int64),
        ("dtype", c_int32),
    ]


class DGEError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} (status {status})")


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"libdge.so not found at {LIB_PATH}; build it with "
            "`python -m paper_2609_33334_amd.build` (there is no fallback path)")
    L = ctypes.CDLL(LIB_PATH)
    GP = POINTER(Geom)
    L.dge_abi_version.restype = c_int
    L.dge_abi_version.argtypes = []
    L.dge_status_string.restype = c_char_p
    L.dge_status_string.argtypes = [c_int]
    L.dge_workspace_size.restype = c_int
    L.dge_workspace_size.argtypes = [GP, c_int32, POINTER(c_size_t)]
    L.dge_score.restype = c_int
    L.dge_score.argtypes = [GP, c_int32, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]
    L.dge_score_noalloc.restype = c_int
    L.dge_score_noalloc.argtypes = [GP, c_int32, c_void_p, c_void_p, c_void_p, c_void_p]
    L.dge_score_with_lse.restype = c_int
    L.dge_score_with_lse.argtypes = [GP, c_int32, c_void_p, c_void_p, c_void_p, c_void_p,
                                     c_void_p, c_size_t, c_void_p]
    L.dge_evicted_mass.restype = c_int
    L.dge_evicted_mass.argtypes = [GP, c_void_p, c_int32, c_int32, c_void_p, c_int32, c_int32,
                                   c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p]
    L.dge_score_lse.restype = c_int
    L.dge_score_lse.argtypes = [GP, c_int32, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p]
    L.dge_select_topb.restype = c_int
    L.dge_select_topb.argtypes = [GP, c_void_p, c_int32, c_int32, c_int32, c_void_p, c_void_p,
                                  c_void_p, c_size_t, c_void_p]
    L.dge_select_compact.restype = c_int
    L.dge_select_compact.argtypes = [GP, c_void_p, c_int32, c_int32, c_int32, c_void_p, c_void_p,
                                     c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t,
                                     c_void_p]
    L.dge_select_compact_layers.restype = c_int
    L.dge_select_compact_layers.argtypes = [GP, c_int32, c_void_p, c_int32, c_int32,
                                            POINTER(c_int32), c_void_p, c_void_p, c_void_p,
                                            c_void_p, c_void_p, c_void_p, c_void_p, c_size_t,
                                            c_void_p]
    L.dge_select_streaming.restype = c_int
    L.dge_select_streaming.argtypes = [GP, c_int32, c_int32, c_void_p, c_void_p, c_void_p]
    L.dge_compact.restype = c_int
    L.dge_compact.argtypes = [GP, c_void_p, c_void_p, c_int32, c_int32, c_void_p, c_void_p,
                              c_void_p, c_void_p, c_void_p]
    L.dge_compact_inplace.restype = c_int
    L.dge_compact_inplace.argtypes = [GP, c_void_p, c_void_p, c_int32, c_int32, c_void_p,
                                      c_void_p, c_void_p]
    L.dge_h2o_colsum.restype = c_int
    L.dge_cache_attention.restype = c_int
    L.dge_cache_attention.argtypes = [GP, c_void_p, c_int32, c_int32, c_void_p, c_void_p, c_int32,
                                      c_int32, c_void_p, c_void_p, c_void_p, c_void_p]
    L.dge_h2o_colsum.argtypes = [GP, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t,
                                 c_void_p]
    L.dge_rope.restype = c_int
    L.dge_rope.argtypes = [c_int32, c_int32, c_int32, c_int32, c_int64, c_void_p, c_double,
                           c_void_p, c_void_p]
    L.dge_project_rope.restype = c_int
    L.dge_project_rope.argtypes = [c_int32, c_int32, c_void_p, c_int32, c_int32, c_void_p, c_void_p,
                                   c_double, c_void_p, c_void_p, c_size_t, c_void_p]
    L.dge_project_rope_workspace.restype = c_int
    L.dge_project_rope_workspace.argtypes = [c_int32, c_int32, c_int32, c_int32, POINTER(c_size_t)]
    L.dge_retained_runs.restype = c_int
    L.dge_retained_runs.argtypes = [GP, c_void_p, c_void_p, c_int32, c_void_p, c_void_p, c_void_p]
    L.dge_pyramid_budgets.restype = c_int
    L.dge_pyramid_budgets.argtypes = [c_int32, c_int32, c_int32, c_int32, POINTER(c_int32)]
    if L.dge_abi_version() != ABI_VERSION:
        raise RuntimeError(f"libdge.so ABI {L.dge_abi_version()} != binding ABI {ABI_VERSION}; rebuild")
    _lib = L
    return L


def status_string(status: int) -> str:
    return lib().dge_status_string(int(status)).decode()


def check(status: int, where: str) -> None:
    if status != DGE_OK:
        raise DGEError(status, where)
