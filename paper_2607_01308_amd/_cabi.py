"""ctypes view of libcmerge.so (include/cmerge.h). Loading fails loudly if the
library has not been built; there is no other implementation to fall back to."""

from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcmerge.so")

CM_OK = 0
CM_EINVAL = -1
CM_ESHAPE = -2
CM_EDTYPE = -3
CM_ENONFINITE = -4
CM_EHIP = -5
CM_EWORKSPACE = -6

CM_F32 = 0
CM_BF16 = 1
CM_ROPE_HALF = 0
CM_ROPE_INTERLEAVED = 1
CM_MAX_FRAGMENTS = 1024
NOALLOC_SCRATCH_BYTES = 64 << 20     # CM_NOALLOC_SCRATCH_BYTES

PLAN_STATUS, PLAN_N, PLAN_NUNIQUE, PLAN_TOUT, PLAN_HEADER = 0, 1, 2, 3, 4

# every symbol include/cmerge.h declares
EXPORTS = (
    "cm_version", "cm_last_error", "cm_status_string", "cm_plan_elems", "cm_workspace_size",
    "cm_fragment_hash", "cm_fragment_hash_select", "cm_fragment_knorm", "cm_equal_key_mask",
    "cm_canonical_order", "cm_multiset_order", "cm_bag_plan", "cm_render_merge",
    "cm_render_merge_devplan", "cm_render_merge_range", "cm_render_merge_hash", "cm_render_set",
    "cm_render_deliveries", "cm_render_deliveries_noalloc", "cm_render_deliveries_graph",
    "cm_graph_launch", "cm_graph_destroy",
    "cm_paged_workspace_size", "cm_paged_order", "cm_paged_hash_select", "cm_paged_tables",
    "cm_paged_render", "cm_paged_render_hash", "cm_paged_deliveries",
    "cm_timing_enable", "cm_timing_reset", "cm_timing_query",
)


class CmFragset(ctypes.Structure):
    _fields_ = [
        ("n", ctypes.c_int32),
        ("L", ctypes.c_int32),
        ("H", ctypes.c_int32),
        ("d", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
        ("table_host", ctypes.c_void_p),
        ("table_dev", ctypes.c_void_p),
    ]


class CmPagedset(ctypes.Structure):
    _fields_ = [
        ("n", ctypes.c_int32),
        ("L", ctypes.c_int32),
        ("H", ctypes.c_int32),
        ("d", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("block", ctypes.c_int32),
        ("pages", ctypes.c_int64),
        ("pool_dev", ctypes.c_void_p),
        ("table_host", ctypes.c_void_p),
        ("table_dev", ctypes.c_void_p),
        ("blocks_host", ctypes.c_void_p),
        ("blocks_dev", ctypes.c_void_p),
        ("n_blocks", ctypes.c_int64),
    ]


class CmRope(ctypes.Structure):
    _fields_ = [("base", ctypes.c_double), ("style", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class CmError(RuntimeError):
    def __init__(self, status: int, where: str, message: str):
        self.status = status
        super().__init__(f"{where}: {status_name(status)} ({status}): {message}")


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(
                f"{LIB_PATH} is missing: build it with paper_2607_01308_amd.build.build() "
                "(hipcc for gfx950); there is no CPU implementation of this library")
        L = ctypes.CDLL(LIB_PATH)
        P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        FS = ctypes.POINTER(CmFragset)
        PS = ctypes.POINTER(CmPagedset)
        sig = {
            "cm_version": (I32, []),
            "cm_last_error": (ctypes.c_char_p, []),
            "cm_status_string": (ctypes.c_char_p, [I32]),
            "cm_plan_elems": (SZ, [I32]),
            "cm_workspace_size": (I32, [FS, ctypes.POINTER(SZ)]),
            "cm_fragment_hash": (I32, [FS, P, P, SZ, P]),
            "cm_fragment_hash_select": (I32, [FS, P, I32, P, P, SZ, P]),
            "cm_equal_key_mask": (I32, [FS, P, P, P]),
            "cm_fragment_knorm": (I32, [FS, I32, I64, P, P, SZ, P]),
            "cm_canonical_order": (I32, [FS, P, P, P, P]),
            "cm_multiset_order": (I32, [FS, P, P, P, P]),
            "cm_bag_plan": (I32, [FS, P, I32, P]),
            "cm_render_merge": (I32, [FS, P, P, ctypes.POINTER(CmRope), P, I64, P, SZ, P]),
            "cm_render_merge_devplan": (I32, [FS, P, ctypes.POINTER(CmRope), P, I64, P, SZ, P]),
            "cm_render_merge_range": (I32, [FS, P, P, ctypes.POINTER(CmRope), I32, P, I64, P, SZ,
                                            P]),
            "cm_render_merge_hash": (I32, [FS, P, P, ctypes.POINTER(CmRope), P, P, P, I64, P, SZ,
                                           P]),
            "cm_render_set": (I32, [FS, P, I32, I64, ctypes.POINTER(CmRope), P, P, P, I64, P, SZ,
                                    P]),
            "cm_render_deliveries": (I32, [FS, I32, I64, ctypes.POINTER(CmRope), P, P, P, P, P,
                                           I64, P, SZ, P]),
            "cm_render_deliveries_noalloc": (I32, [FS, I32, I64, ctypes.POINTER(CmRope), P, P, P,
                                                   P, P, I64, P]),
            "cm_render_deliveries_graph": (I32, [FS, I32, I64, ctypes.POINTER(CmRope), P, P, P, P,
                                                 P, I64, P, SZ, ctypes.POINTER(P)]),
            "cm_graph_launch": (I32, [P, P]),
            "cm_graph_destroy": (I32, [P]),
            "cm_paged_workspace_size": (I32, [PS, ctypes.POINTER(SZ)]),
            "cm_paged_order": (I32, [PS, I32, I64, P, P, P, P, P, SZ, P]),
            "cm_paged_hash_select": (I32, [PS, P, I32, P, I32, P, SZ, P]),
            "cm_paged_tables": (I32, [PS, P, P, I64, P, P, P, ctypes.POINTER(I64)]),
            "cm_paged_render": (I32, [PS, P, P, ctypes.POINTER(CmRope), P, P, P, I64, P, SZ, P]),
            "cm_paged_render_hash": (I32, [PS, P, P, ctypes.POINTER(CmRope), P, P, P, P, P, P, P,
                                           SZ, P]),
            "cm_paged_deliveries": (I32, [PS, I32, I64, ctypes.POINTER(CmRope), P, P, I64, P, P,
                                          P, P, P, P, P, P, SZ, P]),
            "cm_timing_enable": (I32, [I32]),
            "cm_timing_reset": (I32, []),
            "cm_timing_query": (I32, [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                      ctypes.POINTER(I64)]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype, f.argtypes = res, args
        _lib = L
    return _lib


def status_name(status: int) -> str:
    return lib().cm_status_string(status).decode()


def check(status: int, where: str) -> None:
    if status != CM_OK:
        raise CmError(status, where, lib().cm_last_error().decode())
