"""ctypes binding of libdresd.so (the C ABI declared in include/dresd.h).

Argument marshalling only: every step of the search runs in the library's
HIP kernels.  There is no fallback: if the library cannot be loaded, loading
raises.
"""
from __future__ import annotations

import ctypes
import os
import threading

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdresd.so")

OK, EINVAL, ENOMEM, EDEVICE, EUNSUPPORTED = 0, 1, 2, 3, 4
K_MAX = 1024
F32, F16, BF16 = 0, 1, 2

EXPORTS = ["dresd_index_create", "dresd_search", "dresd_index_info", "dresd_index_destroy",
           "dresd_last_error", "dresd_profile_enable", "dresd_profile_read",
           "dresd_search_plan", "dresd_search_filtered", "dresd_transform",
           "dresd_pack_drafts", "dresd_ivf_create", "dresd_ivf_destroy", "dresd_ivf_info",
           "dresd_ivf_search", "dresd_ivf_search_filtered", "dresd_ivf_search_probes",
           "dresd_ivf_create_by_token", "dresd_ivf_search_next_token", "dresd_ivf_profile_enable",
           "dresd_ivf_profile_read", "dresd_kmeans_assign", "dresd_kmeans_update",
           "dresd_kmeans_init", "dresd_bw_probe", "dresd_search_noalloc"]

_lock = threading.Lock()
_lib = None


class DresdError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("dresd status %d: %s" % (status, msg))
        self.status = status


def _declare(lib):
    P, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.dresd_index_create.argtypes = [P, P, I64, I32, I32, I32, P, ctypes.POINTER(P)]
    lib.dresd_index_create.restype = ctypes.c_int
    lib.dresd_search.argtypes = [P, P, I32, I32, P, P, P, P]
    lib.dresd_search.restype = ctypes.c_int
    lib.dresd_search_filtered.argtypes = [P, P, P, I32, I32, P, P, P, P]
    lib.dresd_search_filtered.restype = ctypes.c_int
    F = ctypes.c_float
    lib.dresd_transform.argtypes = [P, I64, I32, P, P, F, P, I32, F, P, P]
    lib.dresd_transform.restype = ctypes.c_int
    lib.dresd_pack_drafts.argtypes = [P, I32, I32, I32, I32, I32, I32, P, P, P]
    lib.dresd_pack_drafts.restype = ctypes.c_int
    lib.dresd_ivf_create.argtypes = [P, P, I64, I32, I32, I32, P, I32, P, P, ctypes.POINTER(P)]
    lib.dresd_ivf_create.restype = ctypes.c_int
    lib.dresd_ivf_destroy.argtypes = [P]
    lib.dresd_ivf_destroy.restype = None
    lib.dresd_ivf_info.argtypes = [P, ctypes.POINTER(I64), ctypes.POINTER(I32),
                                   ctypes.POINTER(I32), ctypes.POINTER(I32), ctypes.POINTER(I32),
                                   ctypes.POINTER(I64)]
    lib.dresd_ivf_info.restype = ctypes.c_int
    lib.dresd_ivf_search.argtypes = [P, P, I32, I32, I32, P, P, P, P]
    lib.dresd_ivf_search.restype = ctypes.c_int
    lib.dresd_ivf_search_filtered.argtypes = [P, P, P, I32, I32, I32, P, P, P, P]
    lib.dresd_ivf_search_filtered.restype = ctypes.c_int
    lib.dresd_ivf_search_probes.argtypes = [P, P, P, I32, P, I32, I32, P, P, P, P]
    lib.dresd_ivf_search_probes.restype = ctypes.c_int
    lib.dresd_ivf_create_by_token.argtypes = [P, P, I64, I32, I32, I32, P, ctypes.POINTER(P)]
    lib.dresd_ivf_create_by_token.restype = ctypes.c_int
    lib.dresd_ivf_search_next_token.argtypes = [P, P, P, I32, I32, P, P, P, P]
    lib.dresd_ivf_search_next_token.restype = ctypes.c_int
    lib.dresd_ivf_profile_enable.argtypes = [P, I32]
    lib.dresd_ivf_profile_enable.restype = ctypes.c_int
    lib.dresd_ivf_profile_read.argtypes = [P, ctypes.POINTER(ctypes.c_double),
                                           ctypes.POINTER(ctypes.c_double), ctypes.POINTER(I64)]
    lib.dresd_ivf_profile_read.restype = ctypes.c_int
    lib.dresd_kmeans_assign.argtypes = [P, I64, I32, I32, P, I32, P, P, P]
    lib.dresd_kmeans_assign.restype = ctypes.c_int
    lib.dresd_kmeans_update.argtypes = [P, I64, I32, I32, P, I32, P, P, P]
    lib.dresd_kmeans_update.restype = ctypes.c_int
    lib.dresd_kmeans_init.argtypes = [P, I64, I32, I32, I32, ctypes.c_uint64, P, P]
    lib.dresd_kmeans_init.restype = ctypes.c_int
    lib.dresd_index_info.argtypes = [P, ctypes.POINTER(I64), ctypes.POINTER(I32),
                                     ctypes.POINTER(I32), ctypes.POINTER(I32)]
    lib.dresd_index_info.restype = ctypes.c_int
    lib.dresd_index_destroy.argtypes = [P]
    lib.dresd_index_destroy.restype = None
    lib.dresd_last_error.argtypes = []
    lib.dresd_last_error.restype = ctypes.c_char_p
    lib.dresd_profile_enable.argtypes = [P, I32]
    lib.dresd_profile_enable.restype = ctypes.c_int
    lib.dresd_profile_read.argtypes = [P, ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(ctypes.c_double), ctypes.POINTER(I64)]
    lib.dresd_profile_read.restype = ctypes.c_int
    lib.dresd_search_plan.argtypes = [P, I32, I32, ctypes.POINTER(I32), ctypes.POINTER(I32),
                                      ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(I32),
                                      ctypes.POINTER(I32)]
    lib.dresd_search_plan.restype = ctypes.c_int
    lib.dresd_bw_probe.argtypes = [P, I64, I32, I32, ctypes.POINTER(ctypes.c_double), P]
    lib.dresd_bw_probe.restype = ctypes.c_int
    lib.dresd_search_noalloc.argtypes = [P, P, I32, I32, P, P, P, P]
    lib.dresd_search_noalloc.restype = ctypes.c_int
    return lib


def load(path: str | None = None):
    """Load the library (building it first only if no build exists)."""
    global _lib
    with _lock:
        if _lib is None:
            p = path or LIB_PATH
            if not os.path.exists(p):
                from . import build as _build
                _build.build()
            _lib = _declare(ctypes.CDLL(p))
    return _lib


def check(status: int):
    if status != OK:
        raise DresdError(status, load().dresd_last_error().decode())
