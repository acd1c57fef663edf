"""Loader of the in-tree ``libpace.so`` and its C signatures (include/pace.h)."""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
library_path = os.path.join(_HERE, "libpace.so")
_lib = None


class PaceParams(ctypes.Structure):
    """Mirror of ``pace_params``."""
    _fields_ = [("w_wait", ctypes.c_double), ("gamma", ctypes.c_int32),
                ("window_min", ctypes.c_int32), ("beta", ctypes.c_double),
                ("r_max", ctypes.c_double)]


# (name, restype, argtypes) of every exported entry point.
P, i64, i32, d, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_double, ctypes.c_size_t
SIGNATURES = [
    ("pace_default_params", None, [P]),
    ("pace_workspace_bytes", ctypes.c_int, [ctypes.c_int, i64, i64, P]),
    ("pace_score", ctypes.c_int, [P, P, i64, i64, P, i32, P, P, i64, P, P, P, P, P, sz, P]),
    ("pace_budget", ctypes.c_int, [i64, i64, P, P, P]),
    ("pace_select", ctypes.c_int, [P, i64, i64, P, P, P, sz, P]),
    ("pace_compact", ctypes.c_int, [P, i64, i64, P, ctypes.c_int, P, P, P, P, P, P, P, sz, P]),
    ("pace_validate", ctypes.c_int, [P, P, i64, i64, P, i32, P, i64, P, P]),
    ("pace_filter_step", ctypes.c_int, [P, P, i64, i64, P, i32, P, P, i64, i64, i64, P, P, P, P, P, P,
                                        P, P, ctypes.c_int, P, P, P, P, P, P, P, sz, P]),
    ("pace_filter_step_noalloc", ctypes.c_int, [P, P, i64, i64, P, i32, P, P, i64, i64, i64, P, P, P, P, P,
                                                P, P, P, ctypes.c_int, P, P, P, P, P, P, P]),
    ("pace_group_score", ctypes.c_int, [P, i64, P, i64, P, P]),
    ("pace_group_expand", ctypes.c_int, [P, i64, i64, P, P, P]),
    ("pace_validate_groups", ctypes.c_int, [P, i64, i64, P, P]),
    ("pace_group_filter_step", ctypes.c_int, [P, P, i64, i64, P, i32, P, P, i64, P, i64, i64, i64, P, P, P,
                                              P, P, P, P, P, P, P, ctypes.c_int, P, P, P, P, P, P, P, sz, P]),
    ("pace_stream_admit", ctypes.c_int, [P, i64, d, P, i64, P, i64, P, P, P, P, P, P, P]),
    ("pace_stream_step", ctypes.c_int, [P, P, i64, i64, P, i32, P, P, i64, i64, i64, P, P, i64, P, i64, P,
                                        P, P, P, P, P, P, P, P, ctypes.c_int, P, P, P, P, P, P, P, sz, P]),
    ("pace_prefix_score", ctypes.c_int, [P, P, P, P, i64, i64, i64, i64, P, P]),
    ("pace_stale_k", ctypes.c_int, [P, P, P, i32, i64, i64, P, P, P]),
    ("pace_diagnostics", ctypes.c_int, [P, P, P, P, i32, P, i64, P, ctypes.c_int, P, P, P]),
    ("pace_time_next_kernel", ctypes.c_int, [ctypes.c_int, P, P]),
    ("pace_strerror", ctypes.c_char_p, [ctypes.c_int]),
]


def load(path: str = library_path):
    """Open the library; raises if it has not been built (no fallback exists)."""
    if not os.path.exists(path):
        raise ImportError("libpace.so is not built at %s; run __graft_entry__.build() "
                          "or python -m paper_2609_36830_amd.build" % path)
    h = ctypes.CDLL(path)
    for name, res, args in SIGNATURES:
        fn = getattr(h, name)
        fn.restype = res
        fn.argtypes = args
    return h


def lib():
    global _lib
    if _lib is None:
        _lib = load()
    return _lib
