"""ctypes binding of librettention.so (C ABI in include/rettention.h).

Argument marshalling only: every computation runs in the HIP library.  The
library must be built (``python -m paper_2505_22918_amd.build``); loading fails
loudly when it is missing.
"""

from __future__ import annotations

import ctypes
import os
import re

_PKG = os.path.dirname(os.path.abspath(__file__))
# RT_LIB_PATH selects another build of the same C ABI (the host-only sanitizer
# build that the CPU tests drive); there is still no fallback when it is missing.
LIB_PATH = os.environ.get("RT_LIB_PATH") or os.path.join(_PKG, "librettention.so")
HEADER = os.path.join(os.path.dirname(_PKG), "include", "rettention.h")

RT_OK, RT_EINVAL, RT_EUNSUPPORTED, RT_ECAPACITY, RT_EHIP = range(5)

c_int32 = ctypes.c_int32
c_float = ctypes.c_float
c_void_p = ctypes.c_void_p


class RtDims(ctypes.Structure):
    _fields_ = [("B", c_int32), ("H", c_int32), ("T", c_int32), ("D", c_int32)]


class RtBsr(ctypes.Structure):
    _fields_ = [
        ("row_ptr", c_void_p),
        ("col_idx", c_void_p),
        ("block", c_int32),
        ("n_qblk", c_int32),
        ("nnz", c_int32),
        ("n_masks", c_int32),
    ]


class RtPattern(ctypes.Structure):
    _fields_ = [
        ("kind", c_int32),
        ("mask", c_void_p),
        ("host_mask", c_void_p),
        ("grid_h", c_int32),
        ("grid_w", c_int32),
        ("frames", c_int32),
        ("n_text", c_int32),
        ("keep", c_int32),
        ("n_masks", c_int32),
    ]


_SIGS = {
    "rt_bsr_check": (c_int32, [ctypes.POINTER(RtBsr), c_void_p, c_void_p]),
    "rt_dynamic_index_workspace": (c_int32, [RtDims, c_int32, c_int32, ctypes.POINTER(ctypes.c_int64)]),
    "rt_dynamic_index_noalloc": (c_int32, [c_void_p, c_void_p, RtDims, c_int32, c_int32, c_void_p, c_void_p,
                                           c_int32, c_void_p]),
    "rt_dynamic_index": (c_int32, [c_void_p, c_void_p, RtDims, c_int32, c_int32, c_void_p, c_void_p, c_int32,
                                   c_void_p, ctypes.c_int64, c_void_p]),
    "rt_index_size": (c_int32, [ctypes.POINTER(RtPattern), c_int32, c_int32, ctypes.POINTER(c_int32)]),
    "rt_index_build": (c_int32, [ctypes.POINTER(RtPattern), c_int32, c_int32, c_void_p, c_void_p,
                                 c_int32, c_void_p]),
    "rt_attn_full": (c_int32, [c_void_p, c_void_p, c_void_p, RtDims, c_int32, c_void_p, c_void_p,
                               c_void_p, c_void_p]),
    "rt_attn_sparse": (c_int32, [c_void_p, c_void_p, c_void_p, RtDims, ctypes.POINTER(RtBsr),
                                 c_void_p, c_void_p, c_void_p, c_void_p]),
    "rt_attn_cache": (c_int32, [c_void_p, c_void_p, c_void_p, RtDims, ctypes.POINTER(RtBsr), c_void_p,
                                c_void_p, c_void_p, c_void_p, c_void_p, c_void_p]),
    "rt_attn_postmask": (c_int32, [c_void_p, c_void_p, c_void_p, RtDims, ctypes.POINTER(RtBsr), c_void_p,
                                   c_void_p]),
    "rt_cache_build": (c_int32, [c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, RtDims,
                                 c_void_p, c_void_p, c_void_p]),
    "rt_attn_sparse_reshape": (c_int32, [c_void_p, c_void_p, c_void_p, RtDims, ctypes.POINTER(RtBsr),
                                         c_void_p, c_void_p, c_float, c_void_p, c_void_p, c_void_p,
                                         c_void_p]),
    "rt_reshape_apply": (c_int32, [c_void_p, c_void_p, c_void_p, c_float, RtDims, c_void_p, c_void_p]),
    "rt_status_str": (ctypes.c_char_p, [c_int32]),
    "rt_last_error": (ctypes.c_char_p, []),
    "rt_version": (c_int32, []),
}

_lib = None


def header_symbols(path: str = HEADER):
    """Function names the public header declares."""
    with open(path) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(rt_\w+)\s*\(", text, re.M)))


def load(path: str = LIB_PATH):
    """Loads (once) and returns the library with typed entry points."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            f"librettention.so not found at {path}; build it with "
            "`python -m paper_2505_22918_amd.build` (there is no fallback path)")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


class RettentionError(RuntimeError):
    def __init__(self, fn, status, msg):
        super().__init__(f"{fn} failed: status {status} ({msg})")
        self.status = status


def check(fn_name: str, status: int):
    if status != RT_OK:
        lib = load()
        msg = lib.rt_last_error().decode() or lib.rt_status_str(status).decode()
        raise RettentionError(fn_name, status, msg)
