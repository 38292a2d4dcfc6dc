"""ctypes loader for libcompact.so and the raw C signatures of include/compact.h."""
from __future__ import annotations

import ctypes
import os

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "libcompact.so")

c_i64, c_u64, c_int, c_size, c_vp, c_f64 = (ctypes.c_int64, ctypes.c_uint64, ctypes.c_int,
                                           ctypes.c_size_t, ctypes.c_void_p, ctypes.c_double)

SIGNATURES = {
    "compact_fwd": (c_int, [c_vp, c_i64, c_vp, c_i64, c_vp, c_i64, c_vp, c_i64, c_i64, c_i64,
                            c_i64, c_i64, c_u64, c_int, c_int, c_vp, c_size, c_vp]),
    "compact_fwd_workspace_bytes": (c_size, [c_i64, c_i64, c_i64, c_int]),
    "compact_fwd_group": (c_int, [c_vp, c_i64, c_vp, c_i64, c_vp, c_i64, c_vp, c_i64, c_i64, c_i64,
                                  ctypes.c_int32, ctypes.POINTER(c_i64), ctypes.POINTER(c_i64),
                                  ctypes.POINTER(c_u64), c_int, c_int, c_vp, c_size, c_vp]),
    "compact_fwd_group_workspace_bytes": (c_size, [c_i64, ctypes.c_int32, ctypes.POINTER(c_i64),
                                                   ctypes.POINTER(c_i64), c_int]),
    "compact_bwd": (c_int, [c_vp, c_i64, c_vp, c_i64, c_vp, c_i64, c_vp, c_i64, c_vp, c_i64,
                            c_i64, c_i64, c_i64, c_int, c_vp, c_size, c_vp]),
    "compact_bwd_workspace_bytes": (c_size, [c_i64, c_i64, c_i64, c_i64, c_int]),
    "compact_bwd_noalloc": (c_int, [c_vp, c_i64, c_vp, c_i64, c_vp, c_i64, c_vp, c_i64, c_vp, c_i64,
                                    c_i64, c_i64, c_i64, c_int, c_vp]),
    "compact_bwd_group": (c_int, [c_vp, c_i64, c_vp, c_i64, c_vp, c_i64, c_vp, c_i64,
                                  ctypes.POINTER(c_vp), c_i64, c_i64, ctypes.c_int32, ctypes.POINTER(c_i64),
                                  ctypes.POINTER(c_i64), c_int, c_int, c_vp, c_size, c_vp]),
    "compact_bwd_group_workspace_bytes": (c_size, [c_i64, c_i64, ctypes.c_int32, ctypes.POINTER(c_i64),
                                                   ctypes.POINTER(c_i64), c_int]),
    "compact_step": (c_int, [c_vp, c_i64, c_vp, c_vp, c_vp, c_i64, c_i64, c_i64, c_u64, c_i64,
                             c_f64, c_f64, c_f64, c_f64, c_f64, c_int, c_int, c_int, c_vp, c_size,
                             c_vp]),
    "compact_step_workspace_bytes": (c_size, [c_i64, c_i64, c_i64, c_int]),
    "compact_pstream": (c_int, [c_u64, c_i64, c_i64, c_vp, c_i64, c_vp]),
    "compact_projection": (c_int, [c_u64, c_i64, c_i64, c_int, c_vp, c_i64, c_vp]),
    "compact_pstream_boxmuller": (c_int, [c_vp, c_vp, c_vp, c_vp, c_i64, c_vp]),
    "compact_next_seed": (c_u64, [c_u64, c_i64, c_i64]),
    "compact_saved_activation_elems": (c_i64, [c_i64, c_i64, c_i64]),
    "compact_status_string": (ctypes.c_char_p, [c_int]),
    "compact_last_error": (ctypes.c_char_p, []),
    "compact_version": (c_int, []),
}


class CompactLayer(ctypes.Structure):
    """compact_layer of include/compact.h."""
    _fields_ = [("W", c_vp), ("ldw", c_i64), ("G", c_vp), ("M", c_vp), ("V", c_vp),
                ("n", c_i64), ("m", c_i64), ("r", c_i64), ("seed", c_u64), ("alpha", c_f64)]


SIGNATURES["compact_step_batched"] = (c_int, [ctypes.POINTER(CompactLayer), ctypes.c_int32, c_i64, c_f64,
                                              c_f64, c_f64, c_f64, c_int, c_int, c_int, c_vp, c_size,
                                              c_vp])
SIGNATURES["compact_step_batched_workspace_bytes"] = (c_size, [ctypes.POINTER(CompactLayer),
                                                              ctypes.c_int32, c_int])

_lib = None


class CompactLibraryMissing(RuntimeError):
    pass


def load(path: str = LIB_PATH):
    """Load the HIP library (raises CompactLibraryMissing if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise CompactLibraryMissing(
            f"{path} is not built; run `python -m paper_2410_15352_amd.build` "
            "(there is no fallback implementation)")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib
