"""ctypes binding of libkmip.so (include/kmip.h).  Argument marshalling only."""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libkmip.so")

KMIP_OK = 0
KMIP_ERR_INVALID_ARG = 1
KMIP_ERR_UNSUPPORTED = 2
KMIP_ERR_WORKSPACE = 3
KMIP_ERR_HIP = 4
MAX_K = 512        # largest k for d <= 64
MAX_K_WIDE = 128   # largest k for d = 128

# kmip_bwd_variant_t
BWD_AUTO = 0
BWD_ATOMIC = 1
BWD_SEGMENTED = 2
BWD_BUCKETED = 3
BWD_KEY_AGGREGATED = 4

# Every symbol declared in include/kmip.h.
EXPORTS = (
    "kmip_topk_workspace_size", "kmip_topk", "kmip_topk_with_events", "kmip_attend", "kmip_fwd_workspace_size",
    "kmip_fwd", "kmip_attend_ex", "kmip_fwd_ex", "kmip_fwd_ex_with_events", "kmip_bwd_workspace_size", "kmip_bwd",
    "kmip_bwd_ex_workspace_size", "kmip_bwd_ex", "kmip_fwd_noalloc", "kmip_topk_prefilter_workspace_size",
    "kmip_topk_prefilter", "kmip_status_string", "kmip_last_error",
)

# bytes of the fixed per-device array kmip_fwd_noalloc works in
NOALLOC_SCRATCH_BYTES = 256 * 1024 * 1024

_lib = None


class KmipError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        super().__init__(f"kmip status {status}: {detail}")


def load(path: str = LIB_PATH):
    """Load libkmip.so.  Raises if it has not been built: there is no fallback."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is missing: build it with `python -m paper_2604_03815_amd.build` "
            "(or __graft_entry__.build()); k-MIP attention has no CPU fallback")
    lib = ctypes.CDLL(path)
    P, sz = ctypes.c_void_p, ctypes.c_size_t
    i32, i64, f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    lib.kmip_topk_workspace_size.argtypes = [i64, i32, i32, i32, i32]
    lib.kmip_topk_workspace_size.restype = sz
    lib.kmip_fwd_workspace_size.argtypes = [i64, i32, i32, i32, i32]
    lib.kmip_fwd_workspace_size.restype = sz
    lib.kmip_bwd_workspace_size.argtypes = [i64, i32, i32, i32, i32]
    lib.kmip_bwd_workspace_size.restype = sz
    lib.kmip_bwd_ex_workspace_size.argtypes = [i64, i32, i32, i32, i32, i32]
    lib.kmip_bwd_ex_workspace_size.restype = sz
    lib.kmip_topk.argtypes = [P, P, P, i32, i64, i32, i32, i32, P, P, sz, P]
    lib.kmip_topk_with_events.argtypes = [P, P, P, i32, i64, i32, i32, i32, P, P, sz, P, P, P]
    lib.kmip_attend.argtypes = [P, P, P, i64, i32, i32, i32, f32, P, P, P, P]
    lib.kmip_fwd.argtypes = [P, P, P, P, i32, i64, i32, i32, i32, f32, P, P, P, P, sz, P]
    lib.kmip_bwd.argtypes = [P, P, P, P, P, P, i64, i32, i32, i32, f32, P, P, P, i32, P, sz, P]
    lib.kmip_fwd_noalloc.argtypes = [P, P, P, i64, i32, i32, i32, f32, P, P, P, P]
    lib.kmip_attend_ex.argtypes = [P, P, P, i64, i32, i32, i32, i32, f32, P, P, f32, P, P, P]
    lib.kmip_fwd_ex.argtypes = [P, P, P, P, i32, i64, i32, i32, i32, i32, f32, P, f32, P, P, P, P, sz, P]
    lib.kmip_fwd_ex_with_events.argtypes = [P, P, P, P, i32, i64, i32, i32, i32, i32, f32, P, f32, P, P, P, P, sz, P,
                                            P, P, P]
    lib.kmip_bwd_ex.argtypes = [P, P, P, P, P, P, P, f32, i64, i32, i32, i32, i32, f32, P, P, P, i32, P, sz, P]
    lib.kmip_topk_prefilter_workspace_size.argtypes = [i64, i32, i32, i32]
    lib.kmip_topk_prefilter_workspace_size.restype = sz
    lib.kmip_topk_prefilter.argtypes = [P, P, i64, i32, i32, i32, P, P, P, sz, P]
    for f in ("kmip_topk", "kmip_topk_with_events", "kmip_attend", "kmip_fwd", "kmip_bwd",
              "kmip_fwd_noalloc", "kmip_attend_ex", "kmip_fwd_ex", "kmip_fwd_ex_with_events", "kmip_bwd_ex",
              "kmip_topk_prefilter"):
        getattr(lib, f).restype = ctypes.c_int
    lib.kmip_status_string.argtypes = [ctypes.c_int]
    lib.kmip_status_string.restype = ctypes.c_char_p
    lib.kmip_last_error.argtypes = []
    lib.kmip_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def check(status: int) -> None:
    if status != KMIP_OK:
        lib = load()
        detail = lib.kmip_last_error().decode() or lib.kmip_status_string(status).decode()
        raise KmipError(status, detail)
