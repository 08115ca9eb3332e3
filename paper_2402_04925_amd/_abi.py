"""ctypes view of the C ABI declared in include/tpdq.h (argument marshalling only)."""
from __future__ import annotations

import ctypes
import os
import threading

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtpdq.so")

OK, ERR_NULL, ERR_SHAPE, ERR_ALIGN, ERR_GIDX, ERR_WORKSPACE, ERR_UNSUPPORTED, ERR_HIP = range(8)
FP16, BF16 = 0, 1
PATH_ACTORDER, PATH_ORDERED, PATH_ACTORDER_GLOBAL = 0, 1, 2
OP_REORDER, OP_GEMM, OP_MLP, OP_GATED_MLP = 0, 1, 2, 3
LAYOUT_GPTQ, LAYOUT_TILED = 0, 1

EXPORTED = (
    "tpdq_reorder", "tpdq_pack_tiled", "tpdq_w4a16_gemm", "tpdq_mlp_shard", "tpdq_mlp_shard_noalloc",
    "tpdq_gated_mlp_shard",
    "tpdq_workspace_bytes",
    "tpdq_status_string", "tpdq_last_error", "tpdq_version",
)


class W4(ctypes.Structure):
    """struct tpdq_w4."""
    _fields_ = [
        ("qweight", ctypes.c_void_p), ("ld_q", ctypes.c_int64),
        ("scales", ctypes.c_void_p), ("ld_s", ctypes.c_int64),
        ("qzeros", ctypes.c_void_p), ("ld_z", ctypes.c_int64),
        ("g_idx", ctypes.c_void_p),
        ("K", ctypes.c_int32), ("N", ctypes.c_int32),
        ("group_size", ctypes.c_int32), ("num_groups", ctypes.c_int32),
        ("layout", ctypes.c_int32), ("zero_offset", ctypes.c_int32),
    ]


_lock = threading.Lock()
_lib = None


def _declare(lib):
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    pw = ctypes.POINTER(W4)
    lib.tpdq_reorder.argtypes = [pw, pw, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_int, ctypes.c_int,
                                 vp, sz, vp]
    lib.tpdq_reorder.restype = ctypes.c_int
    lib.tpdq_pack_tiled.argtypes = [pw, vp, vp]
    lib.tpdq_pack_tiled.restype = ctypes.c_int
    lib.tpdq_w4a16_gemm.argtypes = [vp, i64, i32, vp, pw, ctypes.c_int, ctypes.c_int, vp, i64, vp,
                                    sz, vp]
    lib.tpdq_w4a16_gemm.restype = ctypes.c_int
    lib.tpdq_mlp_shard.argtypes = [vp, i64, i32, vp, pw, pw, ctypes.c_int, ctypes.c_int, vp, vp, vp,
                                   sz, vp]
    lib.tpdq_mlp_shard.restype = ctypes.c_int
    lib.tpdq_mlp_shard_noalloc.argtypes = [vp, i64, i32, vp, pw, pw, ctypes.c_int, ctypes.c_int, vp,
                                           vp, vp]
    lib.tpdq_mlp_shard_noalloc.restype = ctypes.c_int
    lib.tpdq_gated_mlp_shard.argtypes = [vp, i64, i32, vp, pw, pw, pw, ctypes.c_int, ctypes.c_int, vp,
                                         vp, vp, sz, vp]
    lib.tpdq_gated_mlp_shard.restype = ctypes.c_int
    lib.tpdq_workspace_bytes.argtypes = [ctypes.c_int, i32, pw, pw]
    lib.tpdq_workspace_bytes.restype = sz
    lib.tpdq_status_string.argtypes = [ctypes.c_int]
    lib.tpdq_status_string.restype = ctypes.c_char_p
    lib.tpdq_last_error.argtypes = []
    lib.tpdq_last_error.restype = ctypes.c_char_p
    lib.tpdq_version.argtypes = []
    lib.tpdq_version.restype = ctypes.c_char_p
    return lib


def lib():
    """The loaded libtpdq.so. Raises if it has not been built: there is no
    fallback implementation."""
    global _lib
    if _lib is None:
        with _lock:
            if _lib is None:
                # torch bundles its own HIP runtime under a different file name;
                # loading torch first makes libtpdq bind to that same runtime
                # (one runtime per process) instead of pulling in a second one.
                try:
                    import torch  # noqa: F401
                except ImportError:
                    pass
                if not os.path.exists(LIB_PATH):
                    raise RuntimeError(
                        f"{LIB_PATH} is missing; build it with `python -m paper_2402_04925_amd.build`")
                _lib = _declare(ctypes.CDLL(LIB_PATH))
    return _lib


class TpdqError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        self.detail = detail
        name = lib().tpdq_status_string(status).decode()
        super().__init__(f"tpdq status {status} ({name}): {detail}")


def check(status: int) -> None:
    if status != OK:
        raise TpdqError(status, lib().tpdq_last_error().decode())
