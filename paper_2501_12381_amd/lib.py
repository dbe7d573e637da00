"""ctypes binding of libgspn.so: the C ABI declared in include/gspn.h.

Functions here have the C names and take plain integers for pointers and the
stream; `paper_2501_12381_amd.ops` wraps them for torch tensors.  Loading fails
loudly if the library has not been built: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libgspn.so")

GSPN_F32, GSPN_BF16 = 0, 1
GSPN_DIR_T2B, GSPN_DIR_B2T, GSPN_DIR_L2R, GSPN_DIR_R2L = 1, 2, 4, 8
GSPN_ALGO_AUTO, GSPN_ALGO_RESIDENT, GSPN_ALGO_STREAM, GSPN_ALGO_RESIDENT_GENERIC = 0, 1, 2, 3
GSPN_ALGO_TWO_PASS = 4
GSPN_FLAG_W_LOGITS, GSPN_FLAG_EDGE_RENORM, GSPN_FLAG_LAM_PER_DIR = 1, 2, 4
GSPN_FLAG_U_PER_DIR, GSPN_FLAG_Y_PER_DIR, GSPN_FLAG_SAVE_STATE = 8, 16, 32
GSPN_MAX_LINE = 4096
STATUS = {0: "GSPN_OK", 1: "GSPN_ERR_NULL", 2: "GSPN_ERR_SHAPE", 3: "GSPN_ERR_MASK",
          4: "GSPN_ERR_DTYPE", 5: "GSPN_ERR_ALIGN", 6: "GSPN_ERR_ALIAS",
          7: "GSPN_ERR_UNSUPPORTED", 8: "GSPN_ERR_WORKSPACE", 9: "GSPN_ERR_HIP"}

# every symbol include/gspn.h declares
EXPORTS = ("gspn_scan_fwd_workspace_bytes", "gspn_scan_fwd", "gspn_scan_fwd_noalloc",
           "gspn_scan_bwd_workspace_bytes", "gspn_scan_bwd", "gspn_copy_calibration", "gspn_strerror",
           "gspn_version")
GSPN_NOALLOC_SCRATCH_BYTES = 64 << 20

_lib = None

_p, _i64, _u32, _i, _sz = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint32, ctypes.c_int,
                           ctypes.c_size_t)


class GSPNError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)} ({gspn_strerror(status)})")


def load() -> ctypes.CDLL:
    """Load libgspn.so (once).  Raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2501_12381_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    ws_args = [_i64, _i64, _i64, _i64, _u32, _i, _i64, _i64, _u32, _i]
    lib.gspn_scan_fwd_workspace_bytes.argtypes = ws_args
    lib.gspn_scan_fwd_workspace_bytes.restype = _sz
    lib.gspn_scan_bwd_workspace_bytes.argtypes = ws_args
    lib.gspn_scan_bwd_workspace_bytes.restype = _sz
    lib.gspn_scan_fwd.argtypes = [_p, _p, _p, _p, _p, _i64, _i64, _i64, _i64, _u32, _i, _i64, _i64, _u32,
                                  _i, _p, _sz, _p]
    lib.gspn_scan_fwd.restype = _i
    lib.gspn_scan_fwd_noalloc.argtypes = [_p, _p, _p, _p, _p, _i64, _i64, _i64, _i64, _u32, _i, _i64, _i64,
                                          _u32, _p]
    lib.gspn_scan_fwd_noalloc.restype = _i
    lib.gspn_scan_bwd.argtypes = [_p, _p, _p, _p, _p, _p, _p, _p, _p, _i64, _i64, _i64, _i64, _u32,
                                  _i, _i64, _i64, _u32, _i, _p, _sz, _p]
    lib.gspn_scan_bwd.restype = _i
    lib.gspn_copy_calibration.argtypes = [_p, _p, _sz, _p]
    lib.gspn_copy_calibration.restype = _i
    lib.gspn_strerror.argtypes = [_i]
    lib.gspn_strerror.restype = ctypes.c_char_p
    lib.gspn_version.argtypes = []
    lib.gspn_version.restype = _i
    _lib = lib
    return lib


def gspn_scan_fwd_workspace_bytes(B, C, H, W, mask, dtype, group_h=0, group_w=0, flags=0,
                                  algo=GSPN_ALGO_AUTO) -> int:
    return int(load().gspn_scan_fwd_workspace_bytes(B, C, H, W, mask, dtype, group_h, group_w, flags,
                                                    algo))


def gspn_scan_bwd_workspace_bytes(B, C, H, W, mask, dtype, group_h=0, group_w=0, flags=0,
                                  algo=GSPN_ALGO_AUTO) -> int:
    return int(load().gspn_scan_bwd_workspace_bytes(B, C, H, W, mask, dtype, group_h, group_w, flags,
                                                    algo))


def gspn_scan_fwd(x, w, lam, u, y, B, C, H, W, mask, dtype, group_h, group_w, flags, algo, workspace,
                  workspace_bytes, stream) -> int:
    return int(load().gspn_scan_fwd(x, w, lam, u, y, B, C, H, W, mask, dtype, group_h, group_w, flags,
                                    algo, workspace, workspace_bytes, stream))


def gspn_scan_fwd_noalloc(x, w, lam, u, y, B, C, H, W, mask, dtype, group_h, group_w, flags,
                          stream) -> int:
    return int(load().gspn_scan_fwd_noalloc(x, w, lam, u, y, B, C, H, W, mask, dtype, group_h, group_w,
                                            flags, stream))


def gspn_scan_bwd(dy, x, w, lam, u, dx, dw, dlam, du, B, C, H, W, mask, dtype, group_h, group_w, flags,
                  algo, workspace, workspace_bytes, stream) -> int:
    return int(load().gspn_scan_bwd(dy, x, w, lam, u, dx, dw, dlam, du, B, C, H, W, mask, dtype,
                                    group_h, group_w, flags, algo, workspace, workspace_bytes, stream))


def gspn_copy_calibration(src, dst, nbytes, stream) -> int:
    return int(load().gspn_copy_calibration(src, dst, nbytes, stream))


def gspn_strerror(status: int) -> str:
    return load().gspn_strerror(status).decode()


def gspn_version() -> int:
    return int(load().gspn_version())
