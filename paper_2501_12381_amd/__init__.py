"""GSPN 2D line-scan propagation on AMD Instinct MI355X (gfx950).

The scan itself lives in libgspn.so (HIP kernels behind the C ABI of
include/gspn.h); this package holds its build script, a ctypes binding
(`lib`), torch wrappers (`ops`) and the seeded input generators (`synth`).
"""
from .lib import (GSPN_ALGO_AUTO, GSPN_ALGO_RESIDENT, GSPN_ALGO_STREAM, GSPN_BF16,
                  GSPN_DIR_B2T, GSPN_DIR_L2R, GSPN_DIR_R2L, GSPN_DIR_T2B, GSPN_F32, GSPNError)

__all__ = ["GSPN_ALGO_AUTO", "GSPN_ALGO_RESIDENT", "GSPN_ALGO_STREAM", "GSPN_BF16",
           "GSPN_DIR_B2T", "GSPN_DIR_L2R", "GSPN_DIR_R2L", "GSPN_DIR_T2B", "GSPN_F32", "GSPNError"]
