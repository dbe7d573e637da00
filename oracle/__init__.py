"""Float64 CPU oracle for the GSPN line scan (test infrastructure only)."""
from .gspn_oracle import (ALL_DIRS, B2T, L2R, R2L, T2B, adjoint_direction, dirs_of,
                          g_blocks_t2b, line_matrix, normalize_logits,
                          normalize_logits_vjp, scan_bwd, scan_direction, scan_fwd,
                          scan_fwd_dirs)

__all__ = ["ALL_DIRS", "T2B", "B2T", "L2R", "R2L", "adjoint_direction", "dirs_of",
           "g_blocks_t2b", "line_matrix", "normalize_logits",
           "normalize_logits_vjp", "scan_bwd", "scan_direction", "scan_fwd",
           "scan_fwd_dirs"]
