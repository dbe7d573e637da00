"""Torch-facing wrappers over the C ABI (argument marshalling only).

Every step of the scan runs in libgspn.so's HIP kernels; torch provides the
device memory and the current stream.  Tensors must live on a ROCm device:
there is no CPU path.
"""
from __future__ import annotations

import torch

from . import lib as L

_DT = {torch.float32: L.GSPN_F32, torch.bfloat16: L.GSPN_BF16}


def n_dirs(mask: int) -> int:
    return bin(mask & 0xF).count("1")


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype not in _DT:
        raise TypeError(f"GSPN scan supports float32 and bfloat16, got {t.dtype}")
    return _DT[t.dtype]


def _check(x, w, lam, u, mask):
    for name, t in (("x", x), ("w", w), ("lam", lam), ("u", u)):
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{name} must be a tensor")
        if t.device.type != "cuda":
            raise RuntimeError(f"{name} is on {t.device}: the GSPN scan runs on the GPU only")
        if t.dtype != x.dtype:
            raise TypeError(f"{name} has dtype {t.dtype}, expected {x.dtype}")
        if t.device != x.device:
            raise RuntimeError(f"{name} is on {t.device}, expected {x.device}")
    if x.dim() != 4:
        raise ValueError("x must be (B, C, H, W)")
    if lam.shape != x.shape or u.shape != x.shape:
        raise ValueError("lam and u must have the shape of x")
    if w.shape != (n_dirs(mask), 3) + tuple(x.shape):
        raise ValueError(f"w must be {(n_dirs(mask), 3) + tuple(x.shape)}, got {tuple(w.shape)}")


def _stream(dev) -> int:
    return torch.cuda.current_stream(dev).cuda_stream


def _ptr(t):
    return t.data_ptr() if t is not None else None


def gspn_scan_fwd(x, w, lam, u, mask: int, *, algo: int = L.GSPN_ALGO_AUTO, y=None,
                  workspace=None) -> torch.Tensor:
    """y = u * sum_{d in mask} h_d (forward line scan of all directions in mask)."""
    _check(x, w, lam, u, mask)
    x, w, lam, u = (t.contiguous() for t in (x, w, lam, u))
    B, C, H, W = x.shape
    dt = _dtype_code(x)
    if y is None:
        y = torch.empty_like(x)
    elif y.shape != x.shape or y.dtype != x.dtype or not y.is_contiguous():
        raise ValueError("y must be a contiguous tensor shaped and typed like x")
    need = L.gspn_scan_fwd_workspace_bytes(B, C, H, W, mask, dt, algo)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    with torch.cuda.device(x.device):
        st = L.gspn_scan_fwd(_ptr(x), _ptr(w), _ptr(lam), _ptr(u), _ptr(y), B, C, H, W, mask, dt,
                             algo, _ptr(workspace), workspace.numel(), _stream(x.device))
    if st != 0:
        raise L.GSPNError(st, "gspn_scan_fwd")
    return y


def gspn_scan_bwd(dy, x, w, lam, u, mask: int, *, algo: int = L.GSPN_ALGO_AUTO, workspace=None):
    """Gradients (dx, dw, dlam, du) of <dy, y> for the forward above."""
    _check(x, w, lam, u, mask)
    if dy.shape != x.shape or dy.dtype != x.dtype or dy.device != x.device:
        raise ValueError("dy must be shaped, typed and placed like x")
    dy, x, w, lam, u = (t.contiguous() for t in (dy, x, w, lam, u))
    B, C, H, W = x.shape
    dt = _dtype_code(x)
    dx, dlam, du, dw = (torch.empty_like(x), torch.empty_like(x), torch.empty_like(x),
                        torch.empty_like(w))
    need = L.gspn_scan_bwd_workspace_bytes(B, C, H, W, mask, dt, algo)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    with torch.cuda.device(x.device):
        st = L.gspn_scan_bwd(_ptr(dy), _ptr(x), _ptr(w), _ptr(lam), _ptr(u), _ptr(dx), _ptr(dw),
                             _ptr(dlam), _ptr(du), B, C, H, W, mask, dt, algo, _ptr(workspace),
                             workspace.numel(), _stream(x.device))
    if st != 0:
        raise L.GSPNError(st, "gspn_scan_bwd")
    return dx, dw, dlam, du


class GSPNScan(torch.autograd.Function):
    """Autograd wrapper: forward and backward both run the HIP kernels."""

    @staticmethod
    def forward(ctx, x, w, lam, u, mask: int, algo: int = L.GSPN_ALGO_AUTO):
        ctx.mask, ctx.algo = mask, algo
        ctx.save_for_backward(x, w, lam, u)
        return gspn_scan_fwd(x, w, lam, u, mask, algo=algo)

    @staticmethod
    def backward(ctx, dy):
        x, w, lam, u = ctx.saved_tensors
        dx, dw, dlam, du = gspn_scan_bwd(dy.contiguous(), x, w, lam, u, ctx.mask, algo=ctx.algo)
        return dx, dw, dlam, du, None, None


def gspn_scan(x, w, lam, u, mask: int = 0xF, algo: int = L.GSPN_ALGO_AUTO) -> torch.Tensor:
    """Differentiable 4-direction (or masked) GSPN line scan."""
    return GSPNScan.apply(x, w, lam, u, mask, algo)


def gspn_copy_calibration(src: torch.Tensor, dst: torch.Tensor) -> None:
    """Copy src into dst with the library's reference copy kernel (known traffic)."""
    if src.device.type != "cuda" or dst.device != src.device:
        raise RuntimeError("gspn_copy_calibration runs on the GPU only")
    n = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() < n:
        raise ValueError("dst is smaller than src")
    with torch.cuda.device(src.device):
        st = L.gspn_copy_calibration(src.data_ptr(), dst.data_ptr(), n, _stream(src.device))
    if st != 0:
        raise L.GSPNError(st, "gspn_copy_calibration")
