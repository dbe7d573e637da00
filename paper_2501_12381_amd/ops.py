"""Torch-facing wrappers over the C ABI (argument marshalling only).

Every step of the scan runs in libgspn.so's HIP kernels; torch provides the
device memory and the current stream.  Tensors must live on a ROCm device:
there is no CPU path.

Options (keyword arguments, all default off):
  group_h, group_w : local-GSPN group lengths along the rows (T2B/B2T) and
                     columns (L2R/R2L); 0 is the global scan;
  logits, renorm   : w holds logits normalised by Eq. 6 inside the call
                     (renorm: over the on-line neighbours only);
  lam_per_dir, u_per_dir, y_per_dir : lam / u / y (and dy) stacked per
                     direction, shape (n, B, C, H, W);
  save_state       : the forward keeps its states in the workspace for the
                     backward, which then does not recompute them (pass the
                     same `workspace` tensor, from `scan_workspace`, to both
                     calls; the two-pass kernels use it, others ignore it).
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

from . import lib as L

_DT = {torch.float32: L.GSPN_F32, torch.bfloat16: L.GSPN_BF16}


def n_dirs(mask: int) -> int:
    return bin(mask & 0xF).count("1")


@dataclass(frozen=True)
class ScanOptions:
    group_h: int = 0
    group_w: int = 0
    logits: bool = False
    renorm: bool = False
    lam_per_dir: bool = False
    u_per_dir: bool = False
    y_per_dir: bool = False
    save_state: bool = False

    @property
    def flags(self) -> int:
        return ((L.GSPN_FLAG_W_LOGITS if self.logits else 0) | (L.GSPN_FLAG_EDGE_RENORM if self.renorm else 0)
                | (L.GSPN_FLAG_LAM_PER_DIR if self.lam_per_dir else 0)
                | (L.GSPN_FLAG_U_PER_DIR if self.u_per_dir else 0)
                | (L.GSPN_FLAG_Y_PER_DIR if self.y_per_dir else 0)
                | (L.GSPN_FLAG_SAVE_STATE if self.save_state else 0))


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype not in _DT:
        raise TypeError(f"GSPN scan supports float32 and bfloat16, got {t.dtype}")
    return _DT[t.dtype]


def _shape(base, per_dir: bool, n: int):
    return ((n,) if per_dir else ()) + tuple(base)


def _check(x, w, lam, u, mask, opt: ScanOptions):
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
    n = n_dirs(mask)
    if lam.shape != _shape(x.shape, opt.lam_per_dir, n):
        raise ValueError(f"lam must be {_shape(x.shape, opt.lam_per_dir, n)}, got {tuple(lam.shape)}")
    if u.shape != _shape(x.shape, opt.u_per_dir, n):
        raise ValueError(f"u must be {_shape(x.shape, opt.u_per_dir, n)}, got {tuple(u.shape)}")
    if w.shape != (n, 3) + tuple(x.shape):
        raise ValueError(f"w must be {(n, 3) + tuple(x.shape)}, got {tuple(w.shape)}")


def _stream(dev) -> int:
    return torch.cuda.current_stream(dev).cuda_stream


def _ptr(t):
    return t.data_ptr() if t is not None else None


def scan_workspace(x, mask: int, *, algo: int = L.GSPN_ALGO_AUTO, group_h: int = 0, group_w: int = 0,
                   **options) -> torch.Tensor:
    """A workspace that serves a forward call and the backward call that
    follows it (the backward's size covers the forward's; with save_state the
    forward leaves its states at the start for the backward)."""
    opt = ScanOptions(group_h, group_w, **options)
    B, C, H, W = x.shape
    dt = _dtype_code(x)
    need = max(L.gspn_scan_fwd_workspace_bytes(B, C, H, W, mask, dt, group_h, group_w, opt.flags, algo),
               L.gspn_scan_bwd_workspace_bytes(B, C, H, W, mask, dt, group_h, group_w, opt.flags, algo))
    return torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)


def gspn_scan_fwd(x, w, lam, u, mask: int, *, algo: int = L.GSPN_ALGO_AUTO, y=None, workspace=None,
                  group_h: int = 0, group_w: int = 0, logits: bool = False, renorm: bool = False,
                  lam_per_dir: bool = False, u_per_dir: bool = False,
                  y_per_dir: bool = False, save_state: bool = False) -> torch.Tensor:
    """y = u * sum_{d in mask} h_d (forward line scan of all directions in mask)."""
    opt = ScanOptions(group_h, group_w, logits, renorm, lam_per_dir, u_per_dir, y_per_dir, save_state)
    _check(x, w, lam, u, mask, opt)
    if save_state and workspace is None:
        raise ValueError("save_state keeps the forward's states in `workspace`: pass one (scan_workspace)")
    x, w, lam, u = (t.contiguous() for t in (x, w, lam, u))
    B, C, H, W = x.shape
    dt = _dtype_code(x)
    yshape = _shape(x.shape, y_per_dir, n_dirs(mask))
    if y is None:
        y = torch.empty(yshape, dtype=x.dtype, device=x.device)
    elif y.shape != yshape or y.dtype != x.dtype or not y.is_contiguous():
        raise ValueError(f"y must be a contiguous {x.dtype} tensor of shape {yshape}")
    need = L.gspn_scan_fwd_workspace_bytes(B, C, H, W, mask, dt, group_h, group_w, opt.flags, algo)
    if workspace is None or workspace.numel() < need:
        if save_state:
            raise ValueError(f"the workspace holds {workspace.numel()} bytes, the forward needs {need}")
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    with torch.cuda.device(x.device):
        st = L.gspn_scan_fwd(_ptr(x), _ptr(w), _ptr(lam), _ptr(u), _ptr(y), B, C, H, W, mask, dt,
                             group_h, group_w, opt.flags, algo, _ptr(workspace), workspace.numel(),
                             _stream(x.device))
    if st != 0:
        raise L.GSPNError(st, "gspn_scan_fwd")
    return y


def gspn_scan_bwd(dy, x, w, lam, u, mask: int, *, algo: int = L.GSPN_ALGO_AUTO, workspace=None,
                  out=None, group_h: int = 0, group_w: int = 0, logits: bool = False,
                  renorm: bool = False, lam_per_dir: bool = False, u_per_dir: bool = False,
                  y_per_dir: bool = False, save_state: bool = False):
    """Gradients (dx, dw, dlam, du) of <dy, y> for the forward above.

    `out` = (dx, dw, dlam, du): optional contiguous output tensors (else new ones).
    save_state: `workspace` is the one the forward (called with save_state)
    filled, unchanged since."""
    opt = ScanOptions(group_h, group_w, logits, renorm, lam_per_dir, u_per_dir, y_per_dir, save_state)
    _check(x, w, lam, u, mask, opt)
    if save_state and workspace is None:
        raise ValueError("save_state reads the forward's states from `workspace`: pass the forward's")
    if dy.shape != _shape(x.shape, y_per_dir, n_dirs(mask)) or dy.dtype != x.dtype or dy.device != x.device:
        raise ValueError("dy must be shaped like y, typed and placed like x")
    dy, x, w, lam, u = (t.contiguous() for t in (dy, x, w, lam, u))
    B, C, H, W = x.shape
    dt = _dtype_code(x)
    if out is None:
        dx, dlam, du, dw = (torch.empty_like(x), torch.empty_like(lam), torch.empty_like(u),
                            torch.empty_like(w))
    else:
        dx, dw, dlam, du = out
        for t, ref in ((dx, x), (dw, w), (dlam, lam), (du, u)):
            if t.shape != ref.shape or t.dtype != x.dtype or t.device != x.device or not t.is_contiguous():
                raise ValueError("out tensors must be contiguous and shaped like (x, w, lam, u)")
    need = L.gspn_scan_bwd_workspace_bytes(B, C, H, W, mask, dt, group_h, group_w, opt.flags, algo)
    if workspace is None or workspace.numel() < need:
        if save_state:
            raise ValueError(f"the workspace holds {workspace.numel()} bytes, the backward needs {need}")
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    with torch.cuda.device(x.device):
        st = L.gspn_scan_bwd(_ptr(dy), _ptr(x), _ptr(w), _ptr(lam), _ptr(u), _ptr(dx), _ptr(dw),
                             _ptr(dlam), _ptr(du), B, C, H, W, mask, dt, group_h, group_w, opt.flags,
                             algo, _ptr(workspace), workspace.numel(), _stream(x.device))
    if st != 0:
        raise L.GSPNError(st, "gspn_scan_bwd")
    return dx, dw, dlam, du


class GSPNScan(torch.autograd.Function):
    """Autograd wrapper: forward and backward both run the HIP kernels."""

    @staticmethod
    def forward(ctx, x, w, lam, u, mask: int, algo: int = L.GSPN_ALGO_AUTO, opt: ScanOptions = ScanOptions()):
        ctx.mask, ctx.algo, ctx.opt = mask, algo, opt
        ctx.save_for_backward(x, w, lam, u)
        # with save_state the workspace carries the forward's states to the backward
        ctx.ws = scan_workspace(x, mask, algo=algo, **opt.__dict__) if opt.save_state else None
        return gspn_scan_fwd(x, w, lam, u, mask, algo=algo, workspace=ctx.ws, **opt.__dict__)

    @staticmethod
    def backward(ctx, dy):
        x, w, lam, u = ctx.saved_tensors
        dx, dw, dlam, du = gspn_scan_bwd(dy.contiguous(), x, w, lam, u, ctx.mask, algo=ctx.algo,
                                         workspace=ctx.ws, **ctx.opt.__dict__)
        ctx.ws = None
        return dx, dw, dlam, du, None, None, None


def gspn_scan(x, w, lam, u, mask: int = 0xF, algo: int = L.GSPN_ALGO_AUTO, **options) -> torch.Tensor:
    """Differentiable 4-direction (or masked) GSPN line scan; `options` as in ScanOptions."""
    return GSPNScan.apply(x, w, lam, u, mask, algo, ScanOptions(**options))


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
