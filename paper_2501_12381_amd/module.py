"""The GSPN module around the line scan (Sec. 4.1 "GSPN Module", Sec. 4.2
"Learnable merging", App. "Guaranteeing Dense Pairwise Connections").

A shared 1x1 convolution reduces the input to `hidden` channels; that reduced
map is the scan's x.  Three further 1x1 convolutions of it give the scan's
input-dependent parameters: u, the three weight logits of every direction and
lambda.  The scan (libgspn.so) normalises the logits with Eq. 6 in its load
prologue, runs the directions of `mask` (optionally as local GSPN groups) and
returns one map per direction, y_d = u * h_d.  A learnable linear layer (a
1x1 convolution over the n_dirs * hidden stacked maps) merges the directions
and projects back to `dim` channels.

The 1x1 convolutions are plain GEMMs and run through PyTorch's library
kernels; every step of the scan and its adjoint runs in the HIP kernels.
"""
from __future__ import annotations

import torch
from torch import nn

from . import ops


class GSPNModule(nn.Module):
    """y = merge(scan(reduce(inp); u, w, lambda from reduce(inp)))."""

    def __init__(self, dim: int, hidden: int, mask: int = 0xF, group_h: int = 0, group_w: int = 0,
                 edge_renorm: bool = False, bias: bool = True):
        super().__init__()
        if not 1 <= mask <= 15:
            raise ValueError("mask must be in [1, 15]")
        self.dim, self.hidden, self.mask = dim, hidden, mask
        self.n = ops.n_dirs(mask)
        self.group_h, self.group_w, self.edge_renorm = group_h, group_w, edge_renorm
        self.reduce = nn.Conv2d(dim, hidden, 1, bias=bias)
        self.proj_u = nn.Conv2d(hidden, hidden, 1, bias=bias)
        self.proj_w = nn.Conv2d(hidden, 3 * self.n * hidden, 1, bias=bias)
        self.proj_lam = nn.Conv2d(hidden, hidden, 1, bias=bias)
        self.merge = nn.Conv2d(self.n * hidden, dim, 1, bias=bias)

    def scan_inputs(self, inp: torch.Tensor):
        """x, w logits (n, 3, B, C, H, W), lambda and u of the scan."""
        x = self.reduce(inp)
        B, C, H, W = x.shape
        logits = self.proj_w(x).view(B, self.n, 3, C, H, W).permute(1, 2, 0, 3, 4, 5).contiguous()
        return x.contiguous(), logits, self.proj_lam(x).contiguous(), self.proj_u(x).contiguous()

    def forward(self, inp: torch.Tensor) -> torch.Tensor:
        x, logits, lam, u = self.scan_inputs(inp)
        ys = ops.gspn_scan(x, logits, lam, u, self.mask, group_h=self.group_h, group_w=self.group_w,
                           logits=True, renorm=self.edge_renorm, y_per_dir=True)  # (n, B, C, H, W)
        B, C, H, W = x.shape
        return self.merge(ys.permute(1, 0, 2, 3, 4).reshape(B, self.n * C, H, W))
