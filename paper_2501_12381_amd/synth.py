"""Seeded synthetic inputs for the GSPN line scan.

This module is shared by the tests, the smoke check and the benchmark.  It only
draws random numbers and shapes them; it contains none of the propagation
arithmetic, so the oracle and the HIP path stay independent of each other.

Workloads (shape, dtype, direction mask, distributions) stand in for the
feature maps the paper runs GSPN on: classification stages at 224^2 input
(56^2 and 28^2 maps, Sec. 4.1 and the classification-model table) and diffusion
latents (128^2 for 1024^2 images, 2048^2 for the ~16K images of Sec. 5.6).
No dataset or trained weight is used.

Weights are produced the way the workloads prescribe: three logits per pixel
and direction, normalised over the three with a softmax so each row of the
tridiagonal w_i is stochastic (the Stability-Context Condition, Sec. 3.2).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import torch

DIR_T2B, DIR_B2T, DIR_L2R, DIR_R2L = 1, 2, 4, 8
DIR_NAMES = {DIR_T2B: "T2B", DIR_B2T: "B2T", DIR_L2R: "L2R", DIR_R2L: "R2L"}

# tensor ids used to derive one seed per generated tensor
_TID_X, _TID_LAM, _TID_U, _TID_DY = 0, 1, 2, 15


def mask_dirs(mask: int) -> list[int]:
    """Directions of a mask in increasing bit order (the packing order of w)."""
    return [d for d in (DIR_T2B, DIR_B2T, DIR_L2R, DIR_R2L) if mask & d]


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    C: int
    H: int
    W: int
    mask: int
    dtype: str  # "f32" or "bf16"
    x: str = "normal"  # N(0,1)
    lam: str = "uniform"  # "uniform" U(0,1) | "sigmoid" sigmoid(N(0,1)) | "ones"
    u: str = "ones"
    w_logit_std: float = 1.0
    backward: bool = False
    seed: int = 0
    extra: dict = field(default_factory=dict)
    logits: bool = False  # w holds the raw Eq. 6 logits (the call normalises them)

    @property
    def n_dirs(self) -> int:
        return len(mask_dirs(self.mask))

    @property
    def planes(self) -> int:
        return self.B * self.C

    def with_shape(self, **kw) -> "Workload":
        d = dict(self.__dict__)
        d.update(kw)
        return Workload(**d)


# The five workloads the hot path is measured and checked on (shapes, dtypes and
# distributions of the classification stages and diffusion latents above).
WORKLOADS = {
    "t2b_16": Workload("t2b_16", 1, 8, 16, 16, DIR_T2B, "f32", lam="uniform", u="ones",
                       w_logit_std=1.0, seed=1),
    "cls56_f32": Workload("cls56_f32", 8, 64, 56, 56, 0xF, "f32", lam="sigmoid", u="sigmoid",
                          w_logit_std=1.0, seed=2),
    "cls28_bf16_fb": Workload("cls28_bf16_fb", 32, 192, 28, 28, 0xF, "bf16", lam="uniform",
                              u="ones", w_logit_std=1.0, backward=True, seed=3),
    "lat128_bf16": Workload("lat128_bf16", 2, 640, 128, 128, 0xF, "bf16", lam="sigmoid",
                            u="sigmoid", w_logit_std=math.sqrt(2.0), seed=4),
    "lat2048_bf16": Workload("lat2048_bf16", 1, 320, 2048, 2048, 0xF, "bf16", lam="uniform",
                             u="ones", w_logit_std=1.0, seed=5),
}
# The two latent shapes with the backward as well (training at those sizes):
# same inputs, plus dy ~ N(0, 1).
WORKLOADS["lat128_bf16_fb"] = WORKLOADS["lat128_bf16"].with_shape(name="lat128_bf16_fb", backward=True)
WORKLOADS["lat2048_bf16_fb"] = WORKLOADS["lat2048_bf16"].with_shape(name="lat2048_bf16_fb", backward=True)
# The paper's own weights (Eq. 6): the logits go to the call, which normalises
# them (sigmoid, then the sum over the three neighbours) as it reads them.
WORKLOADS["cls28_bf16_lg_fb"] = WORKLOADS["cls28_bf16_fb"].with_shape(name="cls28_bf16_lg_fb", logits=True)
WORKLOADS["lat128_bf16_lg_fb"] = WORKLOADS["lat128_bf16_fb"].with_shape(name="lat128_bf16_lg_fb", logits=True)


def torch_dtype(dt: str) -> torch.dtype:
    return {"f32": torch.float32, "bf16": torch.bfloat16}[dt]


def _gen(device, seed: int, tid: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed((seed * 1_000_003 + tid * 7919 + 12345) & 0x7FFF_FFFF_FFFF)
    return g


def _draw(kind: str, shape, device, seed: int, tid: int) -> torch.Tensor:
    g = _gen(device, seed, tid)
    if kind == "normal":
        return torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if kind == "uniform":
        return torch.rand(shape, generator=g, device=device, dtype=torch.float32)
    if kind == "sigmoid":
        return torch.sigmoid(torch.randn(shape, generator=g, device=device, dtype=torch.float32))
    if kind == "ones":
        return torch.ones(shape, device=device, dtype=torch.float32)
    raise ValueError(kind)


def make_weights(wl: Workload, device="cpu") -> torch.Tensor:
    """w packed as [n][3][B][C][H][W]: per pixel and direction, softmax of 3 logits
    (or the logits themselves for a workload whose call normalises them)."""
    n = wl.n_dirs
    out = torch.empty((n, 3, wl.B, wl.C, wl.H, wl.W), device=device, dtype=torch_dtype(wl.dtype))
    for di in range(n):  # one direction at a time keeps the fp32 temporaries small
        g = _gen(device, wl.seed, 3 + 3 * di)
        logits = torch.randn((3, wl.B, wl.C, wl.H, wl.W), generator=g, device=device,
                             dtype=torch.float32)
        logits.mul_(wl.w_logit_std)
        out[di].copy_(logits if wl.logits else torch.softmax(logits, dim=0))
        del logits
    return out


def make_inputs(wl: Workload, device="cpu", with_dy: bool | None = None) -> dict:
    """All inputs of one workload as device tensors in the workload dtype."""
    shape = (wl.B, wl.C, wl.H, wl.W)
    dt = torch_dtype(wl.dtype)
    t = {
        "x": _draw(wl.x, shape, device, wl.seed, _TID_X).to(dt),
        "lam": _draw(wl.lam, shape, device, wl.seed, _TID_LAM).to(dt),
        "u": _draw(wl.u, shape, device, wl.seed, _TID_U).to(dt),
        "w": make_weights(wl, device),
    }
    if with_dy if with_dy is not None else wl.backward:
        t["dy"] = _draw("normal", shape, device, wl.seed, _TID_DY).to(dt)
    return t


def random_general(shape, n_dirs: int, device="cpu", seed: int = 0, dtype=torch.float32,
                   signed_weights: bool = True) -> dict:
    """Inputs with arbitrary (not row-stochastic, possibly negative) weights.

    The scan is defined for any w; tests use this to make sure no kernel relies
    on the weights being normalised.  Weights are scaled so that long chains
    stay bounded: |w0|+|w1|+|w2| <= 1 elementwise.
    """
    B, C, H, W = shape
    g = _gen(device, seed, 99)
    x = torch.randn(shape, generator=g, device=device)
    lam = torch.rand(shape, generator=g, device=device) * 2 - 0.5
    u = torch.randn(shape, generator=g, device=device)
    w = torch.rand((n_dirs, 3, B, C, H, W), generator=g, device=device)
    if signed_weights:
        w = w * torch.where(torch.rand(w.shape, generator=g, device=device) < 0.3, -1.0, 1.0)
    w = w / (w.abs().sum(dim=1, keepdim=True) + 0.05)
    dy = torch.randn(shape, generator=g, device=device)
    return {k: v.to(dtype) for k, v in dict(x=x, lam=lam, u=u, w=w, dy=dy).items()}


def numpy_planes(wl: Workload, planes: int, seed: int = 0) -> dict:
    """`planes` planes of the workload's distributions as float64 NumPy arrays
    (B = 1, C = planes), drawn with NumPy instead of torch.

    For CPU timing runs in worker processes that must not use torch: same
    shapes and distributions as make_inputs (the values differ, and they are
    not rounded to the workload dtype).
    """
    import numpy as np

    rng = np.random.default_rng([wl.seed, seed, planes])
    shape = (1, planes, wl.H, wl.W)

    def draw(kind):
        if kind == "normal":
            return rng.standard_normal(shape)
        if kind == "uniform":
            return rng.random(shape)
        if kind == "sigmoid":
            return 1.0 / (1.0 + np.exp(-rng.standard_normal(shape)))
        if kind == "ones":
            return np.ones(shape)
        raise ValueError(kind)

    out = {"x": draw(wl.x), "lam": draw(wl.lam), "u": draw(wl.u)}
    logits = rng.standard_normal((wl.n_dirs, 3) + shape) * wl.w_logit_std
    e = np.exp(logits - logits.max(axis=1, keepdims=True))
    out["w"] = e / e.sum(axis=1, keepdims=True)
    out["dy"] = rng.standard_normal(shape) if wl.backward else None
    return out
