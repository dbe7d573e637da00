"""Helpers for the GPU-vs-oracle parity tests."""
import numpy as np
import torch

import oracle as O

# normwise relative tolerance per output tensor: max|gpu - ref| / max|ref|
TOL = {torch.float32: 1e-5, torch.bfloat16: 2e-2}


def np64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float64).numpy()


def normwise(got, ref) -> float:
    got = np64(got) if isinstance(got, torch.Tensor) else np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = np.abs(ref).max()
    err = np.abs(got - ref).max()
    if scale == 0:
        return float(err)
    return float(err / scale)


def assert_close(got, ref, dtype, what=""):
    e = normwise(got, ref)
    assert np.isfinite(np64(got)).all(), f"{what}: non-finite output"
    assert e <= TOL[dtype], f"{what}: normwise error {e:.3e} > {TOL[dtype]:.0e}"
    return e


def oracle_fwd(inp, mask):
    return O.scan_fwd(np64(inp["x"]), np64(inp["w"]), np64(inp["lam"]), np64(inp["u"]), mask)


def oracle_bwd(inp, mask):
    return O.scan_bwd(np64(inp["dy"]), np64(inp["x"]), np64(inp["w"]), np64(inp["lam"]),
                      np64(inp["u"]), mask)
