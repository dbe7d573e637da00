"""Backward parity: HIP adjoint scan (through the C ABI) vs the float64 oracle,
and vs central finite differences of the oracle's loss."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2501_12381_amd import lib as L
from paper_2501_12381_amd import ops, synth
from paper_2501_12381_amd.synth import WORKLOADS
from tests.parity_util import assert_close, np64, oracle_bwd

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
ALGOS = [L.GSPN_ALGO_AUTO, L.GSPN_ALGO_STREAM, L.GSPN_ALGO_RESIDENT, L.GSPN_ALGO_RESIDENT_GENERIC,
         L.GSPN_ALGO_TWO_PASS]
ALGO_NAMES = {0: "auto", 1: "resident", 2: "stream", 3: "resident_generic", 4: "two_pass"}


def run_bwd(inp, mask, algo):
    try:
        return ops.gspn_scan_bwd(inp["dy"], inp["x"], inp["w"], inp["lam"], inp["u"], mask, algo=algo)
    except L.GSPNError as e:
        if e.status == 7 and algo in (L.GSPN_ALGO_RESIDENT, L.GSPN_ALGO_RESIDENT_GENERIC, L.GSPN_ALGO_TWO_PASS):
            pytest.skip("this kernel family does not take this shape")
        raise


def check_grads(got, ref, dtype, what):
    dx, dw, dlam, du = got
    rdx, rdw, rdlam, rdu = ref
    assert_close(dx, rdx, dtype, f"{what} dx")
    assert_close(dlam, rdlam, dtype, f"{what} dlam")
    assert_close(du, rdu, dtype, f"{what} du")
    for n in range(rdw.shape[0]):
        for k in range(3):
            assert_close(dw[n, k], rdw[n, k], dtype, f"{what} dw[{n}][{k}]")


@pytest.mark.parametrize("algo", ALGOS, ids=lambda a: ALGO_NAMES[a])
def test_cls28_fwd_bwd_full(algo):
    """4-direction forward+backward, bf16, 32x192x28x28."""
    wl = WORKLOADS["cls28_bf16_fb"]
    print(f"[bwd] cls28 full algo={ALGO_NAMES[algo]}", flush=True)
    inp = synth.make_inputs(wl, DEV)
    got = run_bwd(inp, wl.mask, algo)
    torch.cuda.synchronize()
    check_grads(got, oracle_bwd(inp, wl.mask), torch.bfloat16, "cls28")


SHAPES = [(1, 1), (1, 6), (6, 1), (2, 3), (5, 7), (7, 5), (16, 16), (28, 28), (32, 32), (9, 65), (65, 9),
          (3, 130), (130, 3), (4, 300), (300, 4), (2, 1030), (1030, 2), (56, 56)]


@pytest.mark.parametrize("algo", ALGOS, ids=lambda a: ALGO_NAMES[a])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
def test_bwd_shapes(shape, dtype, algo):
    H, W = shape
    print(f"[bwd] {H}x{W} {dtype} algo={ALGO_NAMES[algo]}", flush=True)
    t = synth.random_general((2, 3, H, W), 4, device=DEV, seed=H * 31 + W)
    inp = {k: v.to(dtype) for k, v in t.items()}
    got = run_bwd(inp, 0xF, algo)
    torch.cuda.synchronize()
    check_grads(got, oracle_bwd(inp, 0xF), dtype, f"{H}x{W}")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("S", [16, 28, 32])
@pytest.mark.parametrize("mask", [1, 2, 4, 8, 3, 12, 5, 15])
def test_bwd_small_square_masks(mask, S, dtype):
    """Small square planes (the LDS-staged kernel under AUTO): every direction
    subset, an odd number of planes (a partial last group)."""
    print(f"[bwd] square {S} mask {mask} {dtype}", flush=True)
    t = synth.random_general((1, 3, S, S), ops.n_dirs(mask), device=DEV, seed=1000 + 16 * S + mask)
    t = {k: v.to(dtype) for k, v in t.items()}
    for algo in (L.GSPN_ALGO_AUTO, L.GSPN_ALGO_RESIDENT_GENERIC):
        got = run_bwd(t, mask, algo)
        torch.cuda.synchronize()
        check_grads(got, oracle_bwd(t, mask), dtype, f"S={S} mask {mask} {ALGO_NAMES[algo]}")


@pytest.mark.parametrize("algo", ALGOS, ids=lambda a: ALGO_NAMES[a])
@pytest.mark.parametrize("mask", [1, 2, 4, 8, 3, 12, 5, 10, 7, 14, 15])
def test_bwd_masks(mask, algo):
    t = synth.random_general((1, 4, 11, 19), ops.n_dirs(mask), device=DEV, seed=100 + mask)
    got = run_bwd(t, mask, algo)
    torch.cuda.synchronize()
    check_grads(got, oracle_bwd(t, mask), torch.float32, f"mask {mask}")


@pytest.mark.parametrize("algo", ALGOS, ids=lambda a: ALGO_NAMES[a])
def test_bwd_matches_oracle_finite_differences(algo):
    """fp32 GPU gradients vs central differences of the oracle's float64 loss <dy, y>."""
    H, W, mask = 4, 5, 0xF
    t = synth.random_general((1, 2, H, W), 4, device=DEV, seed=7)
    dx, dw, dlam, du = (np64(v) for v in run_bwd(t, mask, algo))
    a = {k: np64(v) for k, v in t.items()}
    loss = lambda x, w, lam, u: float((a["dy"] * O.scan_fwd(x, w, lam, u, mask)).sum())
    eps = 1e-6
    rng = np.random.default_rng(3)
    args = [a["x"], a["w"], a["lam"], a["u"]]
    for which, grad in enumerate((dx, dw, dlam, du)):
        for _ in range(4):
            v = rng.standard_normal(args[which].shape)
            p, m = list(args), list(args)
            p[which] = args[which] + eps * v
            m[which] = args[which] - eps * v
            fd = (loss(*p) - loss(*m)) / (2 * eps)
            an = float((grad * v).sum())
            assert abs(fd - an) <= 2e-5 * max(1.0, abs(fd)), (which, fd, an)


@pytest.mark.parametrize("algo", ALGOS, ids=lambda a: ALGO_NAMES[a])
def test_bwd_deterministic(algo):
    wl = WORKLOADS["cls28_bf16_fb"].with_shape(B=2)
    inp = synth.make_inputs(wl, DEV)
    a = run_bwd(inp, wl.mask, algo)
    b = run_bwd(inp, wl.mask, algo)
    torch.cuda.synchronize()
    for u, v in zip(a, b):
        assert torch.equal(u.view(torch.int16), v.view(torch.int16))


def offset_copy(t, elems):
    """Contiguous copy of t starting `elems` elements past the start of its allocation."""
    buf = torch.empty(t.numel() + elems, dtype=t.dtype, device=t.device)
    v = buf[elems:].view(t.shape)
    v.copy_(t)
    return v


@pytest.mark.parametrize("shift", [1, 2, 4])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("S", [16, 28, 32, 56, 64])
def test_bwd_element_aligned_views(S, dtype, shift):
    """Every input and output only element-aligned, workspace sized by AUTO:
    the call must succeed (the resident kernels' vector accesses need 16-byte
    alignment, so AUTO runs another family) and match the oracle."""
    print(f"[bwd] element-aligned views S={S} {dtype} shift={shift}", flush=True)
    t = synth.random_general((1, 3, S, S), 4, device=DEV, seed=900 + S + shift)
    inp = {k: offset_copy(v.to(dtype), shift) for k, v in t.items()}
    outs = (offset_copy(torch.zeros_like(inp["x"]), shift + 1),
            offset_copy(torch.zeros_like(inp["w"]), shift + 1),
            offset_copy(torch.zeros_like(inp["x"]), shift + 2),
            offset_copy(torch.zeros_like(inp["x"]), shift + 3))
    got = ops.gspn_scan_bwd(inp["dy"], inp["x"], inp["w"], inp["lam"], inp["u"], 0xF, out=outs)
    torch.cuda.synchronize()
    assert all(g.data_ptr() == o.data_ptr() for g, o in zip(got, outs))
    check_grads(got, oracle_bwd(inp, 0xF), dtype, f"S={S} shift={shift}")


def test_autograd_function_matches_oracle():
    wl = WORKLOADS["cls28_bf16_fb"].with_shape(B=1, C=8)
    inp = synth.make_inputs(wl, DEV)
    leaves = {k: inp[k].clone().requires_grad_(True) for k in ("x", "w", "lam", "u")}
    y = ops.gspn_scan(leaves["x"], leaves["w"], leaves["lam"], leaves["u"], wl.mask)
    (y.float() * inp["dy"].float()).sum().backward()
    ref = oracle_bwd(inp, wl.mask)
    got = (leaves["x"].grad, leaves["w"].grad, leaves["lam"].grad, leaves["u"].grad)
    check_grads(got, ref, torch.bfloat16, "autograd")


def test_4096_planes_backward_sampled():
    """Backward at 4096 x 4096 (2 planes, bf16), one plane against the oracle."""
    wl = synth.Workload("lat4096fb", 1, 2, 4096, 4096, 0xF, "bf16", lam="uniform", u="ones",
                        backward=True, seed=9)
    print("[bwd] 4096x4096 x 2 planes", flush=True)
    inp = synth.make_inputs(wl, DEV)
    got = run_bwd(inp, wl.mask, L.GSPN_ALGO_AUTO)
    torch.cuda.synchronize()
    sub = {k: (v[:, :, 0:1, 0:1] if k == "w" else v[0:1, 0:1]) for k, v in inp.items()}
    sel = [g[0:1, 0:1] if i != 1 else g[:, :, 0:1, 0:1] for i, g in enumerate(got)]
    check_grads(sel, oracle_bwd(sub, wl.mask), torch.bfloat16, "4096 plane 0")


@pytest.mark.parametrize("name", ["lat128_bf16_fb"])
def test_latent_backward_sampled(name):
    """Backward on the 2 x 640 x 128 x 128 latent workload, sampled planes."""
    wl = WORKLOADS[name]
    print(f"[bwd] {name}", flush=True)
    inp = synth.make_inputs(wl, DEV)
    got = run_bwd(inp, wl.mask, L.GSPN_ALGO_AUTO)
    torch.cuda.synchronize()
    for b, c in ((0, 0), (1, 321), (1, 639)):
        sub = {k: (v[:, :, b:b + 1, c:c + 1] if k == "w" else v[b:b + 1, c:c + 1]) for k, v in inp.items()}
        sel = [g[b:b + 1, c:c + 1] if i != 1 else g[:, :, b:b + 1, c:c + 1] for i, g in enumerate(got)]
        check_grads(sel, oracle_bwd(sub, wl.mask), torch.bfloat16, f"plane ({b},{c})")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("mask", [1, 2, 4, 8, 3, 12, 5, 10, 7, 14, 15])
def test_bwd_128_every_direction_set(mask, dtype):
    """128 x 128 planes (the persistent backward kernel): direction subsets,
    through AUTO and the forced resident family."""
    print(f"[bwd] 128x128 mask {mask} {dtype}", flush=True)
    t = synth.random_general((1, 3, 128, 128), ops.n_dirs(mask), device=DEV, seed=500 + mask)
    t = {k: v.to(dtype) for k, v in t.items()}
    ref = oracle_bwd(t, mask)
    for algo in (L.GSPN_ALGO_AUTO, L.GSPN_ALGO_RESIDENT):
        got = run_bwd(t, mask, algo)
        torch.cuda.synchronize()
        check_grads(got, ref, dtype, f"128 mask {mask} {ALGO_NAMES[algo]}")


@pytest.mark.parametrize("planes", [1, 257, 600])
def test_bwd_128_planes_per_workgroup_counts(planes):
    """More and fewer planes than compute units: each workgroup walks its share."""
    print(f"[bwd] 128x128 planes={planes}", flush=True)
    t = synth.random_general((1, planes, 128, 128), 4, device=DEV, seed=planes)
    t = {k: v.to(torch.bfloat16) for k, v in t.items()}
    got = run_bwd(t, 0xF, L.GSPN_ALGO_AUTO)
    torch.cuda.synchronize()
    idx = sorted({0, planes // 2, planes - 1})
    for c in idx:
        sub = {k: (v[:, :, :, c:c + 1] if k == "w" else v[:, c:c + 1]) for k, v in t.items()}
        sel = [g[:, c:c + 1] if i != 1 else g[:, :, :, c:c + 1] for i, g in enumerate(got)]
        check_grads(sel, oracle_bwd(sub, 0xF), torch.bfloat16, f"plane {c} of {planes}")
    a = run_bwd(t, 0xF, L.GSPN_ALGO_AUTO)
    torch.cuda.synchronize()
    for u, v in zip(a, got):
        assert torch.equal(u.view(torch.int16), v.view(torch.int16))
