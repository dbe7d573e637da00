"""Forward parity: HIP kernels (through the C ABI) vs the float64 oracle."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2501_12381_amd import lib as L
from paper_2501_12381_amd import ops, synth
from paper_2501_12381_amd.synth import WORKLOADS
from tests.parity_util import TOL, assert_close, np64, oracle_fwd

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
ALGOS = [L.GSPN_ALGO_AUTO, L.GSPN_ALGO_STREAM, L.GSPN_ALGO_RESIDENT, L.GSPN_ALGO_RESIDENT_GENERIC,
         L.GSPN_ALGO_TWO_PASS]
ALGO_NAMES = {0: "auto", 1: "resident", 2: "stream", 3: "resident_generic", 4: "two_pass"}
FORCED = (L.GSPN_ALGO_RESIDENT, L.GSPN_ALGO_RESIDENT_GENERIC, L.GSPN_ALGO_TWO_PASS)


def run_fwd(inp, mask, algo):
    try:
        return ops.gspn_scan_fwd(inp["x"], inp["w"], inp["lam"], inp["u"], mask, algo=algo)
    except L.GSPNError as e:
        if e.status == 7 and algo in FORCED:
            pytest.skip(f"{ALGO_NAMES[algo]} kernels do not take this shape")
        raise


def general_inputs(B, C, H, W, mask, dtype, seed):
    t = synth.random_general((B, C, H, W), ops.n_dirs(mask), device=DEV, seed=seed)
    return {k: v.to(dtype) for k, v in t.items()}


@pytest.mark.parametrize("algo", ALGOS, ids=lambda a: ALGO_NAMES[a])
@pytest.mark.parametrize("name", ["t2b_16", "cls56_f32", "cls28_bf16_fb", "lat128_bf16"])
def test_workloads_full(name, algo):
    wl = WORKLOADS[name]
    print(f"[fwd] {name} algo={ALGO_NAMES[algo]}", flush=True)
    inp = synth.make_inputs(wl, DEV, with_dy=False)
    y = run_fwd(inp, wl.mask, algo)
    torch.cuda.synchronize()
    ref = oracle_fwd(inp, wl.mask)
    assert_close(y, ref, y.dtype, name)


@pytest.mark.parametrize("algo", ALGOS, ids=lambda a: ALGO_NAMES[a])
def test_lat2048_sampled_planes(algo):
    """Full 1x320x2048x2048 bf16 forward; the oracle checks sampled planes."""
    wl = WORKLOADS["lat2048_bf16"]
    print(f"[fwd] lat2048 algo={ALGO_NAMES[algo]}", flush=True)
    inp = synth.make_inputs(wl, DEV, with_dy=False)
    y = run_fwd(inp, wl.mask, algo)
    torch.cuda.synchronize()
    assert torch.isfinite(y).all()
    for c in (0, 157, 319):
        sub = {k: (v[:, :, 0:1, c:c + 1] if k == "w" else v[0:1, c:c + 1]) for k, v in inp.items()}
        ref = oracle_fwd(sub, wl.mask)
        assert_close(y[0:1, c:c + 1], ref, y.dtype, f"plane c={c}")
    del inp, y
    torch.cuda.empty_cache()


EDGE_SHAPES = [(1, 1), (1, 7), (7, 1), (2, 2), (5, 7), (7, 5), (3, 64), (64, 3), (9, 63), (63, 9),
               (4, 65), (65, 4), (6, 127), (127, 6), (5, 128), (128, 5), (3, 129), (129, 3),
               (4, 255), (255, 4), (2, 257), (257, 2), (3, 513), (513, 3), (2, 2049), (2049, 2),
               (28, 28), (56, 56), (40, 96), (96, 40)]


@pytest.mark.parametrize("algo", ALGOS, ids=lambda a: ALGO_NAMES[a])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("shape", EDGE_SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
def test_edge_shapes_all_directions(shape, dtype, algo):
    H, W = shape
    print(f"[fwd] edge {H}x{W} {dtype} algo={ALGO_NAMES[algo]}", flush=True)
    inp = general_inputs(2, 3, H, W, 0xF, dtype, seed=H * 10007 + W)
    y = run_fwd(inp, 0xF, algo)
    torch.cuda.synchronize()
    assert_close(y, oracle_fwd(inp, 0xF), dtype, f"{H}x{W}")


# Two-pass family: single and several row bands (halo rows), odd line counts
# (middle-line rule), ragged and odd numbers of column blocks, rows spread over
# one to four waves per direction.
TWO_PASS_SHAPES = [(1, 64), (2, 64), (3, 72), (71, 136), (130, 200), (600, 64), (1000, 40),
                   (1100, 96), (520, 1032), (33, 2056)]


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("shape", TWO_PASS_SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
def test_two_pass_shapes(shape, dtype):
    H, W = shape
    print(f"[fwd] two-pass {H}x{W} {dtype}", flush=True)
    inp = general_inputs(1, 2, H, W, 0xF, dtype, seed=H * 7919 + W)
    y = run_fwd(inp, 0xF, L.GSPN_ALGO_TWO_PASS)
    torch.cuda.synchronize()
    assert_close(y, oracle_fwd(inp, 0xF), dtype, f"{H}x{W}")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("mask", list(range(1, 16)))
def test_two_pass_every_mask(mask, dtype):
    H, W = 67, 136  # odd H, three column blocks in bf16 (the last one short)
    print(f"[fwd] two-pass mask {mask} {dtype}", flush=True)
    inp = general_inputs(2, 2, H, W, mask, dtype, seed=100 + mask)
    y = run_fwd(inp, mask, L.GSPN_ALGO_TWO_PASS)
    torch.cuda.synchronize()
    assert_close(y, oracle_fwd(inp, mask), dtype, f"mask {mask}")


def test_two_pass_deterministic_and_closed_form():
    H, W = 130, 200
    inp = general_inputs(1, 3, H, W, 0xF, torch.bfloat16, seed=3)
    a = run_fwd(inp, 0xF, L.GSPN_ALGO_TWO_PASS)
    b = run_fwd(inp, 0xF, L.GSPN_ALGO_TWO_PASS)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    # middle weight 1: each direction is a cumulative sum of lam*x
    g = torch.Generator(device=DEV).manual_seed(8)
    x = torch.randn(1, 2, 600, 64, device=DEV, generator=g)
    lam = torch.rand(1, 2, 600, 64, device=DEV, generator=g)
    u = torch.ones_like(x)
    lx = np64(lam * x)
    for d, axis, rev in ((1, 2, False), (2, 2, True), (4, 3, False), (8, 3, True)):
        w = torch.zeros(1, 3, 1, 2, 600, 64, device=DEV)
        w[:, 1] = 1.0
        y = run_fwd(dict(x=x, lam=lam, u=u, w=w), d, L.GSPN_ALGO_TWO_PASS)
        ref = np.flip(np.cumsum(np.flip(lx, axis), axis), axis) if rev else np.cumsum(lx, axis)
        assert_close(y, ref, torch.float32, f"dir {d}")


@pytest.mark.parametrize("algo", ALGOS, ids=lambda a: ALGO_NAMES[a])
@pytest.mark.parametrize("mask", list(range(1, 16)))
def test_every_mask(mask, algo):
    print(f"[fwd] mask {mask} algo={ALGO_NAMES[algo]}", flush=True)
    inp = general_inputs(2, 5, 13, 21, mask, torch.float32, seed=mask)
    y = run_fwd(inp, mask, algo)
    torch.cuda.synchronize()
    assert_close(y, oracle_fwd(inp, mask), torch.float32, f"mask {mask}")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("mask", [1, 2, 4, 8, 3, 12, 5, 10, 7, 14, 15])
def test_128_planes_every_direction_set(mask, dtype):
    """128 x 128 planes (the persistent kernel that keeps lam*x on chip):
    direction subsets, including phases with one or no present direction."""
    print(f"[fwd] 128x128 mask {mask} {dtype}", flush=True)
    inp = general_inputs(1, 3, 128, 128, mask, dtype, seed=100 + mask)
    ref = oracle_fwd(inp, mask)
    for algo in (L.GSPN_ALGO_AUTO, L.GSPN_ALGO_RESIDENT):
        y = run_fwd(inp, mask, algo)
        torch.cuda.synchronize()
        assert_close(y, ref, dtype, f"mask {mask} algo {ALGO_NAMES[algo]}")


@pytest.mark.parametrize("planes", [1, 255, 257, 600])
def test_128_planes_per_workgroup_counts(planes):
    """More and fewer planes than compute units: each workgroup walks its share."""
    print(f"[fwd] 128x128 planes={planes}", flush=True)
    inp = general_inputs(1, planes, 128, 128, 0xF, torch.bfloat16, seed=planes)
    y = run_fwd(inp, 0xF, L.GSPN_ALGO_RESIDENT)
    torch.cuda.synchronize()
    assert_close(y, oracle_fwd(inp, 0xF), torch.bfloat16, f"planes {planes}")


def offset_copy(t, elems):
    """Contiguous copy of t starting `elems` elements past the start of its allocation."""
    buf = torch.empty(t.numel() + elems, dtype=t.dtype, device=t.device)
    v = buf[elems:].view(t.shape)
    v.copy_(t)
    return v


@pytest.mark.parametrize("shift", [1, 2, 4])
@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32], ids=["bf16", "f32"])
@pytest.mark.parametrize("S", [16, 28, 56, 128])
def test_size_specialised_kernels_unaligned_u_y(S, dtype, shift):
    """u and y only element-aligned (the ABI's requirement): the size-specialised
    kernels' epilogues take u and y as vectors only when their alignment allows,
    and 128 x 128 leaves the persistent kernel (it needs 16-byte u and y).
    Three planes: a partly filled last group for the two-plane-per-wave sizes."""
    print(f"[fwd] unaligned u/y S={S} {dtype} shift={shift}", flush=True)
    inp = general_inputs(1, 3, S, S, 0xF, dtype, seed=700 + S + shift)
    inp["u"] = offset_copy(inp["u"], shift)
    ref = oracle_fwd(inp, 0xF)
    for algo in (L.GSPN_ALGO_AUTO, L.GSPN_ALGO_RESIDENT):
        y = offset_copy(torch.zeros_like(inp["x"]), shift + 1)
        out = ops.gspn_scan_fwd(inp["x"], inp["w"], inp["lam"], inp["u"], 0xF, algo=algo, y=y)
        torch.cuda.synchronize()
        assert out.data_ptr() == y.data_ptr()
        assert_close(out, ref, dtype, f"S={S} shift={shift} algo={ALGO_NAMES[algo]}")


@pytest.mark.parametrize("algo", ALGOS, ids=lambda a: ALGO_NAMES[a])
def test_single_direction_closed_form(algo):
    """Middle weight 1, others 0: each direction is a cumulative sum of lam*x."""
    H, W = 37, 45
    g = torch.Generator(device=DEV).manual_seed(5)
    x = torch.randn(1, 4, H, W, device=DEV, generator=g)
    lam = torch.rand(1, 4, H, W, device=DEV, generator=g)
    u = torch.ones_like(x)
    lx = np64(lam * x)
    for d, axis, rev in ((1, 2, False), (2, 2, True), (4, 3, False), (8, 3, True)):
        w = torch.zeros(1, 3, 1, 4, H, W, device=DEV)
        w[:, 1] = 1.0
        y = run_fwd(dict(x=x, lam=lam, u=u, w=w), d, algo)
        ref = np.flip(np.cumsum(np.flip(lx, axis), axis), axis) if rev else np.cumsum(lx, axis)
        assert_close(y, ref, torch.float32, f"dir {d}")


@pytest.mark.parametrize("algo", ALGOS, ids=lambda a: ALGO_NAMES[a])
def test_deterministic(algo):
    wl = WORKLOADS["cls28_bf16_fb"].with_shape(B=4)
    inp = synth.make_inputs(wl, DEV, with_dy=False)
    a = run_fwd(inp, wl.mask, algo)
    b = run_fwd(inp, wl.mask, algo)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_long_chain_fp32_stays_bounded():
    """Row-stochastic weights over 4096 lines: no growth, oracle parity at fp32."""
    wl = synth.Workload("long", 1, 4, 4096, 24, 0xF, "f32", seed=11)
    inp = synth.make_inputs(wl, DEV, with_dy=False)
    y = run_fwd(inp, wl.mask, L.GSPN_ALGO_AUTO)
    torch.cuda.synchronize()
    ref = oracle_fwd(inp, wl.mask)
    # fp32 error grows at most linearly with the chain length; 4096 lines stay within 2e-5
    e = np.abs(np64(y) - ref).max() / np.abs(ref).max()
    assert e < 2e-5, e


def test_cpu_tensors_rejected():
    x = torch.zeros(1, 1, 4, 4)
    with pytest.raises(RuntimeError, match="GPU only"):
        ops.gspn_scan_fwd(x, torch.zeros(1, 3, 1, 1, 4, 4), x, x, 1)


def test_errors_surface_as_exceptions():
    x = torch.zeros(1, 1, 4, 4, device=DEV)
    with pytest.raises(ValueError):
        ops.gspn_scan_fwd(x, torch.zeros(2, 3, 1, 1, 4, 4, device=DEV), x, x, 1)
    big = torch.zeros(1, 1, 1, L.GSPN_MAX_LINE + 1, device=DEV)
    with pytest.raises(L.GSPNError) as ei:
        ops.gspn_scan_fwd(big, torch.zeros(1, 3, 1, 1, 1, L.GSPN_MAX_LINE + 1, device=DEV), big,
                          big, 1)
    assert ei.value.status == 7


def test_copy_calibration_kernel():
    src = torch.randint(0, 255, (3 * 1024 * 1024 + 37,), dtype=torch.uint8, device=DEV)
    dst = torch.zeros_like(src)
    ops.gspn_copy_calibration(src[:-5], dst[:-5])  # 16-byte aligned starts, ragged tail
    torch.cuda.synchronize()
    assert torch.equal(dst[:-5], src[:-5]) and not dst[-5:].any()


def test_4096_planes_forward_sampled():
    """The longest lines the library takes: 2 planes of 4096 x 4096 bf16
    (two-pass kernels), one plane checked against the oracle in full."""
    wl = synth.Workload("lat4096", 1, 2, 4096, 4096, 0xF, "bf16", lam="uniform", u="ones", seed=9)
    print("[fwd] 4096x4096 x 2 planes", flush=True)
    inp = synth.make_inputs(wl, DEV, with_dy=False)
    y = run_fwd(inp, wl.mask, L.GSPN_ALGO_AUTO)
    torch.cuda.synchronize()
    assert torch.isfinite(y).all()
    sub = {k: (v[:, :, 0:1, 1:2] if k == "w" else v[0:1, 1:2]) for k, v in inp.items()}
    assert_close(y[0:1, 1:2], oracle_fwd(sub, wl.mask), y.dtype, "4096 plane 1")
