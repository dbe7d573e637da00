"""Two-pass backward against the float64 oracle (GPU, through the C ABI).

The horizontal directions run on the column-block kernels (a recompute of h,
then the adjoint over blocks in reverse scan order, each workgroup owning a
band of rows with K halo rows towards each neighbouring band); the vertical
ones on the vertical recompute and the paired vertical adjoint.  Cases: one band and several (halo rows crossing band and
plane edges), ragged last column blocks, every direction set with a
horizontal direction, several planes, local GSPN groups whose boundaries fall
inside a column block, row counts around the band-count transitions, and
sampled planes of the full 2048 x 2048 workload."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2501_12381_amd import lib as L
from paper_2501_12381_amd import ops, synth
from paper_2501_12381_amd.synth import WORKLOADS
from tests.parity_util import assert_close, np64, oracle_bwd, oracle_fwd

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
TWO_PASS = L.GSPN_ALGO_TWO_PASS


def inputs(B, C, H, W, mask, dtype, seed):
    t = synth.random_general((B, C, H, W), ops.n_dirs(mask), device=DEV, seed=seed)
    return {k: v.to(dtype) for k, v in t.items()}


def check(inp, mask, dtype, what, **opt):
    dx, dw, dlam, du = ops.gspn_scan_bwd(inp["dy"], inp["x"], inp["w"], inp["lam"], inp["u"], mask,
                                         algo=TWO_PASS, **opt)
    torch.cuda.synchronize()
    a = {k: np64(v) for k, v in inp.items()}
    rdx, rdw, rdlam, rdu = O.scan_bwd(a["dy"], a["x"], a["w"], a["lam"], a["u"], mask,
                                      group_h=opt.get("group_h", 0), group_w=opt.get("group_w", 0))
    assert_close(dx, rdx, dtype, f"{what} dx")
    assert_close(dlam, rdlam, dtype, f"{what} dlam")
    assert_close(du, rdu, dtype, f"{what} du")
    for n in range(rdw.shape[0]):
        for k in range(3):
            assert_close(dw[n, k], rdw[n, k], dtype, f"{what} dw[{n}][{k}]")


# (H, W): 1 row; one band (H <= 512); several bands (H > 512, halo rows);
# W a whole number of column blocks or a ragged last block (window shifted
# back), for both element sizes (blocks of 64 bf16 / 32 fp32 columns)
SHAPES = [(1, 64), (5, 72), (63, 64), (64, 128), (65, 136), (130, 200), (511, 64), (512, 96),
          (513, 64), (700, 136), (1030, 72)]


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
def test_two_pass_bwd_shapes(shape, dtype):
    H, W = shape
    print(f"[bwd2] {H}x{W} {dtype}", flush=True)
    planes = 3 if H * W <= 200 * 200 else 1
    inp = inputs(1, planes, H, W, 0xF, dtype, seed=H * 7919 + W)
    check(inp, 0xF, dtype, f"{H}x{W}")


@pytest.mark.parametrize("mask", [4, 8, 12, 5, 6, 9, 10, 7, 11, 13, 14, 15])
def test_two_pass_bwd_masks(mask):
    print(f"[bwd2] mask {mask}", flush=True)
    inp = inputs(2, 2, 600, 136, mask, torch.float32, seed=50 + mask)
    check(inp, mask, torch.float32, f"mask {mask}")


def test_two_pass_bwd_vertical_only_is_refused():
    """Without a horizontal direction the forced two-pass backward has nothing
    of its own to run and refuses; AUTO takes another family."""
    inp = inputs(1, 1, 600, 64, 3, torch.float32, seed=3)
    with pytest.raises(L.GSPNError) as e:
        ops.gspn_scan_bwd(inp["dy"], inp["x"], inp["w"], inp["lam"], inp["u"], 3, algo=TWO_PASS)
    assert e.value.status == 7


# (H, W, group_h, group_w): group boundaries inside a column block, groups of
# one column, groups longer than a block, ragged last groups
GROUP_CASES = [(130, 200, 33, 64), (600, 136, 100, 7), (520, 200, 0, 50), (70, 64, 9, 1), (40, 520, 5, 300)]


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("case", GROUP_CASES, ids=lambda c: "x".join(map(str, c)))
def test_two_pass_bwd_groups(case, dtype):
    H, W, gh, gw = case
    print(f"[bwd2] groups {case} {dtype}", flush=True)
    inp = inputs(1, 2, H, W, 0xF, dtype, seed=H + W * 3 + gh + gw)
    check(inp, 0xF, dtype, f"groups {case}", group_h=gh, group_w=gw)


# Row counts around the band-count transitions of the horizontal kernels
# (every band takes 512 lanes; the first and last keep K more rows than the
# others, K = 64 columns for bf16 and 32 for fp32): bf16 changes from two to
# three bands between 896 and 897 rows, fp32 between 960 and 961.
BAND_EDGE_H = [896, 897, 960, 961, 1281]


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("H", BAND_EDGE_H)
def test_two_pass_band_transitions(H, dtype):
    print(f"[bwd2] band transition {H} rows {dtype}", flush=True)
    inp = inputs(1, 1, H, 64, 0xF, dtype, seed=H + 17)
    y = ops.gspn_scan_fwd(inp["x"], inp["w"], inp["lam"], inp["u"], 0xF, algo=TWO_PASS)
    torch.cuda.synchronize()
    assert_close(y, oracle_fwd(inp, 0xF), dtype, f"forward, {H} rows")
    check(inp, 0xF, dtype, f"backward, {H} rows")


def test_two_pass_bwd_deterministic():
    """Every addition happens in a fixed order: two runs agree bit for bit."""
    inp = inputs(1, 4, 700, 200, 0xF, torch.bfloat16, seed=11)
    a = ops.gspn_scan_bwd(inp["dy"], inp["x"], inp["w"], inp["lam"], inp["u"], 0xF, algo=TWO_PASS)
    b = ops.gspn_scan_bwd(inp["dy"], inp["x"], inp["w"], inp["lam"], inp["u"], 0xF, algo=TWO_PASS)
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_lat2048_backward_sampled():
    """Backward of the full 1 x 320 x 2048 x 2048 bf16 workload (AUTO picks
    the two-pass family); the oracle checks sampled planes."""
    wl = WORKLOADS["lat2048_bf16_fb"]
    print("[bwd2] lat2048 fwd+bwd workload", flush=True)
    inp = synth.make_inputs(wl, DEV)
    got = ops.gspn_scan_bwd(inp["dy"], inp["x"], inp["w"], inp["lam"], inp["u"], wl.mask)
    torch.cuda.synchronize()
    for g in got:
        assert torch.isfinite(g).all()
    for c in (0, 319):
        sub = {k: (v[:, :, 0:1, c:c + 1] if k == "w" else v[0:1, c:c + 1]) for k, v in inp.items()}
        sel = [g[0:1, c:c + 1] if i != 1 else g[:, :, 0:1, c:c + 1] for i, g in enumerate(got)]
        ref = oracle_bwd(sub, wl.mask)
        for name, x, r in zip(("dx", "dw", "dlam", "du"), sel, ref):
            if name == "dw":
                for n in range(r.shape[0]):
                    for k in range(3):
                        assert_close(x[n, k], r[n, k], torch.bfloat16, f"plane {c} dw[{n}][{k}]")
            else:
                assert_close(x, r, torch.bfloat16, f"plane {c} {name}")
    del inp, got
    torch.cuda.empty_cache()
