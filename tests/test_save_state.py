"""GSPN_FLAG_SAVE_STATE on the GPU, through the C ABI: the two-pass forward
keeps every direction's h and sum_d h_d in its workspace, and the backward
reads them there instead of recomputing the forward scan (Alg. 2 takes the
forward's states as an input).

Checked against the float64 oracle and against the recomputing backward on
the same inputs: dx, dw and dlam must be the same bits (the same kernels add
the same values), du agrees to rounding (the directions are added in the
forward's order).  Cases: every direction set with a horizontal direction,
one and several row bands, ragged column blocks, groups, Eq. 6 logits, both
element sizes; problems the flag does not apply to (no horizontal direction,
planes kept on chip) give the results of a plain call; the autograd path; and
sampled planes of the full 2048 x 2048 workload."""
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


def inputs(B, C, H, W, mask, dtype, seed, logits=False):
    t = synth.random_general((B, C, H, W), ops.n_dirs(mask), device=DEV, seed=seed)
    if logits:
        g = torch.Generator(device="cpu").manual_seed(seed + 1)
        t["w"] = (2.0 * torch.randn(t["w"].shape, generator=g)).to(DEV)
    return {k: v.to(dtype) for k, v in t.items()}


def run_pair(inp, mask, algo, **opt):
    """(y, grads) of a plain forward + backward and of a saved-state pair."""
    x, w, lam, u, dy = inp["x"], inp["w"], inp["lam"], inp["u"], inp["dy"]
    y0 = ops.gspn_scan_fwd(x, w, lam, u, mask, algo=algo, **opt)
    g0 = ops.gspn_scan_bwd(dy, x, w, lam, u, mask, algo=algo, **opt)
    ws = ops.scan_workspace(x, mask, algo=algo, save_state=True, **opt)
    ws.fill_(0xFF)  # NaN patterns: a state the forward did not write shows up
    y1 = ops.gspn_scan_fwd(x, w, lam, u, mask, algo=algo, workspace=ws, save_state=True, **opt)
    g1 = ops.gspn_scan_bwd(dy, x, w, lam, u, mask, algo=algo, workspace=ws, save_state=True, **opt)
    torch.cuda.synchronize()
    return (y0, g0), (y1, g1)


def compare(plain, saved, inp, mask, dtype, what, **opt):
    (y0, (dx0, dw0, dl0, du0)), (y1, (dx1, dw1, dl1, du1)) = plain, saved
    assert torch.equal(y0, y1), f"{what}: y"
    assert torch.equal(dx0, dx1), f"{what}: dx"
    assert torch.equal(dw0, dw1), f"{what}: dw"
    assert torch.equal(dl0, dl1), f"{what}: dlam"
    a = {k: np64(v) for k, v in inp.items()}
    kw = dict(group_h=opt.get("group_h", 0), group_w=opt.get("group_w", 0), logits=opt.get("logits", False))
    ref = O.scan_bwd(a["dy"], a["x"], a["w"], a["lam"], a["u"], mask, **kw)
    assert_close(du1, ref[3], dtype, f"{what}: du")
    assert_close(du1, np64(du0), dtype, f"{what}: du against the recomputing backward")
    assert_close(dx1, ref[0], dtype, f"{what}: dx")
    assert_close(dl1, ref[2], dtype, f"{what}: dlam")
    for n in range(ref[1].shape[0]):
        for k in range(3):
            assert_close(dw1[n, k], ref[1][n, k], dtype, f"{what}: dw[{n}][{k}]")


# direction sets with a horizontal direction: one or two of each kind
MASKS = [4, 8, 12, 5, 6, 9, 10, 7, 13, 14, 15]


@pytest.mark.parametrize("mask", MASKS)
def test_saved_state_every_mask(mask):
    print(f"[save] mask {mask}", flush=True)
    inp = inputs(2, 2, 600, 136, mask, torch.float32, seed=300 + mask)
    plain, saved = run_pair(inp, mask, TWO_PASS)
    compare(plain, saved, inp, mask, torch.float32, f"mask {mask}")


# one band, several bands, ragged column blocks, several planes
SHAPES = [(1, 64), (63, 200), (130, 200), (513, 64), (1030, 72)]


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
def test_saved_state_shapes(shape, dtype):
    H, W = shape
    print(f"[save] {H}x{W} {dtype}", flush=True)
    inp = inputs(1, 3 if H * W < 40000 else 1, H, W, 0xF, dtype, seed=H * 31 + W)
    plain, saved = run_pair(inp, 0xF, TWO_PASS)
    compare(plain, saved, inp, 0xF, dtype, f"{H}x{W}")


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
def test_saved_state_groups_and_logits(dtype):
    print(f"[save] groups and logits {dtype}", flush=True)
    inp = inputs(1, 2, 600, 136, 0xF, dtype, seed=77, logits=True)
    opt = dict(group_h=100, group_w=7, logits=True)
    plain, saved = run_pair(inp, 0xF, TWO_PASS, **opt)
    compare(plain, saved, inp, 0xF, dtype, "groups and logits", **opt)


@pytest.mark.parametrize("case", [(3, 600, 136), (0xF, 28, 28), (0xF, 128, 128)],
                         ids=["vertical-only", "28x28", "128x128"])
def test_saved_state_ignored_elsewhere(case):
    """Without a horizontal direction, or with planes kept on chip (AUTO), the
    flag changes nothing: the results are those of plain calls."""
    mask, H, W = case
    print(f"[save] ignored: mask {mask} {H}x{W}", flush=True)
    inp = inputs(2, 2, H, W, mask, torch.bfloat16, seed=H + mask)
    (y0, g0), (y1, g1) = run_pair(inp, mask, L.GSPN_ALGO_AUTO)
    assert torch.equal(y0, y1)
    for a, b in zip(g0, g1):
        assert torch.equal(a, b)


def test_saved_state_autograd():
    """The autograd wrapper carries the workspace from forward to backward."""
    print("[save] autograd", flush=True)
    inp = inputs(1, 2, 700, 136, 0xF, torch.float32, seed=5)
    leaves = {k: inp[k].clone().requires_grad_(True) for k in ("x", "w", "lam", "u")}
    y = ops.gspn_scan(leaves["x"], leaves["w"], leaves["lam"], leaves["u"], 0xF, algo=TWO_PASS, save_state=True)
    y.backward(inp["dy"])
    torch.cuda.synchronize()
    ref = oracle_bwd(inp, 0xF)
    assert_close(y, oracle_fwd(inp, 0xF), torch.float32, "y")
    for name, r in zip(("x", "w", "lam", "u"), ref):
        got = leaves[name].grad
        if name == "w":
            for n in range(r.shape[0]):
                for k in range(3):
                    assert_close(got[n, k], r[n, k], torch.float32, f"dw[{n}][{k}]")
        else:
            assert_close(got, r, torch.float32, f"d{name}")


def test_lat2048_saved_state_sampled():
    """Forward + backward of the full 1 x 320 x 2048 x 2048 bf16 workload with
    the state kept; the oracle checks sampled planes."""
    wl = WORKLOADS["lat2048_bf16_fb"]
    print("[save] lat2048 fwd+bwd with the state kept", flush=True)
    inp = synth.make_inputs(wl, DEV, with_dy=True)
    x, w, lam, u, dy = inp["x"], inp["w"], inp["lam"], inp["u"], inp["dy"]
    ws = ops.scan_workspace(x, wl.mask, save_state=True)
    y = ops.gspn_scan_fwd(x, w, lam, u, wl.mask, workspace=ws, save_state=True)
    got = ops.gspn_scan_bwd(dy, x, w, lam, u, wl.mask, workspace=ws, save_state=True)
    torch.cuda.synchronize()
    for c in (0, 319):
        sub = {k: (v[:, :, 0:1, c:c + 1] if k == "w" else v[0:1, c:c + 1]) for k, v in inp.items()}
        assert_close(y[0:1, c:c + 1], oracle_fwd(sub, wl.mask), torch.bfloat16, f"plane {c} y")
        sel = [g[0:1, c:c + 1] if i != 1 else g[:, :, 0:1, c:c + 1] for i, g in enumerate(got)]
        ref = oracle_bwd(sub, wl.mask)
        for name, gt, r in zip(("dx", "dw", "dlam", "du"), sel, ref):
            if name == "dw":
                for n in range(r.shape[0]):
                    for k in range(3):
                        assert_close(gt[n, k], r[n, k], torch.bfloat16, f"plane {c} dw[{n}][{k}]")
            else:
                assert_close(gt, r, torch.bfloat16, f"plane {c} {name}")
    del inp, x, w, lam, u, dy, ws, y, got
    torch.cuda.empty_cache()
