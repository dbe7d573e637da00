"""Parity of the scan options against the float64 oracle (GPU, through the C ABI):
local GSPN groups (Sec. 4.1, Alg. 1's kNItems groups), Eq. 6 logit
normalisation with and without edge renormalisation, and per-direction
lam / u / y maps.  Every kernel family that takes an option is run on it
(families that do not take it refuse with GSPN_ERR_UNSUPPORTED and are
skipped)."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2501_12381_amd import lib as L
from paper_2501_12381_amd import ops, synth
from tests.parity_util import assert_close, np64

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
ALGO_NAMES = {0: "auto", 1: "resident", 2: "stream", 3: "resident_generic", 4: "two_pass"}
FWD_ALGOS = [0, 1, 2, 3, 4]
BWD_ALGOS = [0, 1, 2, 3, 4]


def inputs(B, C, H, W, mask, dtype, seed, lam_pd=False, u_pd=False, y_pd=False, logits=False):
    n = ops.n_dirs(mask)
    t = synth.random_general((B, C, H, W), n, device=DEV, seed=seed)
    g = torch.Generator(device=DEV).manual_seed(seed + 17)
    if logits:
        t["w"] = torch.randn(t["w"].shape, generator=g, device=DEV) * 1.5
    if lam_pd:
        t["lam"] = torch.rand((n, B, C, H, W), generator=g, device=DEV) * 2 - 0.5
    if u_pd:
        t["u"] = torch.randn((n, B, C, H, W), generator=g, device=DEV)
    if y_pd:
        t["dy"] = torch.randn((n, B, C, H, W), generator=g, device=DEV)
    return {k: v.to(dtype) for k, v in t.items()}


def run(fn, algo, **kw):
    try:
        return fn(algo=algo, **kw)
    except L.GSPNError as e:
        if e.status == 7 and algo != 0:
            pytest.skip(f"{ALGO_NAMES[algo]} kernels do not take this problem")
        raise


def fwd(inp, mask, algo, **opt):
    return run(lambda **kw: ops.gspn_scan_fwd(inp["x"], inp["w"], inp["lam"], inp["u"], mask, **kw),
               algo, **opt)


def bwd(inp, mask, algo, **opt):
    return run(lambda **kw: ops.gspn_scan_bwd(inp["dy"], inp["x"], inp["w"], inp["lam"], inp["u"], mask,
                                              **kw), algo, **opt)


def oracle_kw(opt):
    return dict(group_h=opt.get("group_h", 0), group_w=opt.get("group_w", 0),
                logits=opt.get("logits", False), renorm=opt.get("renorm", False),
                lam_per_dir=opt.get("lam_per_dir", False), u_per_dir=opt.get("u_per_dir", False),
                y_per_dir=opt.get("y_per_dir", False))


def check_fwd(inp, mask, algo, dtype, what, **opt):
    y = fwd(inp, mask, algo, **opt)
    torch.cuda.synchronize()
    a = {k: np64(v) for k, v in inp.items()}
    ref = O.scan_fwd(a["x"], a["w"], a["lam"], a["u"], mask, **oracle_kw(opt))
    assert_close(y, ref, dtype, what)


def check_bwd(inp, mask, algo, dtype, what, **opt):
    dx, dw, dlam, du = bwd(inp, mask, algo, **opt)
    torch.cuda.synchronize()
    a = {k: np64(v) for k, v in inp.items()}
    rdx, rdw, rdlam, rdu = O.scan_bwd(a["dy"], a["x"], a["w"], a["lam"], a["u"], mask, **oracle_kw(opt))
    assert_close(dx, rdx, dtype, f"{what} dx")
    for name, got, ref in (("dlam", dlam, rdlam), ("du", du, rdu)):
        if ref.ndim == 5:
            for n in range(ref.shape[0]):
                assert_close(got[n], ref[n], dtype, f"{what} {name}[{n}]")
        else:
            assert_close(got, ref, dtype, f"{what} {name}")
    for n in range(rdw.shape[0]):
        for k in range(3):
            assert_close(dw[n, k], rdw[n, k], dtype, f"{what} dw[{n}][{k}]")


# ---------------------------------------------------------------------------
# local GSPN groups
# ---------------------------------------------------------------------------
# (H, W, group_h, group_w): tile-aligned and mid-tile group boundaries, ragged
# last groups, one-line groups, groups longer than the axis
GROUP_CASES = [(16, 16, 4, 8), (28, 28, 2, 2), (28, 28, 5, 9), (32, 32, 1, 31), (56, 56, 7, 3),
               (64, 64, 16, 5), (13, 21, 4, 0), (13, 21, 0, 6), (128, 128, 32, 17), (128, 128, 2, 64),
               (130, 200, 33, 64), (600, 64, 100, 7), (520, 1032, 128, 300)]


@pytest.mark.parametrize("algo", FWD_ALGOS, ids=lambda a: ALGO_NAMES[a])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("case", GROUP_CASES, ids=lambda c: "x".join(map(str, c)))
def test_groups_fwd(case, dtype, algo):
    H, W, gh, gw = case
    print(f"[opt] groups fwd {case} {dtype} {ALGO_NAMES[algo]}", flush=True)
    planes = 3 if H * W <= 128 * 128 else 1
    inp = inputs(1, planes, H, W, 0xF, dtype, seed=H * 131 + W + gh + gw)
    check_fwd(inp, 0xF, algo, dtype, f"groups {case}", group_h=gh, group_w=gw)


@pytest.mark.parametrize("algo", FWD_ALGOS, ids=lambda a: ALGO_NAMES[a])
@pytest.mark.parametrize("mask", [1, 2, 4, 8, 3, 12, 5, 10, 7, 14, 15])
def test_groups_fwd_masks(mask, algo):
    print(f"[opt] groups fwd mask {mask} {ALGO_NAMES[algo]}", flush=True)
    inp = inputs(1, 2, 28, 28, mask, torch.float32, seed=300 + mask)
    check_fwd(inp, mask, algo, torch.float32, f"mask {mask}", group_h=6, group_w=10)


@pytest.mark.parametrize("algo", BWD_ALGOS, ids=lambda a: ALGO_NAMES[a])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("case", [c for c in GROUP_CASES if c[0] * c[1] <= 130 * 200],
                         ids=lambda c: "x".join(map(str, c)))
def test_groups_bwd(case, dtype, algo):
    H, W, gh, gw = case
    print(f"[opt] groups bwd {case} {dtype} {ALGO_NAMES[algo]}", flush=True)
    inp = inputs(1, 3, H, W, 0xF, dtype, seed=H * 17 + W + gh)
    check_bwd(inp, 0xF, algo, dtype, f"groups {case}", group_h=gh, group_w=gw)


@pytest.mark.parametrize("algo", BWD_ALGOS, ids=lambda a: ALGO_NAMES[a])
@pytest.mark.parametrize("mask", [1, 2, 4, 8, 3, 12, 5, 15])
def test_groups_bwd_masks(mask, algo):
    print(f"[opt] groups bwd mask {mask} {ALGO_NAMES[algo]}", flush=True)
    inp = inputs(1, 3, 16, 16, mask, torch.float32, seed=400 + mask)
    check_bwd(inp, mask, algo, torch.float32, f"mask {mask}", group_h=3, group_w=5)


def test_group_one_line_is_pointwise():
    """One-line groups: every direction is lam*x, so y = u * n * lam * x."""
    inp = inputs(2, 3, 28, 28, 0xF, torch.float32, seed=5)
    y = ops.gspn_scan_fwd(inp["x"], inp["w"], inp["lam"], inp["u"], 0xF, group_h=1, group_w=1)
    torch.cuda.synchronize()
    ref = np64(inp["u"]) * 4 * np64(inp["lam"]) * np64(inp["x"])
    assert_close(y, ref, torch.float32, "one-line groups")


# ---------------------------------------------------------------------------
# Eq. 6: logits normalised inside the call
# ---------------------------------------------------------------------------
LOGIT_SHAPES = [(1, 1), (5, 7), (16, 16), (28, 28), (33, 70), (130, 200)]


@pytest.mark.parametrize("renorm", [False, True], ids=["all3", "renorm"])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("shape", LOGIT_SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
def test_logits_fwd_bwd(shape, dtype, renorm):
    H, W = shape
    print(f"[opt] logits {shape} {dtype} renorm={renorm}", flush=True)
    inp = inputs(1, 2, H, W, 0xF, dtype, seed=H * 7 + W, logits=True)
    for algo in (0, 2):
        check_fwd(inp, 0xF, algo, dtype, f"logits {shape}", logits=True, renorm=renorm)
        check_bwd(inp, 0xF, algo, dtype, f"logits {shape}", logits=True, renorm=renorm)


# shapes that reach each kernel family with logits: size-specialised forward
# and staged backward (16, 28, 32), per-wave resident backward (56, 64),
# generic resident forward (128 and ragged), two-pass forward and backward
# (one band, several bands with halos, ragged last column block)
LOGIT_FAMILY_SHAPES = [(16, 16), (28, 28), (32, 32), (56, 56), (64, 64), (128, 128), (40, 72), (130, 200),
                       (600, 136)]


@pytest.mark.parametrize("algo", [1, 3, 4], ids=lambda a: ALGO_NAMES[a])
@pytest.mark.parametrize("renorm", [False, True], ids=["all3", "renorm"])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("shape", LOGIT_FAMILY_SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
def test_logits_every_family(shape, dtype, renorm, algo):
    H, W = shape
    print(f"[opt] logits family {shape} {dtype} renorm={renorm} {ALGO_NAMES[algo]}", flush=True)
    planes = 3 if H * W <= 64 * 64 else 1
    inp = inputs(1, planes, H, W, 0xF, dtype, seed=H * 13 + W + renorm, logits=True)
    check_fwd(inp, 0xF, algo, dtype, f"logits {shape}", logits=True, renorm=renorm)
    check_bwd(inp, 0xF, algo, dtype, f"logits {shape}", logits=True, renorm=renorm)


@pytest.mark.parametrize("algo", [0, 1, 3, 4], ids=lambda a: ALGO_NAMES[a])
@pytest.mark.parametrize("case", [(28, 28, 5, 9, 0x5), (64, 64, 16, 5, 0xA), (130, 200, 33, 64, 0xF),
                                  (600, 136, 100, 7, 0xC)], ids=lambda c: "x".join(map(str, c)))
def test_logits_with_groups_and_masks(case, algo):
    H, W, gh, gw, mask = case
    print(f"[opt] logits groups {case} {ALGO_NAMES[algo]}", flush=True)
    inp = inputs(1, 2, H, W, mask, torch.float32, seed=H + W + gh + gw, logits=True)
    opt = dict(group_h=gh, group_w=gw, logits=True, renorm=True)
    check_fwd(inp, mask, algo, torch.float32, f"logits groups {case}", **opt)
    check_bwd(inp, mask, algo, torch.float32, f"logits groups {case}", **opt)


@pytest.mark.parametrize("name", ["cls28_bf16_lg_fb", "lat128_bf16_lg_fb"])
def test_logit_workloads_sampled(name):
    """The benchmark's logits workloads (full size, AUTO): forward and backward
    of sampled planes against the oracle with Eq. 6 inside."""
    wl = synth.WORKLOADS[name]
    print(f"[opt] workload {name}", flush=True)
    inp = synth.make_inputs(wl, DEV)
    y = ops.gspn_scan_fwd(inp["x"], inp["w"], inp["lam"], inp["u"], wl.mask, logits=True)
    dx, dw, dlam, du = ops.gspn_scan_bwd(inp["dy"], inp["x"], inp["w"], inp["lam"], inp["u"], wl.mask, logits=True)
    torch.cuda.synchronize()
    last = (wl.B - 1, wl.C - 1)
    for b, c in ((0, 0), last):
        a = {k: np64(v[:, :, b:b + 1, c:c + 1] if k == "w" else v[b:b + 1, c:c + 1]) for k, v in inp.items()}
        ry = O.scan_fwd(a["x"], a["w"], a["lam"], a["u"], wl.mask, logits=True)
        assert_close(y[b:b + 1, c:c + 1], ry, torch.bfloat16, f"{name} y ({b},{c})")
        rdx, rdw, rdlam, rdu = O.scan_bwd(a["dy"], a["x"], a["w"], a["lam"], a["u"], wl.mask, logits=True)
        assert_close(dx[b:b + 1, c:c + 1], rdx, torch.bfloat16, f"{name} dx ({b},{c})")
        assert_close(dlam[b:b + 1, c:c + 1], rdlam, torch.bfloat16, f"{name} dlam ({b},{c})")
        assert_close(du[b:b + 1, c:c + 1], rdu, torch.bfloat16, f"{name} du ({b},{c})")
        for n in range(rdw.shape[0]):
            for k in range(3):
                assert_close(dw[n, k, b:b + 1, c:c + 1], rdw[n, k], torch.bfloat16, f"{name} dw[{n}][{k}] ({b},{c})")
    del inp, y, dx, dw, dlam, du
    torch.cuda.empty_cache()


def test_logits_of_stochastic_weights_match_the_plain_call():
    """Logits with sigmoid(l) = p and sum p = 1 give exactly the plain-weight result."""
    wl = synth.WORKLOADS["cls28_bf16_fb"].with_shape(B=1, C=4, dtype="f32")
    inp = synth.make_inputs(wl, DEV, with_dy=False)
    p = inp["w"].double().clamp(1e-6, 1 - 1e-6)
    lg = (torch.log(p) - torch.log1p(-p)).float()
    y0 = ops.gspn_scan_fwd(inp["x"], inp["w"], inp["lam"], inp["u"], 0xF)
    y1 = ops.gspn_scan_fwd(inp["x"], lg, inp["lam"], inp["u"], 0xF, logits=True)
    torch.cuda.synchronize()
    assert_close(y1, np64(y0), torch.float32, "logits of p")


# ---------------------------------------------------------------------------
# per-direction lam, u and outputs
# ---------------------------------------------------------------------------
PD = [(True, False, False), (False, True, False), (False, False, True), (True, True, False),
      (False, True, True), (True, True, True)]


@pytest.mark.parametrize("pd", PD, ids=lambda p: "".join("LUY"[i] if f else "-" for i, f in enumerate(p)))
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("mask", [15, 6, 1])
def test_per_direction_maps(mask, dtype, pd):
    lpd, upd, ypd = pd
    print(f"[opt] per-direction {pd} mask {mask} {dtype}", flush=True)
    inp = inputs(2, 2, 19, 24, mask, dtype, seed=mask * 10 + sum(pd), lam_pd=lpd, u_pd=upd, y_pd=ypd)
    opt = dict(lam_per_dir=lpd, u_per_dir=upd, y_per_dir=ypd, group_h=5)
    check_fwd(inp, mask, 0, dtype, f"per-dir {pd}", **opt)
    check_bwd(inp, mask, 0, dtype, f"per-dir {pd}", **opt)


# square planes that the per-wave resident backward takes, and a ragged one
# for the generic resident forward (its backward streams)
PD_SHAPES = [(16, 16), (28, 28), (56, 56), (64, 64), (40, 72)]


@pytest.mark.parametrize("algo", [0, 1, 3], ids=lambda a: ALGO_NAMES[a])
@pytest.mark.parametrize("pd", PD, ids=lambda p: "".join("LUY"[i] if f else "-" for i, f in enumerate(p)))
@pytest.mark.parametrize("shape", PD_SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
def test_per_direction_maps_resident(shape, pd, algo):
    """Per-direction maps on the resident families (forced and AUTO), with
    logits, against the oracle."""
    H, W = shape
    lpd, upd, ypd = pd
    print(f"[opt] per-direction resident {shape} {pd} {ALGO_NAMES[algo]}", flush=True)
    mask = 0xB
    inp = inputs(1, 3, H, W, mask, torch.bfloat16, seed=H + W + sum(pd), lam_pd=lpd, u_pd=upd, y_pd=ypd,
                 logits=True)
    opt = dict(lam_per_dir=lpd, u_per_dir=upd, y_per_dir=ypd, logits=True)
    check_fwd(inp, mask, algo, torch.bfloat16, f"per-dir {shape} {pd}", **opt)
    check_bwd(inp, mask, algo, torch.bfloat16, f"per-dir {shape} {pd}", **opt)


@pytest.mark.parametrize("algo", [0, 4], ids=lambda a: ALGO_NAMES[a])
@pytest.mark.parametrize("mask", [15, 5, 12, 9])
@pytest.mark.parametrize("shape", [(64, 128), (128, 128), (600, 136)], ids=lambda s: f"{s[0]}x{s[1]}")
def test_per_direction_outputs_two_pass(shape, mask, algo):
    """Unmerged outputs (and dy) on the two-pass family, with logits: every
    direction writes its own y_d; the backward seeds each direction from its
    own dy_d and forms du = sum_d dy_d h_d."""
    H, W = shape
    print(f"[opt] two-pass unmerged {shape} mask {mask} {ALGO_NAMES[algo]}", flush=True)
    inp = inputs(1, 2, H, W, mask, torch.bfloat16, seed=H + W + mask, y_pd=True, logits=True)
    opt = dict(y_per_dir=True, logits=True)
    check_fwd(inp, mask, algo, torch.bfloat16, f"two-pass unmerged {shape}", **opt)
    check_bwd(inp, mask, algo, torch.bfloat16, f"two-pass unmerged {shape}", **opt)


def test_all_options_together_autograd():
    """Groups, logits with edge renormalisation and per-direction maps through
    the autograd wrapper."""
    mask = 0xF
    inp = inputs(1, 2, 12, 17, mask, torch.float32, seed=77, lam_pd=True, u_pd=True, y_pd=True, logits=True)
    opt = dict(group_h=5, group_w=4, logits=True, renorm=True, lam_per_dir=True, u_per_dir=True,
               y_per_dir=True)
    leaves = {k: inp[k].clone().requires_grad_(True) for k in ("x", "w", "lam", "u")}
    y = ops.gspn_scan(leaves["x"], leaves["w"], leaves["lam"], leaves["u"], mask, **opt)
    (y * inp["dy"]).sum().backward()
    a = {k: np64(v) for k, v in inp.items()}
    ref = O.scan_bwd(a["dy"], a["x"], a["w"], a["lam"], a["u"], mask, **oracle_kw(opt))
    for got, r, name in zip((leaves[k].grad for k in ("x", "w", "lam", "u")), ref, ("dx", "dw", "dlam", "du")):
        assert_close(got, r, torch.float32, name)
