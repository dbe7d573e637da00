"""The allocation-free forward (gspn_scan_fwd_noalloc) against the regular
forward with a caller workspace, through the C ABI: two calls in a row on
problems whose kernels use scratch memory, the second one smaller, so the
second call runs on what the first left in the library's fixed array."""
import ctypes

import pytest
import torch

from paper_2501_12381_amd import lib as L
from paper_2501_12381_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
DT = {torch.float32: L.GSPN_F32, torch.bfloat16: L.GSPN_BF16}


def _inputs(B, C, H, W, mask, dtype, seed):
    t = synth.random_general((B, C, H, W), bin(mask).count("1"), device=DEV, seed=seed)
    return {k: v.to(dtype).contiguous() for k, v in t.items()}


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _regular(inp, mask, group_h=0):
    B, C, H, W = inp["x"].shape
    dt = DT[inp["x"].dtype]
    need = L.gspn_scan_fwd_workspace_bytes(B, C, H, W, mask, dt, group_h, 0, 0, L.GSPN_ALGO_AUTO)
    assert need > 0, "the case must use scratch memory"
    ws = torch.empty(need, dtype=torch.uint8, device=DEV)
    y = torch.empty_like(inp["x"])
    st = L.gspn_scan_fwd(inp["x"].data_ptr(), inp["w"].data_ptr(), inp["lam"].data_ptr(), inp["u"].data_ptr(),
                         y.data_ptr(), B, C, H, W, mask, dt, group_h, 0, 0, L.GSPN_ALGO_AUTO, ws.data_ptr(),
                         need, _stream())
    assert st == 0, L.gspn_strerror(st)
    return y


def _noalloc(inp, mask, group_h=0):
    B, C, H, W = inp["x"].shape
    y = torch.full_like(inp["x"], float("nan"))
    st = L.gspn_scan_fwd_noalloc(inp["x"].data_ptr(), inp["w"].data_ptr(), inp["lam"].data_ptr(),
                                 inp["u"].data_ptr(), y.data_ptr(), B, C, H, W, mask, DT[inp["x"].dtype],
                                 group_h, 0, 0, _stream())
    assert st == 0, L.gspn_strerror(st)
    return y


# (first problem, second smaller problem): two-pass kernels (partial sums and
# column state in scratch), then the streaming family (fp32 accumulator)
CASES = [
    ((1, 3, 300, 256, 0xF, torch.bfloat16, 0), (1, 1, 300, 64, 0xF, torch.bfloat16, 0)),
    ((1, 2, 520, 1032, 0xF, torch.bfloat16, 0), (1, 1, 400, 64, 0x7, torch.bfloat16, 0)),
    ((2, 2, 90, 2049, 0xF, torch.float32, 0), (1, 1, 33, 2049, 0xB, torch.float32, 0)),
    ((1, 2, 300, 256, 0xF, torch.float32, 40), (1, 1, 100, 2049, 0xF, torch.float32, 7)),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[0][2]}x{c[0][3]}-then-{c[1][2]}x{c[1][3]}")
def test_noalloc_matches_workspace_forward(case):
    for k, (B, C, H, W, mask, dtype, gh) in enumerate(case):
        print(f"[noalloc] call {k}: {B}x{C}x{H}x{W} mask {mask} {dtype} group_h {gh}", flush=True)
        inp = _inputs(B, C, H, W, mask, dtype, seed=1000 * k + H + W)
        ref = _regular(inp, mask, gh)
        got = _noalloc(inp, mask, gh)
        torch.cuda.synchronize()
        # the same kernels on the same inputs: bitwise equal
        assert torch.equal(got.view(torch.int16 if dtype == torch.bfloat16 else torch.int32),
                           ref.view(torch.int16 if dtype == torch.bfloat16 else torch.int32)), (k, case)


def test_noalloc_rejects_problems_beyond_its_scratch():
    B, C, H, W = 1, 8, 2048, 2048  # two-pass partial sums alone: 256 MiB
    need = L.gspn_scan_fwd_workspace_bytes(B, C, H, W, 0xF, L.GSPN_BF16, 0, 0, 0, L.GSPN_ALGO_AUTO)
    assert need > L.GSPN_NOALLOC_SCRATCH_BYTES
    # real tensors of the full size (the size check comes before any launch)
    t = {k: torch.zeros(shape, dtype=torch.bfloat16, device=DEV)
         for k, shape in (("x", (B, C, H, W)), ("lam", (B, C, H, W)), ("u", (B, C, H, W)), ("y", (B, C, H, W)),
                          ("w", (4, 3, B, C, H, W)))}
    st = L.gspn_scan_fwd_noalloc(t["x"].data_ptr(), t["w"].data_ptr(), t["lam"].data_ptr(), t["u"].data_ptr(),
                                 t["y"].data_ptr(), B, C, H, W, 0xF, L.GSPN_BF16, 0, 0, 0, _stream())
    assert st == 8
    torch.cuda.synchronize()
    assert not t["y"].any()  # nothing was written
    del t
    torch.cuda.empty_cache()


def test_noalloc_without_scratch_needs_no_lookup():
    """Problems the resident kernels take need no scratch at all."""
    inp = _inputs(2, 3, 28, 28, 0xF, torch.bfloat16, seed=3)
    got = _noalloc(inp, 0xF)
    B, C, H, W = inp["x"].shape
    y = torch.empty_like(inp["x"])
    st = L.gspn_scan_fwd(inp["x"].data_ptr(), inp["w"].data_ptr(), inp["lam"].data_ptr(), inp["u"].data_ptr(),
                         y.data_ptr(), B, C, H, W, 0xF, L.GSPN_BF16, 0, 0, 0, L.GSPN_ALGO_AUTO, None, 0, _stream())
    assert st == 0
    torch.cuda.synchronize()
    assert torch.equal(got.view(torch.int16), y.view(torch.int16))
