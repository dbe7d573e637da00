"""C ABI contract checks that need no GPU.

The library must load, export every function include/gspn.h declares, size
workspaces on the host, and reject bad arguments before touching the device
(every call below returns from host-side validation; none launches a kernel).
"""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gspn.h")

L = pytest.importorskip("paper_2501_12381_amd.lib")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(L.LIB_PATH):
        pytest.fail("libgspn.so is not built (run __graft_entry__.build())")
    return L.load()


def header_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(gspn_[a-z_0-9]+)\s*\(", src)))


def test_header_declares_expected_api():
    assert header_functions() == sorted(L.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    for name in header_functions():
        assert hasattr(lib, name), name
        assert ctypes.cast(getattr(lib, name), ctypes.c_void_p).value


def test_header_constants_match_binding():
    src = open(HEADER).read()
    consts = dict(re.findall(r"\b(GSPN_[A-Z0-9_]+)\s*=\s*(\d+)u?", src))
    for name in ("GSPN_F32", "GSPN_BF16", "GSPN_DIR_T2B", "GSPN_DIR_B2T", "GSPN_DIR_L2R",
                 "GSPN_DIR_R2L", "GSPN_ALGO_AUTO", "GSPN_ALGO_RESIDENT", "GSPN_ALGO_STREAM",
                 "GSPN_ALGO_RESIDENT_GENERIC", "GSPN_ALGO_TWO_PASS", "GSPN_FLAG_W_LOGITS",
                 "GSPN_FLAG_EDGE_RENORM", "GSPN_FLAG_LAM_PER_DIR", "GSPN_FLAG_U_PER_DIR",
                 "GSPN_FLAG_Y_PER_DIR", "GSPN_FLAG_SAVE_STATE"):
        assert int(consts[name]) == getattr(L, name), name
    for code, name in L.STATUS.items():
        assert int(consts[name]) == code, name
    assert int(re.search(r"#define GSPN_MAX_LINE (\d+)", src).group(1)) == L.GSPN_MAX_LINE


def test_strerror_and_version(lib):
    for code in list(L.STATUS) + [42, -1]:
        s = L.gspn_strerror(code)
        assert isinstance(s, str) and s
    assert L.gspn_strerror(0) == "success"
    assert L.gspn_version() >= 200


def test_workspace_sizes():
    f32, bf = L.GSPN_F32, L.GSPN_BF16
    S = L.GSPN_ALGO_STREAM
    npc = 2 * 3 * 5 * 7
    # streaming forward: one fp32 accumulator when several directions are merged
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 7, 0x1, f32, algo=S) == 0
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 7, 0xF, bf, algo=S) >= npc * 4
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 7, 0xF, bf, algo=S) % 256 == 0
    # streaming backward: previous-line state, sum of h, sum of g (fp32 each)
    assert L.gspn_scan_bwd_workspace_bytes(2, 3, 5, 7, 0xF, f32, algo=S) >= 3 * npc * 4
    # two-pass forward: fp32 partial sums (several directions; two arrays when
    # both vertical directions feed a horizontal pass), then the column state of
    # the horizontal pass (2 parities x 2 directions x planes x H floats)
    T = L.GSPN_ALGO_TWO_PASS
    acc, state = 2 * 3 * 5 * 64 * 4, 512  # 7680 is a multiple of 256; 4*6*5*4 = 480 -> 512
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 64, 0xF, bf, algo=T) == 2 * acc + state
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 64, 0x7, bf, algo=T) == 2 * acc + state
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 64, 0xD, bf, algo=T) == acc + state
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 64, 0x3, bf, algo=T) == acc
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 64, 0x4, bf, algo=T) == state
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 64, 0x1, bf, algo=T) == 0
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 60, 0xF, bf, algo=T) == 0  # W*2 not a multiple of 16
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 56, 0xF, bf, algo=T) == 0  # row under 128 bytes
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 32, 0xF, f32, algo=T) == 2 * (2 * 3 * 5 * 32 * 4) + 512
    # two-pass backward (a horizontal direction present): h of one direction,
    # the sum of the horizontal h, the sum of g (fp32 each), bottom-to-top's h
    # when both vertical directions are present, then the column state of the
    # horizontal launches (2 parities x 3 products x planes x H floats: 720 B -> 768)
    assert L.gspn_scan_bwd_workspace_bytes(2, 3, 5, 64, 0xF, bf, algo=T) == 4 * acc + 768
    assert L.gspn_scan_bwd_workspace_bytes(2, 3, 5, 64, 0x4, bf, algo=T) == 3 * acc + 768
    assert L.gspn_scan_bwd_workspace_bytes(2, 3, 5, 64, 0x5, bf, algo=T) == 3 * acc + 768
    assert L.gspn_scan_bwd_workspace_bytes(2, 3, 5, 64, 0x3, bf, algo=T) == 0  # no horizontal direction
    assert L.gspn_scan_bwd_workspace_bytes(2, 3, 5, 60, 0xF, bf, algo=T) == 0
    big_b = L.gspn_scan_bwd_workspace_bytes(1, 2, 2048, 2048, 0xF, bf, algo=L.GSPN_ALGO_AUTO)
    assert big_b == 4 * (2 * 2048 * 2048 * 4) + 6 * 2 * 2048 * 4
    # AUTO takes the two-pass kernels for planes that do not fit on chip
    big = L.gspn_scan_fwd_workspace_bytes(1, 2, 2048, 2048, 0xF, bf, algo=L.GSPN_ALGO_AUTO)
    assert big == 2 * (2 * 2048 * 2048 * 4) + 4 * 2 * 2048 * 4
    # invalid problems report 0
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 7, 0, f32, algo=S) == 0
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 7, 1, 7, algo=S) == 0
    assert L.gspn_scan_fwd_workspace_bytes(0, 3, 5, 7, 0xF, f32, algo=S) == 0


FAKE = 1 << 40  # never dereferenced: every call below fails validation first


def _no_gpu():
    """Fake-pointer calls run only where no GPU exists, so a validation slip can
    never turn into a launch on real hardware."""
    try:
        import torch
        if torch.cuda.is_available():
            pytest.skip("host-validation checks with fake pointers run only without a GPU")
    except ImportError:
        pass


def fwd(x=FAKE, w=FAKE + (1 << 30), lam=FAKE + (2 << 30), u=FAKE + (3 << 30), y=FAKE + (4 << 30),
        B=1, C=2, H=8, W=8, mask=0xF, dtype=L.GSPN_F32, algo=L.GSPN_ALGO_STREAM, ws=FAKE + (5 << 30),
        ws_bytes=1 << 20, group_h=0, group_w=0, flags=0):
    return L.gspn_scan_fwd(x, w, lam, u, y, B, C, H, W, mask, dtype, group_h, group_w, flags, algo, ws,
                           ws_bytes, None)


def test_fwd_rejects_bad_arguments(lib):
    _no_gpu()
    assert fwd(mask=0) == 3
    assert fwd(mask=16) == 3
    assert fwd(dtype=2) == 4
    assert fwd(algo=9) == 7
    assert fwd(B=-1) == 2
    assert fwd(B=1 << 40, C=1 << 40) == 2  # element count overflows int64
    assert fwd(x=None) == 1
    assert fwd(y=None) == 1
    assert fwd(x=FAKE + 2) == 5  # fp32 needs 4-byte alignment
    assert fwd(dtype=L.GSPN_BF16, x=FAKE + 1) == 5
    assert fwd(y=FAKE + 8) == 6  # y overlaps x
    assert fwd(y=FAKE + (1 << 30) + 64) == 6  # y inside w
    assert fwd(H=L.GSPN_MAX_LINE + 1) == 7
    assert fwd(ws=None) == 8
    assert fwd(ws_bytes=16) == 8
    assert fwd(ws=FAKE + (5 << 30) + 64) == 5  # workspace must be 256-byte aligned
    assert fwd(ws=FAKE + 256) == 6  # workspace overlaps x (x spans 512 bytes)
    assert fwd(algo=L.GSPN_ALGO_RESIDENT, H=4096, W=4096) == 7
    assert fwd(algo=L.GSPN_ALGO_TWO_PASS) == 7  # 8 fp32 columns: row under 128 bytes
    # the two-pass kernels need 16-byte aligned tensors when forced
    assert fwd(algo=L.GSPN_ALGO_TWO_PASS, W=64, dtype=L.GSPN_BF16, x=FAKE + 2) == 5
    # options: unknown flags, edge renormalisation without logits, negative groups
    assert fwd(flags=64) == 7
    assert fwd(flags=L.GSPN_FLAG_EDGE_RENORM) == 7
    assert fwd(group_h=-1) == 7
    assert fwd(group_w=-2) == 7
    # per-direction maps: the resident forward takes unmerged outputs and
    # per-direction lam, not a merged y with per-direction u; the two-pass
    # family takes unmerged outputs only (forcing a family that does not take a
    # flag is refused)
    assert fwd(algo=L.GSPN_ALGO_RESIDENT, flags=L.GSPN_FLAG_U_PER_DIR) == 7
    assert fwd(algo=L.GSPN_ALGO_RESIDENT_GENERIC, flags=L.GSPN_FLAG_W_LOGITS | L.GSPN_FLAG_U_PER_DIR) == 7
    assert fwd(algo=L.GSPN_ALGO_TWO_PASS, W=64, dtype=L.GSPN_BF16, flags=L.GSPN_FLAG_U_PER_DIR | L.GSPN_FLAG_Y_PER_DIR) == 7
    # per-direction maps are n times larger: y (4 maps of 512 bytes) overlaps u's
    # second map, lam's fourth map reaches into y
    assert fwd(flags=L.GSPN_FLAG_U_PER_DIR, y=FAKE + (3 << 30) + 512) == 6
    assert fwd(flags=L.GSPN_FLAG_LAM_PER_DIR, lam=FAKE + (4 << 30) - 2048 + 64) == 6
    assert fwd(flags=L.GSPN_FLAG_Y_PER_DIR, y=FAKE - 1024) == 6  # 4 maps of y reach into x


def test_empty_problem_is_a_noop(lib):
    _no_gpu()
    # nothing to compute: OK without looking at the pointers
    assert fwd(B=0, x=None, y=None) == 0
    assert fwd(H=0, x=None, y=None, ws=None) == 0


def test_bwd_rejects_bad_arguments(lib):
    _no_gpu()
    base = [FAKE + (k << 30) for k in range(10)]

    def bwd(**kw):
        p = dict(zip(["dy", "x", "w", "lam", "u", "dx", "dw", "dlam", "du", "ws"], base))
        p.update({k: v for k, v in kw.items() if k in p})
        dims = dict(B=1, C=2, H=8, W=8, mask=0xF, dtype=L.GSPN_F32, algo=L.GSPN_ALGO_STREAM,
                    ws_bytes=1 << 24, group_h=0, group_w=0, flags=0)
        dims.update({k: v for k, v in kw.items() if k in dims})
        return L.gspn_scan_bwd(p["dy"], p["x"], p["w"], p["lam"], p["u"], p["dx"], p["dw"],
                               p["dlam"], p["du"], dims["B"], dims["C"], dims["H"], dims["W"],
                               dims["mask"], dims["dtype"], dims["group_h"], dims["group_w"],
                               dims["flags"], dims["algo"], p["ws"], dims["ws_bytes"], None)

    assert bwd(mask=0) == 3
    assert bwd(dtype=5) == 4
    assert bwd(dw=None) == 1
    assert bwd(du=base[5]) == 6  # du aliases dx
    assert bwd(dx=base[0] + 128) == 6  # dx inside dy
    assert bwd(ws_bytes=100) == 8
    assert bwd(W=-3) == 2
    assert bwd(flags=64) == 7
    assert bwd(group_w=-1) == 7
    assert bwd(flags=L.GSPN_FLAG_Y_PER_DIR, dx=base[0] + 1024) == 6  # dy holds 4 maps: dx inside it


def test_bwd_auto_workspace_covers_element_aligned_pointers():
    """AUTO falls back from the resident backward (16-byte vectors) to the
    streaming family when a tensor is only element-aligned; the AUTO size must
    cover that fallback for every shape the resident kernels take."""
    A, S = L.GSPN_ALGO_AUTO, L.GSPN_ALGO_STREAM
    for dt in (L.GSPN_F32, L.GSPN_BF16):
        for side in (16, 28, 32, 56, 64):
            for mask in (1, 5, 12, 15):
                auto = L.gspn_scan_bwd_workspace_bytes(2, 3, side, side, mask, dt, algo=A)
                stream = L.gspn_scan_bwd_workspace_bytes(2, 3, side, side, mask, dt, algo=S)
                assert stream > 0 and auto >= stream, (dt, side, mask, auto, stream)


def test_workspace_sizes_with_options():
    f32, bf = L.GSPN_F32, L.GSPN_BF16
    A = L.GSPN_ALGO_AUTO
    npc4 = 2 * 3 * 5 * 7 * 4
    # unmerged outputs need no accumulator
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 7, 0xF, f32, flags=L.GSPN_FLAG_Y_PER_DIR, algo=A) == 0
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 7, 0xF, f32, flags=L.GSPN_FLAG_U_PER_DIR, algo=A) >= npc4
    # flags and groups run in the streaming family: its sizes
    assert L.gspn_scan_bwd_workspace_bytes(2, 3, 5, 7, 0xF, bf, flags=L.GSPN_FLAG_W_LOGITS, algo=A) >= 3 * npc4
    # a group at least as long as the axis is the global scan (same family, same size)
    for g in (0, 5, 6, 100):
        assert (L.gspn_scan_fwd_workspace_bytes(1, 2, 5, 64, 0xF, bf, group_h=g, algo=A)
                == L.gspn_scan_fwd_workspace_bytes(1, 2, 5, 64, 0xF, bf, algo=A))
    # invalid options report 0
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 7, 0xF, f32, flags=1 << 7, algo=A) == 0
    assert L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 7, 0xF, f32, group_h=-1, algo=A) == 0


def test_workspace_sizes_with_saved_state():
    """GSPN_FLAG_SAVE_STATE on the two-pass family: the forward keeps the
    present directions' h and sum_d h_d (fp32 arrays) and its column state; the
    backward's size is that plus the sum of g and the column products of the two
    horizontal adjoints.  Problems the flag does not apply to keep their sizes."""
    bf, T, A = L.GSPN_BF16, L.GSPN_ALGO_TWO_PASS, L.GSPN_ALGO_AUTO
    K = L.GSPN_FLAG_SAVE_STATE
    fb, state, bstate = 2 * 3 * 5 * 64 * 4, 512, 768
    fwd_ws = lambda mask, flags=K, algo=T, **kw: L.gspn_scan_fwd_workspace_bytes(2, 3, 5, 64, mask, bf, flags=flags,
                                                                                 algo=algo, **kw)
    bwd_ws = lambda mask, flags=K, algo=T: L.gspn_scan_bwd_workspace_bytes(2, 3, 5, 64, mask, bf, flags=flags,
                                                                           algo=algo)
    # h of T2B, B2T, the sum, h of L2R, R2L, then the column state
    assert fwd_ws(0xF) == 5 * fb + state
    assert fwd_ws(0x4) == 2 * fb + state
    assert fwd_ws(0x5) == 3 * fb + state
    assert fwd_ws(0xE) == 4 * fb + state
    assert fwd_ws(0xF, flags=K | L.GSPN_FLAG_W_LOGITS, group_w=7) == 5 * fb + state
    for m in (0xF, 0x4, 0x5, 0xE, 0x9):
        assert bwd_ws(m) == fwd_ws(m) + fb + 2 * bstate  # one column-product state per horizontal adjoint
    # no horizontal direction, or unmerged outputs: the flag changes nothing
    assert fwd_ws(0x3) == fwd_ws(0x3, flags=0)
    assert bwd_ws(0x3) == bwd_ws(0x3, flags=0) == 0
    Y = L.GSPN_FLAG_Y_PER_DIR
    assert fwd_ws(0xF, flags=K | Y) == fwd_ws(0xF, flags=Y)
    assert bwd_ws(0xF, flags=K | Y) == bwd_ws(0xF, flags=Y)
    # AUTO: the two-pass family for large planes, the flag ignored where a
    # plane stays on chip
    big = 2 * 2048 * 2048 * 4
    assert L.gspn_scan_fwd_workspace_bytes(1, 2, 2048, 2048, 0xF, bf, flags=K, algo=A) == 5 * big + 4 * 2 * 2048 * 4
    assert (L.gspn_scan_bwd_workspace_bytes(1, 2, 2048, 2048, 0xF, bf, flags=K, algo=A)
            == 6 * big + 4 * 2 * 2048 * 4 + 2 * 6 * 2 * 2048 * 4)
    for S in (28, 128):
        assert (L.gspn_scan_fwd_workspace_bytes(4, 8, S, S, 0xF, bf, flags=K, algo=A)
                == L.gspn_scan_fwd_workspace_bytes(4, 8, S, S, 0xF, bf, algo=A))
        assert (L.gspn_scan_bwd_workspace_bytes(4, 8, S, S, 0xF, bf, flags=K, algo=A)
                == L.gspn_scan_bwd_workspace_bytes(4, 8, S, S, 0xF, bf, algo=A))


def test_saved_state_refusals(lib):
    """A kept state must come from the two-pass kernels: the forward refuses
    element-aligned tensors instead of falling back to streaming, and the
    allocation-free forward refuses the flag (fake pointers, rejected before
    any launch)."""
    _no_gpu()
    K = L.GSPN_FLAG_SAVE_STATE
    big = dict(H=2048, W=64, dtype=L.GSPN_BF16, ws_bytes=1 << 30)
    assert fwd(algo=L.GSPN_ALGO_AUTO, flags=K, x=FAKE + 2, **big) == 5
    assert fwd(algo=L.GSPN_ALGO_TWO_PASS, flags=K, u=FAKE + (3 << 30) + 8, **big) == 5
    assert L.gspn_scan_fwd_noalloc(FAKE, FAKE + (1 << 30), FAKE + (2 << 30), FAKE + (3 << 30), FAKE + (4 << 30),
                                   1, 2, 8, 64, 0xF, L.GSPN_BF16, 0, 0, K, None) == 7
