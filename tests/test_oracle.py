"""Pins for the float64 oracle (CPU only).

Each test checks the oracle against something other than itself: a dense
linear solve, closed forms, combinatorial identities, invariants that follow
from the Stability-Context Condition (Sec. 3.2, App. A), adjoint identities and
finite differences.  Every plausible slip in the oracle (a dropped term, a
wrong sign or neighbour offset, a transposed operand, a missing first-line
lambda) breaks at least one of them.
"""
import os

import numpy as np
import pytest

import oracle as O

RNG = np.random.default_rng(20250121)

# ---------------------------------------------------------------------------
# helpers written from the geometry of each direction, independent of the oracle
# ---------------------------------------------------------------------------
# Each direction is a frame (a, b): a = scan coordinate (line index in visiting
# order), b = position along the line.  Neighbour k of frame pixel (a, b) is
# (a - 1, b + k - 1).  The map frame -> image pixel (i, j):
FRAMES = {
    O.T2B: lambda a, b, H, W: (a, b),
    O.B2T: lambda a, b, H, W: (H - 1 - a, b),
    O.L2R: lambda a, b, H, W: (b, a),
    O.R2L: lambda a, b, H, W: (b, W - 1 - a),
}
FRAME_DIMS = {O.T2B: lambda H, W: (H, W), O.B2T: lambda H, W: (H, W),
              O.L2R: lambda H, W: (W, H), O.R2L: lambda H, W: (W, H)}


def dense_M(w3, direction):
    """N x N matrix M with h = M h + lam*x, rows/cols in row-major pixel order."""
    _, H, W = w3.shape
    A, Bn = FRAME_DIMS[direction](H, W)
    f = FRAMES[direction]
    M = np.zeros((H * W, H * W))
    for a in range(A):
        for b in range(Bn):
            i, j = f(a, b, H, W)
            for k in range(3):
                a2, b2 = a - 1, b + k - 1
                if 0 <= a2 < A and 0 <= b2 < Bn:
                    i2, j2 = f(a2, b2, H, W)
                    M[i * W + j, i2 * W + j2] += w3[k, i, j]
    return M


def general_plane(H, W, signed=True, rng=RNG):
    x = rng.standard_normal((H, W))
    lam = rng.uniform(-0.5, 1.5, (H, W))
    w3 = rng.uniform(0, 1, (3, H, W))
    if signed:
        w3 *= np.where(rng.uniform(size=w3.shape) < 0.3, -1.0, 1.0)
    w3 = w3 / (np.abs(w3).sum(0, keepdims=True) + 0.1)
    return x, w3, lam


def stochastic_w(shape, rng=RNG, std=1.0):
    z = rng.standard_normal((3,) + shape) * std
    e = np.exp(z - z.max(0, keepdims=True))
    return e / e.sum(0, keepdims=True)


SHAPES = [(1, 1), (1, 5), (5, 1), (2, 2), (3, 4), (5, 7), (7, 5), (6, 6)]


# ---------------------------------------------------------------------------
# 1. brute force: dense solve of (I - M) h = lam x   (Eq. 1, Eq. 3, Eq. 8)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("direction", O.ALL_DIRS)
def test_dense_solve(shape, direction):
    H, W = shape
    x, w3, lam = general_plane(H, W)
    h = O.scan_direction(x, w3, lam, direction)
    M = dense_M(w3, direction)
    ref = np.linalg.solve(np.eye(H * W) - M, (lam * x).ravel()).reshape(H, W)
    np.testing.assert_allclose(h, ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("shape", [(1, 3), (4, 3), (5, 6), (6, 5)])
def test_eq3_block_products(shape):
    """H = G X with G_ij = w_i ... w_{j+1} lam_j (Eq. 3), top-to-bottom scan."""
    H, W = shape
    x, w3, lam = general_plane(H, W)
    G = O.g_blocks_t2b(w3, lam)
    h = O.scan_direction(x, w3, lam, O.T2B)
    np.testing.assert_allclose(h.ravel(), G @ x.ravel(), rtol=0, atol=1e-12)
    # G is block lower triangular with diag(lam_i) on the diagonal blocks
    for i in range(H):
        np.testing.assert_array_equal(G[i * W:(i + 1) * W, i * W:(i + 1) * W], np.diag(lam[i]))
        assert not np.any(G[i * W:(i + 1) * W, (i + 1) * W:])


def test_line_matrix_is_tridiagonal_with_receiver_rows():
    w = np.arange(1, 3 * 4 + 1, dtype=float).reshape(3, 4)
    m = O.line_matrix(w)
    expect = np.array([[w[1, 0], w[2, 0], 0, 0],
                       [w[0, 1], w[1, 1], w[2, 1], 0],
                       [0, w[0, 2], w[1, 2], w[2, 2]],
                       [0, 0, w[0, 3], w[1, 3]]])
    np.testing.assert_array_equal(m, expect)


# ---------------------------------------------------------------------------
# 2. closed forms that fix the neighbour convention
# ---------------------------------------------------------------------------
# image displacement of neighbour k for each direction (Sec. 3.3 "top-left,
# top-middle, top-right" for top-to-bottom; Alg. 1 for left-to-right:
# G1 <-> (h-1, w-1), G2 <-> (h, w-1), G3 <-> (h+1, w-1))
DISP = {
    O.T2B: [(-1, -1), (-1, 0), (-1, 1)],
    O.B2T: [(1, -1), (1, 0), (1, 1)],
    O.L2R: [(-1, -1), (0, -1), (1, -1)],
    O.R2L: [(-1, 1), (0, 1), (1, 1)],
}


def chain_sum(lx, di, dj):
    """h[p] = sum of lx along p, p+d, p+2d, ... while inside the plane."""
    H, W = lx.shape
    out = np.zeros_like(lx)
    for i in range(H):
        for j in range(W):
            s, a, b = 0.0, i, j
            while 0 <= a < H and 0 <= b < W:
                s += lx[a, b]
                a, b = a + di, b + dj
            out[i, j] = s
    return out


@pytest.mark.parametrize("direction", O.ALL_DIRS)
@pytest.mark.parametrize("k", [0, 1, 2])
@pytest.mark.parametrize("shape", [(6, 9), (9, 6), (1, 4), (4, 1)])
def test_single_neighbour_chains(direction, k, shape):
    H, W = shape
    x = RNG.standard_normal((H, W))
    lam = RNG.uniform(0, 1, (H, W))
    w3 = np.zeros((3, H, W))
    w3[k] = 1.0
    h = O.scan_direction(x, w3, lam, direction)
    di, dj = DISP[direction][k]
    np.testing.assert_allclose(h, chain_sum(lam * x, di, dj), rtol=0, atol=1e-12)


@pytest.mark.parametrize("direction,axis,rev", [(O.T2B, 0, False), (O.B2T, 0, True),
                                                (O.L2R, 1, False), (O.R2L, 1, True)])
def test_middle_weight_is_cumsum(direction, axis, rev):
    H, W = 11, 8
    x = RNG.standard_normal((H, W))
    lam = RNG.uniform(0, 1, (H, W))
    w3 = np.zeros((3, H, W))
    w3[1] = 1.0
    lx = lam * x
    ref = np.flip(np.cumsum(np.flip(lx, axis), axis), axis) if rev else np.cumsum(lx, axis)
    np.testing.assert_allclose(O.scan_direction(x, w3, lam, direction), ref, rtol=0, atol=1e-12)


def test_trinomial_impulse():
    """Uniform weights 1/3, unit impulse at (0, j0): h[n][j0+m] = T(n, m) / 3^n."""
    H, W, j0 = 13, 41, 20
    x = np.zeros((H, W))
    x[0, j0] = 1.0
    lam = np.ones((H, W))
    w3 = np.full((3, H, W), 1.0 / 3.0)
    h = O.scan_direction(x, w3, lam, O.T2B)
    coeff = np.array([1.0])
    for n in range(H):
        m = np.arange(-n, n + 1)
        np.testing.assert_allclose(h[n, j0 + m], coeff / 3.0 ** n, rtol=1e-13, atol=0)
        coeff = np.convolve(coeff, [1.0, 1.0, 1.0])
    path = os.path.join(os.path.dirname(__file__), "golden", "central_trinomial.txt")
    golden = [int(v) for line in open(path) if not line.startswith("#") for v in line.split()]
    for n, t in enumerate(golden):
        assert round(h[n, j0] * 3.0 ** n) == t


# ---------------------------------------------------------------------------
# 3. Stability-Context Condition (Sec. 3.2, Thm 1-2, App. A)
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("direction", O.ALL_DIRS)
def test_interior_cone_keeps_constant_and_max_principle(direction):
    """Row-stochastic w, only the first visited line nonzero with lam*x = c.

    Thm 1: every product of row-stochastic matrices is row-stochastic, so pixels
    whose dependency cone stays inside the plane see exactly c; with zero padding
    the products are sub-stochastic at the edges, so 0 <= h <= c everywhere.
    """
    H = W = 17
    c = 2.5
    w3 = stochastic_w((H, W))
    x = np.zeros((H, W))
    lam = np.ones((H, W))
    first = {O.T2B: (0, slice(None)), O.B2T: (H - 1, slice(None)),
             O.L2R: (slice(None), 0), O.R2L: (slice(None), W - 1)}[direction]
    x[first] = c
    h = O.scan_direction(x, w3, lam, direction)
    assert h.min() >= -1e-15 and h.max() <= c * (1 + 1e-14)
    for a in range(H):  # frame line a: cone [a, L-1-a] along the line
        for b in range(a, W - a):
            i, j = FRAMES[direction](a, b, H, W)
            assert abs(h[i, j] - c) < 1e-13


@pytest.mark.parametrize("direction", [O.T2B, O.L2R])
def test_no_growth_over_long_chains(direction):
    """||h_i||_inf <= ||h_{i-1}||_inf + ||lam_i x_i||_inf for 4096 lines (Thm 2)."""
    L, n = 4096, 8
    shape = (L, n) if direction == O.T2B else (n, L)
    w3 = stochastic_w(shape)
    x = RNG.standard_normal(shape)
    lam = RNG.uniform(0, 1, shape)
    h = O.scan_direction(x, w3, lam, direction)
    hl = h if direction == O.T2B else h.T
    lxl = (lam * x) if direction == O.T2B else (lam * x).T
    prev = 0.0
    for i in range(L):
        cur = np.abs(hl[i]).max()
        assert cur <= prev + np.abs(lxl[i]).max() + 1e-12
        prev = cur
    assert np.isfinite(h).all()


def test_uniform_weight_mass_leak():
    """w = 1/3: sum_j h_i = sum_j h_{i-1} - (h_{i-1}[0] + h_{i-1}[W-1])/3 + sum_j lam x."""
    H, W = 20, 9
    x = RNG.standard_normal((H, W))
    lam = RNG.uniform(0, 1, (H, W))
    w3 = np.full((3, H, W), 1.0 / 3.0)
    h = O.scan_direction(x, w3, lam, O.T2B)
    for i in range(1, H):
        expect = h[i - 1].sum() - (h[i - 1, 0] + h[i - 1, -1]) / 3.0 + (lam[i] * x[i]).sum()
        assert abs(h[i].sum() - expect) < 1e-12


def test_adjoint_mass_leak():
    """Row-stochastic w, u = 1, dy only on the last line (top-to-bottom scan):
    sum g_i = sum g_{i+1} - w0[i+1][0] g_{i+1}[0] - w2[i+1][W-1] g_{i+1}[W-1]."""
    H, W = 15, 10
    w3 = stochastic_w((H, W))
    src = np.zeros((H, W))
    src[-1] = RNG.standard_normal(W)
    g = O.adjoint_direction(src, w3, O.T2B)
    for i in range(H - 1):
        expect = g[i + 1].sum() - w3[0, i + 1, 0] * g[i + 1, 0] - w3[2, i + 1, -1] * g[i + 1, -1]
        assert abs(g[i].sum() - expect) < 1e-12


# ---------------------------------------------------------------------------
# 4. directions as views of top-to-bottom; merge; linearity
# ---------------------------------------------------------------------------
def test_directions_are_views_of_t2b():
    H, W = 6, 9
    x, w3, lam = general_plane(H, W)
    t2b = lambda X, Wt, Lm: O.scan_direction(X, Wt, Lm, O.T2B)
    # B2T = flip rows of T2B on flipped rows
    fl = lambda a: np.flip(a, -2)
    np.testing.assert_allclose(O.scan_direction(x, w3, lam, O.B2T),
                               fl(t2b(fl(x), fl(w3), fl(lam))), atol=1e-13, rtol=0)
    # L2R = transpose of T2B on transposed planes (k unchanged)
    tr = lambda a: np.swapaxes(a, -1, -2)
    np.testing.assert_allclose(O.scan_direction(x, w3, lam, O.L2R),
                               tr(t2b(tr(x), tr(w3), tr(lam))), atol=1e-13, rtol=0)
    # R2L: X'[a, b] = X[b, W-1-a]
    rv = lambda a: np.swapaxes(np.flip(a, -1), -1, -2)
    inv = lambda a: np.flip(np.swapaxes(a, -1, -2), -1)
    np.testing.assert_allclose(O.scan_direction(x, w3, lam, O.R2L),
                               inv(t2b(rv(x), rv(w3), rv(lam))), atol=1e-13, rtol=0)


def test_merge_is_sum_of_directions_and_linear_in_x():
    B, C, H, W = 2, 3, 5, 6
    x = RNG.standard_normal((B, C, H, W))
    x2 = RNG.standard_normal((B, C, H, W))
    lam = RNG.uniform(0, 1, (B, C, H, W))
    u = RNG.standard_normal((B, C, H, W))
    w = np.stack([stochastic_w((B, C, H, W)) for _ in range(4)])
    y = O.scan_fwd(x, w, lam, u, 0xF)
    parts = [O.scan_fwd(x, w[n:n + 1], lam, u, d) for n, d in enumerate(O.ALL_DIRS)]
    np.testing.assert_allclose(y, sum(parts), atol=1e-13, rtol=0)
    # mask with a subset: packing order follows the bits
    y5 = O.scan_fwd(x, w[[0, 2]], lam, u, O.T2B | O.L2R)
    np.testing.assert_allclose(y5, parts[0] + parts[2], atol=1e-13, rtol=0)
    a, b = 0.7, -1.3
    np.testing.assert_allclose(O.scan_fwd(a * x + b * x2, w, lam, u, 0xF),
                               a * y + b * O.scan_fwd(x2, w, lam, u, 0xF), atol=1e-12, rtol=0)


def test_planes_are_independent():
    B, C, H, W = 2, 2, 4, 5
    x = RNG.standard_normal((B, C, H, W))
    lam = RNG.uniform(0, 1, (B, C, H, W))
    u = RNG.standard_normal((B, C, H, W))
    w = np.stack([stochastic_w((B, C, H, W)) for _ in range(4)])
    y = O.scan_fwd(x, w, lam, u, 0xF)
    for b in range(B):
        for c in range(C):
            yp = O.scan_fwd(x[b, c], w[:, :, b, c], lam[b, c], u[b, c], 0xF)
            np.testing.assert_allclose(y[b, c], yp, atol=1e-14, rtol=0)


# ---------------------------------------------------------------------------
# 5. backward: dense adjoint, Euler identities, finite differences
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("shape", [(1, 1), (3, 4), (5, 7), (7, 5), (4, 1)])
@pytest.mark.parametrize("direction", O.ALL_DIRS)
def test_adjoint_equals_dense_transpose_solve(shape, direction):
    H, W = shape
    _, w3, _ = general_plane(H, W)
    src = RNG.standard_normal((H, W))
    g = O.adjoint_direction(src, w3, direction)
    M = dense_M(w3, direction)
    ref = np.linalg.solve((np.eye(H * W) - M).T, src.ravel()).reshape(H, W)
    np.testing.assert_allclose(g, ref, atol=1e-12, rtol=0)


def _rand_problem(B, C, H, W, mask, rng=RNG):
    n = len(O.dirs_of(mask))
    x = rng.standard_normal((B, C, H, W))
    lam = rng.uniform(-0.5, 1.5, (B, C, H, W))
    u = rng.standard_normal((B, C, H, W))
    w = rng.uniform(-0.4, 0.6, (n, 3, B, C, H, W))
    dy = rng.standard_normal((B, C, H, W))
    return dy, x, w, lam, u


@pytest.mark.parametrize("mask", [1, 2, 4, 8, 5, 10, 15])
def test_euler_identities(mask):
    """y is linear in each of x, lam, u separately, so <dy, y> = <dx, x> = <dlam, lam> = <du, u>."""
    dy, x, w, lam, u = _rand_problem(2, 2, 5, 6, mask)
    y = O.scan_fwd(x, w, lam, u, mask)
    dx, dw, dlam, du = O.scan_bwd(dy, x, w, lam, u, mask)
    L = float((dy * y).sum())
    for g, v in ((dx, x), (dlam, lam), (du, u)):
        assert abs(float((g * v).sum()) - L) < 1e-11 * max(1.0, abs(L))


@pytest.mark.parametrize("mask", [1, 2, 4, 8, 15, 6])
@pytest.mark.parametrize("shape", [(3, 4), (4, 3), (1, 3), (3, 1)])
def test_finite_differences(mask, shape):
    H, W = shape
    dy, x, w, lam, u = _rand_problem(1, 2, H, W, mask)
    dx, dw, dlam, du = O.scan_bwd(dy, x, w, lam, u, mask)
    loss = lambda x_, w_, l_, u_: float((dy * O.scan_fwd(x_, w_, l_, u_, mask)).sum())
    eps = 1e-6
    args = [x, w, lam, u]
    grads = [dx, dw, dlam, du]
    for which in range(4):
        for _ in range(3):
            v = RNG.standard_normal(args[which].shape)
            plus = list(args)
            minus = list(args)
            plus[which] = args[which] + eps * v
            minus[which] = args[which] - eps * v
            fd = (loss(*plus) - loss(*minus)) / (2 * eps)
            an = float((grads[which] * v).sum())
            assert abs(fd - an) <= 1e-7 * max(1.0, abs(an)), (which, fd, an)
    # element-wise on dw: every weight of every direction, one by one
    for idx in np.ndindex(w.shape):
        e = np.zeros_like(w)
        e[idx] = eps
        fd = (loss(x, w + e, lam, u) - loss(x, w - e, lam, u)) / (2 * eps)
        assert abs(fd - dw[idx]) <= 1e-7 * max(1.0, abs(dw[idx])), idx


def test_first_line_and_edge_weights_have_zero_gradient():
    """Weights that point outside the plane or before the first line never act."""
    dy, x, w, lam, u = _rand_problem(1, 1, 4, 5, 0xF)
    _, dw, _, _ = O.scan_bwd(dy, x, w, lam, u, 0xF)
    # T2B: first row has no previous line; k=0 at column 0 and k=2 at column W-1 point outside
    assert not dw[0, :, :, :, 0, :].any()
    assert not dw[0, 0, :, :, :, 0].any() and not dw[0, 2, :, :, :, -1].any()
    # B2T: last row has no previous line
    assert not dw[1, :, :, :, -1, :].any()
    # L2R: first column; k=0 on row 0, k=2 on row H-1
    assert not dw[2, :, :, :, :, 0].any()
    assert not dw[2, 0, :, :, 0, :].any() and not dw[2, 2, :, :, -1, :].any()
    # R2L: last column
    assert not dw[3, :, :, :, :, -1].any()


def test_mask_validation():
    with pytest.raises(ValueError):
        O.dirs_of(0)
    with pytest.raises(ValueError):
        O.dirs_of(16)
