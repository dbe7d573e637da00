"""Pins for the oracle's options (CPU only): local GSPN groups (Sec. 4.1 "Local
vs Global GSPN", Alg. 1's kNItems groups), the weight normalisation of Eq. 6
(Sec. 3.3) and per-direction lam / u / y maps.

Each test checks the option against something other than its own code path:
the global scan of a sub-plane, closed forms, the plain-weight path at
weights the logits reproduce exactly, the central trinomial coefficients,
exact invariants that hold only when every row is stochastic, single-direction
runs, Euler identities and finite differences.
"""
import os

import numpy as np
import pytest

import oracle as O

RNG = np.random.default_rng(4096)
VERT = (O.T2B, O.B2T)


def general(B, C, H, W, n, rng=RNG):
    x = rng.standard_normal((B, C, H, W))
    lam = rng.uniform(-0.5, 1.5, (B, C, H, W))
    u = rng.standard_normal((B, C, H, W))
    w = rng.uniform(0, 1, (n, 3, B, C, H, W))
    w *= np.where(rng.uniform(size=w.shape) < 0.3, -1.0, 1.0)
    w = w / (np.abs(w).sum(1, keepdims=True) + 0.1)
    dy = rng.standard_normal((B, C, H, W))
    return dy, x, w, lam, u


# ---------------------------------------------------------------------------
# local GSPN
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("direction", O.ALL_DIRS)
def test_group_zero_or_longer_than_axis_is_global(direction):
    _, x, w, lam, _ = general(1, 2, 7, 9, 1)
    ref = O.scan_direction(x, w[0], lam, direction)
    n = 7 if direction in VERT else 9
    for g in (0, n, n + 3):
        np.testing.assert_array_equal(O.scan_direction(x, w[0], lam, direction, g), ref)


def test_group_of_one_line_is_pointwise():
    """g = n groups of one line (the O(1) extreme of Sec. 4.1): h_d = lam x for
    every direction, so y = u * n_dirs * lam * x."""
    _, x, w, lam, u = general(2, 3, 6, 5, 4)
    y = O.scan_fwd(x, w, lam, u, 0xF, group_h=1, group_w=1)
    np.testing.assert_allclose(y, u * 4 * lam * x, rtol=1e-14, atol=1e-14)


@pytest.mark.parametrize("direction", O.ALL_DIRS)
@pytest.mark.parametrize("G", [2, 3, 4])
def test_each_group_is_a_global_scan_of_its_subplane(direction, G):
    """A group is scanned exactly as the global scan of the sub-plane made of
    its lines alone (the groups' union is the axis, they do not overlap)."""
    H, W = 11, 10
    _, x, w, lam, _ = general(1, 1, H, W, 1)
    h = O.scan_direction(x, w[0], lam, direction, G)
    n = H if direction in VERT else W
    for a in range(0, n, G):
        b = min(a + G, n)
        if direction in VERT:
            sub = O.scan_direction(x[..., a:b, :], w[0][..., a:b, :], lam[..., a:b, :], direction)
            np.testing.assert_allclose(h[..., a:b, :], sub, rtol=0, atol=1e-14)
        else:
            sub = O.scan_direction(x[..., :, a:b], w[0][..., :, a:b], lam[..., :, a:b], direction)
            np.testing.assert_allclose(h[..., :, a:b], sub, rtol=0, atol=1e-14)


def test_groups_split_rows_for_vertical_and_columns_for_horizontal():
    """group_h only acts on T2B/B2T and group_w only on L2R/R2L."""
    _, x, w, lam, u = general(1, 1, 8, 9, 4)
    hs_g = O.scan_fwd_dirs(x, w, lam, 0xF, group_h=3, group_w=0)
    hs = O.scan_fwd_dirs(x, w, lam, 0xF)
    assert not np.allclose(hs_g[0], hs[0]) and not np.allclose(hs_g[1], hs[1])
    np.testing.assert_array_equal(hs_g[2], hs[2])
    np.testing.assert_array_equal(hs_g[3], hs[3])


@pytest.mark.parametrize("direction", O.ALL_DIRS)
def test_group_adjoint_equals_sum_of_subplane_adjoints(direction):
    """The adjoint of a grouped scan splits the same way as the forward."""
    H, W, G = 9, 8, 4
    dy, _, w, _, _ = general(1, 1, H, W, 1)
    g = O.adjoint_direction(dy, w[0], direction, G)
    n = H if direction in VERT else W
    for a in range(0, n, G):
        b = min(a + G, n)
        sl = (Ellipsis, slice(a, b), slice(None)) if direction in VERT else (Ellipsis, slice(None), slice(a, b))
        sub = O.adjoint_direction(dy[sl], w[0][sl], direction)
        np.testing.assert_allclose(g[sl], sub, rtol=0, atol=1e-14)


def _fd_check(loss, args, grads, eps=1e-6, tol=1e-7, reps=3):
    for which in range(len(args)):
        for _ in range(reps):
            v = RNG.standard_normal(args[which].shape)
            plus, minus = list(args), list(args)
            plus[which] = args[which] + eps * v
            minus[which] = args[which] - eps * v
            fd = (loss(*plus) - loss(*minus)) / (2 * eps)
            an = float((grads[which] * v).sum())
            assert abs(fd - an) <= tol * max(1.0, abs(an)), (which, fd, an)


@pytest.mark.parametrize("mask", [15, 5, 10])
@pytest.mark.parametrize("groups", [(2, 3), (3, 2), (1, 4)])
def test_group_finite_differences(mask, groups):
    gh, gw = groups
    n = bin(mask).count("1")
    dy, x, w, lam, u = general(1, 2, 5, 7, n)
    grads = O.scan_bwd(dy, x, w, lam, u, mask, group_h=gh, group_w=gw)
    loss = lambda x_, w_, l_, u_: float((dy * O.scan_fwd(x_, w_, l_, u_, mask, gh, gw)).sum())
    _fd_check(loss, [x, w, lam, u], list(grads))


# ---------------------------------------------------------------------------
# weight normalisation (Eq. 6)
# ---------------------------------------------------------------------------
def _logit(p):
    return np.log(p) - np.log1p(-p)


def stochastic(shape, rng=RNG):
    z = rng.standard_normal((3,) + shape)
    e = np.exp(z - z.max(0, keepdims=True))
    return e / e.sum(0, keepdims=True)


@pytest.mark.parametrize("mask", [1, 6, 15])
def test_logits_of_stochastic_rows_reproduce_the_weights(mask):
    """If sigmoid(l_k) = p_k with sum_k p_k = 1, Eq. 6 returns p itself."""
    n = bin(mask).count("1")
    _, x, _, lam, u = general(1, 2, 6, 7, n)
    p = np.stack([stochastic((1, 2, 6, 7)) for _ in range(n)])
    y_plain = O.scan_fwd(x, p, lam, u, mask)
    y_logit = O.scan_fwd(x, _logit(p), lam, u, mask, logits=True)
    np.testing.assert_allclose(y_logit, y_plain, rtol=1e-12, atol=1e-12)


def test_equal_logits_give_the_trinomial_impulse():
    """Equal logits normalise to 1/3 each: a unit impulse on the first row then
    spreads as the central trinomial coefficients (OEIS A002426)."""
    H, W, j0 = 12, 41, 20
    x = np.zeros((1, 1, H, W))
    x[..., 0, j0] = 1.0
    lam = np.ones_like(x)
    l3 = np.full((1, 3, 1, 1, H, W), 0.7)
    y = O.scan_fwd(x, l3, lam, np.ones_like(x), O.T2B, logits=True)
    path = os.path.join(os.path.dirname(__file__), "golden", "central_trinomial.txt")
    golden = [int(v) for line in open(path) if not line.startswith("#") for v in line.split()]
    for n in range(H):
        assert round(y[0, 0, n, j0] * 3.0 ** n) == golden[n]


@pytest.mark.parametrize("direction", O.ALL_DIRS)
def test_edge_renormalisation_makes_every_row_stochastic(direction):
    """With the sum over the on-line neighbours only, every row of every w_i is
    stochastic, edges included: a constant first line stays exactly constant
    over the whole plane (without it, mass leaks at the line ends)."""
    H, W, c = 9, 8, 1.75
    x = np.zeros((1, 1, H, W))
    first = {O.T2B: (..., 0, slice(None)), O.B2T: (..., H - 1, slice(None)),
             O.L2R: (..., slice(None), 0), O.R2L: (..., slice(None), W - 1)}[direction]
    x[first] = c
    lam = np.ones_like(x)
    l3 = RNG.standard_normal((1, 3, 1, 1, H, W)) * 2
    h = O.scan_fwd_dirs(x, l3, lam, direction, logits=True, renorm=True)[0]
    np.testing.assert_allclose(h, c, rtol=0, atol=1e-13)
    h0 = O.scan_fwd_dirs(x, l3, lam, direction, logits=True, renorm=False)[0]
    assert h0.min() < c - 1e-3


@pytest.mark.parametrize("direction", VERT)
def test_renormalised_single_position_lines_are_cumulative_sums(direction):
    """A line of one position has only the k = 1 neighbour: w_1 = 1 and each
    vertical scan is a cumulative sum of lam x down (or up) the column."""
    H = 9
    x = RNG.standard_normal((1, 1, H, 1))
    lam = RNG.uniform(0, 1, (1, 1, H, 1))
    l3 = RNG.standard_normal((1, 3, 1, 1, H, 1))
    h = O.scan_fwd_dirs(x, l3, lam, direction, logits=True, renorm=True)[0]
    lx = lam * x
    ref = np.cumsum(lx, axis=2) if direction == O.T2B else np.flip(np.cumsum(np.flip(lx, 2), 2), 2)
    np.testing.assert_allclose(h, ref, rtol=0, atol=1e-13)


@pytest.mark.parametrize("renorm", [False, True])
@pytest.mark.parametrize("mask", [15, 3, 12])
def test_logit_finite_differences(mask, renorm):
    n = bin(mask).count("1")
    dy, x, _, lam, u = general(1, 2, 4, 5, n)
    l = RNG.standard_normal((n, 3, 1, 2, 4, 5)) * 1.5
    dx, dl, dlam, du = O.scan_bwd(dy, x, l, lam, u, mask, logits=True, renorm=renorm)
    loss = lambda x_, l_, lam_, u_: float(
        (dy * O.scan_fwd(x_, l_, lam_, u_, mask, logits=True, renorm=renorm)).sum())
    _fd_check(loss, [x, l, lam, u], [dx, dl, dlam, du])
    # element by element on the logits
    eps = 1e-6
    for idx in list(np.ndindex(l.shape))[::7]:
        e = np.zeros_like(l)
        e[idx] = eps
        fd = (loss(x, l + e, lam, u) - loss(x, l - e, lam, u)) / (2 * eps)
        assert abs(fd - dl[idx]) <= 1e-7 * max(1.0, abs(dl[idx])), idx


def test_renorm_zeroes_the_gradient_of_off_line_logits():
    """Logits of neighbours outside the line take no part in Eq. 6 with edge
    renormalisation, so their gradient is exactly zero."""
    dy, x, _, lam, u = general(1, 1, 5, 6, 4)
    l = RNG.standard_normal((4, 3, 1, 1, 5, 6))
    _, dl, _, _ = O.scan_bwd(dy, x, l, lam, u, 0xF, logits=True, renorm=True)
    for n in (0, 1):  # T2B, B2T: positions are columns
        assert not dl[n, 0, ..., :, 0].any() and not dl[n, 2, ..., :, -1].any()
    for n in (2, 3):  # L2R, R2L: positions are rows
        assert not dl[n, 0, ..., 0, :].any() and not dl[n, 2, ..., -1, :].any()


def test_renorm_requires_logits():
    _, x, w, lam, u = general(1, 1, 3, 3, 1)
    with pytest.raises(ValueError):
        O.scan_fwd(x, w, lam, u, 1, renorm=True)


# ---------------------------------------------------------------------------
# per-direction lam, u and outputs
# ---------------------------------------------------------------------------
def test_unmerged_outputs_sum_to_the_merged_output():
    _, x, w, lam, u = general(2, 2, 5, 6, 4)
    ys = O.scan_fwd(x, w, lam, u, 0xF, y_per_dir=True)
    assert ys.shape == (4, 2, 2, 5, 6)
    np.testing.assert_allclose(ys.sum(0), O.scan_fwd(x, w, lam, u, 0xF), rtol=1e-13, atol=1e-13)


def test_per_direction_maps_equal_single_direction_runs():
    dy, x, w, _, _ = general(1, 2, 6, 5, 4)
    lam = RNG.uniform(0, 1, (4, 1, 2, 6, 5))
    u = RNG.standard_normal((4, 1, 2, 6, 5))
    ys = O.scan_fwd(x, w, lam, u, 0xF, lam_per_dir=True, u_per_dir=True, y_per_dir=True)
    for n, d in enumerate(O.ALL_DIRS):
        ref = O.scan_fwd(x, w[n:n + 1], lam[n], u[n], d)
        np.testing.assert_allclose(ys[n], ref, rtol=1e-14, atol=1e-14)
    merged = O.scan_fwd(x, w, lam, u, 0xF, lam_per_dir=True, u_per_dir=True)
    np.testing.assert_allclose(merged, ys.sum(0), rtol=1e-13, atol=1e-13)


def test_identical_per_direction_maps_equal_shared_maps():
    dy, x, w, lam, u = general(1, 2, 5, 5, 4)
    lam4, u4 = np.stack([lam] * 4), np.stack([u] * 4)
    ref = O.scan_fwd(x, w, lam, u, 0xF)
    np.testing.assert_allclose(O.scan_fwd(x, w, lam4, u4, 0xF, lam_per_dir=True, u_per_dir=True), ref,
                               rtol=1e-13, atol=1e-13)
    g = O.scan_bwd(dy, x, w, lam, u, 0xF)
    g4 = O.scan_bwd(dy, x, w, lam4, u4, 0xF, lam_per_dir=True, u_per_dir=True)
    np.testing.assert_allclose(g4[0], g[0], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(g4[1], g[1], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(g4[2].sum(0), g[2], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(g4[3].sum(0), g[3], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("flags", [(True, False, False), (False, True, False), (False, False, True),
                                   (True, True, True), (False, True, True)])
def test_per_direction_finite_differences_and_euler(flags):
    lpd, upd, ypd = flags
    mask, n = 0xB, 3
    _, x, w, lam, u = general(1, 2, 4, 5, n)
    if lpd:
        lam = RNG.uniform(-0.5, 1.5, (n,) + x.shape)
    if upd:
        u = RNG.standard_normal((n,) + x.shape)
    dy = RNG.standard_normal(((n,) if ypd else ()) + x.shape)
    kw = dict(lam_per_dir=lpd, u_per_dir=upd, y_per_dir=ypd)
    grads = O.scan_bwd(dy, x, w, lam, u, mask, group_h=2, **kw)
    loss = lambda x_, w_, l_, u_: float((dy * O.scan_fwd(x_, w_, l_, u_, mask, group_h=2, **kw)).sum())
    _fd_check(loss, [x, w, lam, u], list(grads))
    L = loss(x, w, lam, u)
    for g, v in ((grads[0], x), (grads[2], lam), (grads[3], u)):
        assert abs(float((g * v).sum()) - L) < 1e-11 * max(1.0, abs(L))
