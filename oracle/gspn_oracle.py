"""Float64 CPU oracle for the GSPN 2D line-scan propagation.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call this
module: only the tests, the smoke check and the benchmark's CPU-baseline leg use
it.  It shares no code with the HIP library or its Python binding.

What it computes (paper: Sec. 3.1, Eq. 1-2 and 3-4; Sec. 3.3; supplementary
Eq. 7-9; App. "CUDA Implementation", Alg. 1-2):

  For every (b, c) plane and every direction d of the mask, lines are visited in
  the direction's order.  With h of the line before the first one equal to 0,

      h[line][p] = sum_k w_{d,k}[line][p] * hprev[p + k - 1] + lam[line][p] * x[line][p]

  where p runs along the line, hprev is h of the previously visited line and a
  neighbour outside the line contributes 0 (its weight is lost).  The output is

      y = u * sum_d h_d                                        (Eq. 2, summed over d)

  Weights belong to the receiving pixel and are stored in image coordinates;
  k = 0, 1, 2 is the neighbour at offset -1, 0, +1 along the line coordinate
  (column index for T2B/B2T, row index for L2R/R2L).

  Direction   lines in order       neighbours of (i, j), k = 0, 1, 2
  T2B         rows 0 .. H-1        (i-1, j-1), (i-1, j), (i-1, j+1)
  B2T         rows H-1 .. 0        (i+1, j-1), (i+1, j), (i+1, j+1)
  L2R         cols 0 .. W-1        (i-1, j-1), (i, j-1), (i+1, j-1)
  R2L         cols W-1 .. 0        (i-1, j+1), (i, j+1), (i+1, j+1)

The backward is the exact adjoint of that linear recurrence for the loss
<dy, y>: the reverse scan g = u*dy + (transposed tridiagonal of the next line) g,
then dx = lam * sum_d g_d, dlam = x * sum_d g_d, du = dy * sum_d h_d and
dw_{d,k} = g_d * (neighbour k of the previous line's h_d).

Readings of the paper that this file follows (each listed in the design notes):
  * the first line gets lam*x too (h before the first line is 0), Eq. 3 diagonal blocks;
  * zero padding at the ends of a line, weights are not renormalised there;
  * lam and u are shared by all directions; directions are merged by summation;
  * the adjoint "future contributions" of Alg. 2 are the transposed stencil of
    the next line's weights.

Directions are written out one by one; none is derived from another by flipping
or transposing (that equivalence is checked by the tests instead).
"""
from __future__ import annotations

import numpy as np

T2B, B2T, L2R, R2L = 1, 2, 4, 8
ALL_DIRS = (T2B, B2T, L2R, R2L)


def dirs_of(mask: int) -> list[int]:
    """Directions in increasing bit order: the order w and dw are packed in."""
    if not 1 <= mask <= 15:
        raise ValueError("mask must be in [1, 15]")
    return [d for d in ALL_DIRS if mask & d]


# ---------------------------------------------------------------------------
# shifts along the line coordinate with zero fill
# ---------------------------------------------------------------------------
def _from_lower(v):
    """out[..., p] = v[..., p-1], 0 at p = 0 (the k = 0 neighbour)."""
    out = np.zeros_like(v)
    out[..., 1:] = v[..., :-1]
    return out


def _from_higher(v):
    """out[..., p] = v[..., p+1], 0 at the last p (the k = 2 neighbour)."""
    out = np.zeros_like(v)
    out[..., :-1] = v[..., 1:]
    return out


# ---------------------------------------------------------------------------
# forward, one direction: Eq. 1 (rows), and the same recurrence along columns
# ---------------------------------------------------------------------------
def scan_direction(x, w3, lam, direction):
    """h_d for one direction.  x, lam: (..., H, W); w3: (3, ..., H, W).  float64."""
    x = np.asarray(x, dtype=np.float64)
    lam = np.asarray(lam, dtype=np.float64)
    w3 = np.asarray(w3, dtype=np.float64)
    H, W = x.shape[-2:]
    h = np.zeros_like(x)
    lx = lam * x
    if direction == T2B:
        prev = np.zeros(x.shape[:-2] + (W,))
        for i in range(H):
            h[..., i, :] = (w3[0][..., i, :] * _from_lower(prev) + w3[1][..., i, :] * prev
                            + w3[2][..., i, :] * _from_higher(prev) + lx[..., i, :])
            prev = h[..., i, :]
    elif direction == B2T:
        prev = np.zeros(x.shape[:-2] + (W,))
        for i in range(H - 1, -1, -1):
            h[..., i, :] = (w3[0][..., i, :] * _from_lower(prev) + w3[1][..., i, :] * prev
                            + w3[2][..., i, :] * _from_higher(prev) + lx[..., i, :])
            prev = h[..., i, :]
    elif direction == L2R:
        prev = np.zeros(x.shape[:-2] + (H,))
        for j in range(W):
            h[..., :, j] = (w3[0][..., :, j] * _from_lower(prev) + w3[1][..., :, j] * prev
                            + w3[2][..., :, j] * _from_higher(prev) + lx[..., :, j])
            prev = h[..., :, j]
    elif direction == R2L:
        prev = np.zeros(x.shape[:-2] + (H,))
        for j in range(W - 1, -1, -1):
            h[..., :, j] = (w3[0][..., :, j] * _from_lower(prev) + w3[1][..., :, j] * prev
                            + w3[2][..., :, j] * _from_higher(prev) + lx[..., :, j])
            prev = h[..., :, j]
    else:
        raise ValueError(direction)
    return h


def scan_fwd_dirs(x, w, lam, mask):
    """List of h_d, one per direction of the mask (w packed [n][3][..., H, W])."""
    ds = dirs_of(mask)
    w = np.asarray(w, dtype=np.float64)
    if w.shape[0] != len(ds) or w.shape[1] != 3:
        raise ValueError("w must be [n_dirs][3][..., H, W]")
    return [scan_direction(x, w[n], lam, d) for n, d in enumerate(ds)]


def scan_fwd(x, w, lam, u, mask):
    """y = u * sum_d h_d   (Eq. 2 with the directions merged by summation)."""
    hs = scan_fwd_dirs(x, w, lam, mask)
    total = np.zeros_like(hs[0])
    for h in hs:
        total = total + h
    return np.asarray(u, dtype=np.float64) * total


# ---------------------------------------------------------------------------
# backward: adjoint of the recurrence for one direction
# ---------------------------------------------------------------------------
def _neighbours_prev(h, direction):
    """For each pixel, the three neighbours in the previously visited line (0 if none).

    Returns an array (3, ..., H, W) with entry k = h at neighbour k of the pixel.
    """
    H, W = h.shape[-2:]
    out = np.zeros((3,) + h.shape)
    if direction == T2B:
        for i in range(1, H):
            prev = h[..., i - 1, :]
            out[0][..., i, :] = _from_lower(prev)
            out[1][..., i, :] = prev
            out[2][..., i, :] = _from_higher(prev)
    elif direction == B2T:
        for i in range(H - 1):
            prev = h[..., i + 1, :]
            out[0][..., i, :] = _from_lower(prev)
            out[1][..., i, :] = prev
            out[2][..., i, :] = _from_higher(prev)
    elif direction == L2R:
        for j in range(1, W):
            prev = h[..., :, j - 1]
            out[0][..., :, j] = _from_lower(prev)
            out[1][..., :, j] = prev
            out[2][..., :, j] = _from_higher(prev)
    elif direction == R2L:
        for j in range(W - 1):
            prev = h[..., :, j + 1]
            out[0][..., :, j] = _from_lower(prev)
            out[1][..., :, j] = prev
            out[2][..., :, j] = _from_higher(prev)
    else:
        raise ValueError(direction)
    return out


def adjoint_direction(src, w3, direction):
    """g_d = (I - M_d)^{-T} src, by the reverse scan.

    A pixel q of the line after p (in scan order) received w_k[q] * h[p] when p is
    q's neighbour k, i.e. p = q + (k - 1) along the line.  So
        g[p] = src[p] + sum_k w_k[q = p - (k - 1)] * g[q = p - (k - 1)].
    """
    src = np.asarray(src, dtype=np.float64)
    w3 = np.asarray(w3, dtype=np.float64)
    H, W = src.shape[-2:]
    g = np.zeros_like(src)

    def back(nxt_w, nxt_g):
        # contribution to position p of the current line from the next line:
        # k=0: q = p + 1, k=1: q = p, k=2: q = p - 1
        a0 = nxt_w[0] * nxt_g
        a1 = nxt_w[1] * nxt_g
        a2 = nxt_w[2] * nxt_g
        return _from_higher(a0) + a1 + _from_lower(a2)

    if direction == T2B:  # forward order rows 0..H-1, adjoint runs H-1..0
        g[..., H - 1, :] = src[..., H - 1, :]
        for i in range(H - 2, -1, -1):
            g[..., i, :] = src[..., i, :] + back(w3[:, ..., i + 1, :], g[..., i + 1, :])
    elif direction == B2T:  # forward rows H-1..0, adjoint 0..H-1
        g[..., 0, :] = src[..., 0, :]
        for i in range(1, H):
            g[..., i, :] = src[..., i, :] + back(w3[:, ..., i - 1, :], g[..., i - 1, :])
    elif direction == L2R:  # forward cols 0..W-1, adjoint W-1..0
        g[..., :, W - 1] = src[..., :, W - 1]
        for j in range(W - 2, -1, -1):
            g[..., :, j] = src[..., :, j] + back(w3[:, ..., :, j + 1], g[..., :, j + 1])
    elif direction == R2L:  # forward cols W-1..0, adjoint 0..W-1
        g[..., :, 0] = src[..., :, 0]
        for j in range(1, W):
            g[..., :, j] = src[..., :, j] + back(w3[:, ..., :, j - 1], g[..., :, j - 1])
    else:
        raise ValueError(direction)
    return g


def scan_bwd(dy, x, w, lam, u, mask):
    """Gradients of L = <dy, y> with respect to x, w, lam and u.

    Returns (dx, dw, dlam, du) with dw packed like w: [n][3][..., H, W].
    """
    dy = np.asarray(dy, dtype=np.float64)
    x = np.asarray(x, dtype=np.float64)
    lam = np.asarray(lam, dtype=np.float64)
    u = np.asarray(u, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    ds = dirs_of(mask)
    src = u * dy  # dL/dh_d, identical for every direction
    g_sum = np.zeros_like(x)
    h_sum = np.zeros_like(x)
    dw = np.zeros_like(w)
    for n, d in enumerate(ds):
        h = scan_direction(x, w[n], lam, d)
        g = adjoint_direction(src, w[n], d)
        nb = _neighbours_prev(h, d)
        for k in range(3):
            dw[n, k] = g * nb[k]
        g_sum = g_sum + g
        h_sum = h_sum + h
    dx = lam * g_sum
    dlam = x * g_sum
    du = dy * h_sum
    return dx, dw, dlam, du


# ---------------------------------------------------------------------------
# dense forms for tiny planes (Eq. 3 and supplementary Eq. 8-9)
# ---------------------------------------------------------------------------
def line_matrix(w3_line):
    """The tridiagonal n x n matrix w_i of one line: row p holds w_k[p] at column p+k-1."""
    n = w3_line.shape[-1]
    m = np.zeros((n, n))
    for p in range(n):
        for k in range(3):
            q = p + k - 1
            if 0 <= q < n:
                m[p, q] = w3_line[k, p]
    return m


def g_blocks_t2b(w3, lam):
    """Block matrix G of Eq. 3 for one plane scanned top to bottom.

    w3: (3, H, W) and lam: (H, W).  Block (i, j), j <= i, is
    w_i w_{i-1} ... w_{j+1} diag(lam_j) (the newest line's matrix on the left).
    Returns the dense (H*W, H*W) matrix with rows/cols in row-major pixel order.
    """
    H, W = lam.shape
    G = np.zeros((H * W, H * W))
    mats = [line_matrix(w3[:, i, :]) for i in range(H)]
    for i in range(H):
        for j in range(i + 1):
            # product w_i w_{i-1} ... w_{j+1}
            P = np.eye(W)
            for tau in range(i, j, -1):
                P = P @ mats[tau]
            G[i * W:(i + 1) * W, j * W:(j + 1) * W] = P @ np.diag(lam[j])
    return G
