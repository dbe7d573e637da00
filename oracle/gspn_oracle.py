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

Options (each optional, default off):

  * local GSPN (Sec. 4.1 "Local vs Global GSPN"; App. "CUDA Implementation":
    the scan axis of Alg. 1 is cut into groups of kNItems lines): with a group
    length G the lines of a direction's scan axis form the groups
    [k G, (k+1) G) in image coordinates (the last one may be shorter); the
    state before the first line a direction visits in each group is 0, so no
    weight links a group to the one before it.  group_h applies to the row
    scans (T2B, B2T), group_w to the column scans (L2R, R2L);
  * weight normalisation (Sec. 3.3, Eq. 6): w holds logits l and each pixel
    uses w_k = sigmoid(l_k) / sum_k' sigmoid(l_k'); the sum runs over the three
    neighbours, or, with edge renormalisation, over the neighbours that lie on
    the line (the m_i non-zero entries of row i of the tridiagonal matrix).
    dw is then the gradient with respect to the logits;
  * per-direction lam and u (one map per direction, stacked like w), and
    unmerged outputs y_d = u_d * h_d.

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


def _starts_group(line, n, group, reverse):
    """True when `line` (of n lines) is the first line a scan visits in its group.

    Forward scans (T2B, L2R) enter a group [kG, (k+1)G) at its lowest index,
    reverse scans (B2T, R2L) at its highest one (or at the last line).
    """
    if not group or group >= n:
        return line == (n - 1 if reverse else 0)
    if reverse:
        return line == n - 1 or (line + 1) % group == 0
    return line % group == 0


# ---------------------------------------------------------------------------
# forward, one direction: Eq. 1 (rows), and the same recurrence along columns
# ---------------------------------------------------------------------------
def scan_direction(x, w3, lam, direction, group=0):
    """h_d for one direction.  x, lam: (..., H, W); w3: (3, ..., H, W).  float64.

    group: local-GSPN group length along the scan axis (0 = global).
    """
    x = np.asarray(x, dtype=np.float64)
    lam = np.asarray(lam, dtype=np.float64)
    w3 = np.asarray(w3, dtype=np.float64)
    H, W = x.shape[-2:]
    h = np.zeros_like(x)
    lx = lam * x
    if direction == T2B:
        prev = np.zeros(x.shape[:-2] + (W,))
        for i in range(H):
            if _starts_group(i, H, group, False):
                prev = np.zeros_like(prev)
            h[..., i, :] = (w3[0][..., i, :] * _from_lower(prev) + w3[1][..., i, :] * prev
                            + w3[2][..., i, :] * _from_higher(prev) + lx[..., i, :])
            prev = h[..., i, :]
    elif direction == B2T:
        prev = np.zeros(x.shape[:-2] + (W,))
        for i in range(H - 1, -1, -1):
            if _starts_group(i, H, group, True):
                prev = np.zeros_like(prev)
            h[..., i, :] = (w3[0][..., i, :] * _from_lower(prev) + w3[1][..., i, :] * prev
                            + w3[2][..., i, :] * _from_higher(prev) + lx[..., i, :])
            prev = h[..., i, :]
    elif direction == L2R:
        prev = np.zeros(x.shape[:-2] + (H,))
        for j in range(W):
            if _starts_group(j, W, group, False):
                prev = np.zeros_like(prev)
            h[..., :, j] = (w3[0][..., :, j] * _from_lower(prev) + w3[1][..., :, j] * prev
                            + w3[2][..., :, j] * _from_higher(prev) + lx[..., :, j])
            prev = h[..., :, j]
    elif direction == R2L:
        prev = np.zeros(x.shape[:-2] + (H,))
        for j in range(W - 1, -1, -1):
            if _starts_group(j, W, group, True):
                prev = np.zeros_like(prev)
            h[..., :, j] = (w3[0][..., :, j] * _from_lower(prev) + w3[1][..., :, j] * prev
                            + w3[2][..., :, j] * _from_higher(prev) + lx[..., :, j])
            prev = h[..., :, j]
    else:
        raise ValueError(direction)
    return h


def _vertical(direction):
    return direction in (T2B, B2T)


# ---------------------------------------------------------------------------
# weight normalisation of Eq. 6 (logits -> row-stochastic tridiagonal rows)
# ---------------------------------------------------------------------------
def _neighbour_mask(shape, direction, renorm):
    """m[k] = 1 where neighbour k of the pixel counts in the normalisation.

    Without edge renormalisation all three count.  With it, only neighbours
    that lie on the line: k = 0 (offset -1) is missing at the first position of
    a line, k = 2 (offset +1) at the last one.  The position along the line is
    the column for T2B/B2T and the row for L2R/R2L.
    """
    m = np.ones((3,) + tuple(shape))
    if renorm:
        if _vertical(direction):
            m[0][..., :, 0] = 0.0
            m[2][..., :, -1] = 0.0
        else:
            m[0][..., 0, :] = 0.0
            m[2][..., -1, :] = 0.0
    return m


def _sigmoid(v):
    return 1.0 / (1.0 + np.exp(-v))


def normalize_logits(l3, direction, renorm=False):
    """Eq. 6: w_k = sigmoid(l_k) / sum over the counted k' of sigmoid(l_k')."""
    l3 = np.asarray(l3, dtype=np.float64)
    m = _neighbour_mask(l3.shape[1:], direction, renorm)
    s = m * _sigmoid(l3)
    return s / s.sum(axis=0, keepdims=True)


def normalize_logits_vjp(l3, dw3, direction, renorm=False):
    """Gradient with respect to the logits, given the gradient dw3 of the weights.

    With s_k = m_k sigmoid(l_k), S = sum_k s_k and w_k = s_k / S:
    dw_j/dl_k = m_k sigmoid'(l_k) (delta_jk - w_j) / S, so
    dl_k = m_k sigmoid(l_k) (1 - sigmoid(l_k)) (dw_k - sum_j w_j dw_j) / S.
    """
    l3 = np.asarray(l3, dtype=np.float64)
    dw3 = np.asarray(dw3, dtype=np.float64)
    m = _neighbour_mask(l3.shape[1:], direction, renorm)
    sg = _sigmoid(l3)
    s = m * sg
    S = s.sum(axis=0, keepdims=True)
    w = s / S
    inner = (w * dw3).sum(axis=0, keepdims=True)
    return m * sg * (1.0 - sg) * (dw3 - inner) / S


def _dir_weights(w, n, d, logits, renorm):
    return normalize_logits(w[n], d, renorm) if logits else w[n]


def scan_fwd_dirs(x, w, lam, mask, group_h=0, group_w=0, logits=False, renorm=False,
                  lam_per_dir=False):
    """List of h_d, one per direction of the mask (w packed [n][3][..., H, W])."""
    ds = dirs_of(mask)
    w = np.asarray(w, dtype=np.float64)
    lam = np.asarray(lam, dtype=np.float64)
    if w.shape[0] != len(ds) or w.shape[1] != 3:
        raise ValueError("w must be [n_dirs][3][..., H, W]")
    if renorm and not logits:
        raise ValueError("edge renormalisation applies to logits")
    return [scan_direction(x, _dir_weights(w, n, d, logits, renorm), lam[n] if lam_per_dir else lam,
                           d, group_h if _vertical(d) else group_w)
            for n, d in enumerate(ds)]


def scan_fwd(x, w, lam, u, mask, group_h=0, group_w=0, logits=False, renorm=False,
             lam_per_dir=False, u_per_dir=False, y_per_dir=False):
    """y = u * sum_d h_d   (Eq. 2 with the directions merged by summation).

    With u_per_dir, y = sum_d u_d * h_d; with y_per_dir the stacked y_d = u_d * h_d.
    """
    hs = scan_fwd_dirs(x, w, lam, mask, group_h, group_w, logits, renorm, lam_per_dir)
    u = np.asarray(u, dtype=np.float64)
    if y_per_dir:
        return np.stack([(u[n] if u_per_dir else u) * h for n, h in enumerate(hs)])
    if u_per_dir:
        total = np.zeros_like(hs[0])
        for n, h in enumerate(hs):
            total = total + u[n] * h
        return total
    total = np.zeros_like(hs[0])
    for h in hs:
        total = total + h
    return u * total


# ---------------------------------------------------------------------------
# backward: adjoint of the recurrence for one direction
# ---------------------------------------------------------------------------
def _neighbours_prev(h, direction, group=0):
    """For each pixel, the three neighbours in the previously visited line (0 if
    none: before the first line, and before the first line of a group).

    Returns an array (3, ..., H, W) with entry k = h at neighbour k of the pixel.
    """
    H, W = h.shape[-2:]
    out = np.zeros((3,) + h.shape)
    if direction == T2B:
        for i in range(1, H):
            if _starts_group(i, H, group, False):
                continue
            prev = h[..., i - 1, :]
            out[0][..., i, :] = _from_lower(prev)
            out[1][..., i, :] = prev
            out[2][..., i, :] = _from_higher(prev)
    elif direction == B2T:
        for i in range(H - 1):
            if _starts_group(i, H, group, True):
                continue
            prev = h[..., i + 1, :]
            out[0][..., i, :] = _from_lower(prev)
            out[1][..., i, :] = prev
            out[2][..., i, :] = _from_higher(prev)
    elif direction == L2R:
        for j in range(1, W):
            if _starts_group(j, W, group, False):
                continue
            prev = h[..., :, j - 1]
            out[0][..., :, j] = _from_lower(prev)
            out[1][..., :, j] = prev
            out[2][..., :, j] = _from_higher(prev)
    elif direction == R2L:
        for j in range(W - 1):
            if _starts_group(j, W, group, True):
                continue
            prev = h[..., :, j + 1]
            out[0][..., :, j] = _from_lower(prev)
            out[1][..., :, j] = prev
            out[2][..., :, j] = _from_higher(prev)
    else:
        raise ValueError(direction)
    return out


def adjoint_direction(src, w3, direction, group=0):
    """g_d = (I - M_d)^{-T} src, by the reverse scan.

    A pixel q of the line after p (in scan order) received w_k[q] * h[p] when p is
    q's neighbour k, i.e. p = q + (k - 1) along the line.  So
        g[p] = src[p] + sum_k w_k[q = p - (k - 1)] * g[q = p - (k - 1)].
    When the line after p starts a group, it received nothing from p: g[p] = src[p].
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
            g[..., i, :] = src[..., i, :]
            if not _starts_group(i + 1, H, group, False):
                g[..., i, :] += back(w3[:, ..., i + 1, :], g[..., i + 1, :])
    elif direction == B2T:  # forward rows H-1..0, adjoint 0..H-1
        g[..., 0, :] = src[..., 0, :]
        for i in range(1, H):
            g[..., i, :] = src[..., i, :]
            if not _starts_group(i - 1, H, group, True):
                g[..., i, :] += back(w3[:, ..., i - 1, :], g[..., i - 1, :])
    elif direction == L2R:  # forward cols 0..W-1, adjoint W-1..0
        g[..., :, W - 1] = src[..., :, W - 1]
        for j in range(W - 2, -1, -1):
            g[..., :, j] = src[..., :, j]
            if not _starts_group(j + 1, W, group, False):
                g[..., :, j] += back(w3[:, ..., :, j + 1], g[..., :, j + 1])
    elif direction == R2L:  # forward cols W-1..0, adjoint 0..W-1
        g[..., :, 0] = src[..., :, 0]
        for j in range(1, W):
            g[..., :, j] = src[..., :, j]
            if not _starts_group(j - 1, W, group, True):
                g[..., :, j] += back(w3[:, ..., :, j - 1], g[..., :, j - 1])
    else:
        raise ValueError(direction)
    return g


def scan_bwd(dy, x, w, lam, u, mask, group_h=0, group_w=0, logits=False, renorm=False,
             lam_per_dir=False, u_per_dir=False, y_per_dir=False):
    """Gradients of L = <dy, y> with respect to x, w, lam and u.

    Returns (dx, dw, dlam, du) with dw packed like w: [n][3][..., H, W] (with
    logits: the gradient with respect to the logits); dlam and du are stacked
    per direction when lam or u is.  dy is stacked per direction with y_per_dir.
    """
    dy = np.asarray(dy, dtype=np.float64)
    x = np.asarray(x, dtype=np.float64)
    lam = np.asarray(lam, dtype=np.float64)
    u = np.asarray(u, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    ds = dirs_of(mask)
    if renorm and not logits:
        raise ValueError("edge renormalisation applies to logits")
    per_dir = lam_per_dir or u_per_dir or y_per_dir
    g_sum = np.zeros_like(x)   # sum_d g_d (shared lam)
    lg_sum = np.zeros_like(x)  # sum_d lam_d g_d
    h_sum = np.zeros_like(x)   # sum_d dy_d h_d (shared u)
    dw = np.zeros_like(w)
    dlam = np.zeros_like(lam)
    du = np.zeros_like(u)
    for n, d in enumerate(ds):
        group = group_h if _vertical(d) else group_w
        w3 = _dir_weights(w, n, d, logits, renorm)
        lam_d = lam[n] if lam_per_dir else lam
        u_d = u[n] if u_per_dir else u
        dy_d = dy[n] if y_per_dir else dy
        h = scan_direction(x, w3, lam_d, d, group)
        g = adjoint_direction(u_d * dy_d, w3, d, group)  # dL/dh_d = u_d dy_d
        nb = _neighbours_prev(h, d, group)
        dw3 = np.stack([g * nb[k] for k in range(3)])
        dw[n] = normalize_logits_vjp(w[n], dw3, d, renorm) if logits else dw3
        if not per_dir:
            g_sum = g_sum + g
            h_sum = h_sum + h
            continue
        lg_sum = lg_sum + lam_d * g
        if lam_per_dir:
            dlam[n] = x * g
        else:
            g_sum = g_sum + g
        if u_per_dir:
            du[n] = dy_d * h
        else:
            h_sum = h_sum + dy_d * h
    if not per_dir:
        return lam * g_sum, dw, x * g_sum, dy * h_sum
    if not lam_per_dir:
        dlam = x * g_sum
    if not u_per_dir:
        du = h_sum
    return lg_sum, dw, dlam, du


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
