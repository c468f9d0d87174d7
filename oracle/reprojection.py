"""Reprojection + visibility oracle (Sec. 4.3, Eq. reprojection, Eq. visibility,
design choice (iii)).

For a query token p of target frame t and a retrieved (source) frame s:

    X_t = z_p K_t^{-1} u~_p
    X_s = R_s^T (R_t X_t + c_t - c_s)
    u^_s(p) = pi(K_s X_s)

and the correspondence is kept only if [X_s]_z <= (1 + eps) D_s(u^_s(p)).

Readings fixed here (the paper states the equations on the token grid but
not these details):

* token (row i, col j) has centre u_p = (j + 1/2, i + 1/2) in token units;
  token cell [j, j+1) x [i, i+1) covers latent pixels [p j, p j + p) x
  [p i, p i + p);
* K on the token grid is the depth-map intrinsics divided by p:
  (fx/p, fy/p, cx/p, cy/p);
* z_p = D_t(u_p) is the mean of the token's p x p depth pixels (for p = 2
  this equals bilinear depth at the token centre), summed row by row, left to
  right; D_s(u^) is the same pooled depth of the token cell containing u^;
* K_t^{-1} u~ is ((u_x - cx)/fx, (u_y - cy)/fy, 1); pi(K_s X) divides the
  first two entries of K_s X = (fx X + cx Z, fy Y + cy Z, Z) by the third;
* rejection reasons (design choice (iii) lists them): -1 depth undefined
  (z_p not finite or <= 0), -2 behind the source camera ([X_s]_z <= 0),
  -3 off the source grid (not 0 <= u^_x < w and 0 <= u^_y < h),
  -4 occluded (Eq. visibility fails, including NaN source depth),
  -5 no source frame (a retrieved slot left empty); otherwise the key index
  floor(u^_y) w + floor(u^_x) within the source frame;
* rejection is per (query token, source frame): a token rejected in one
  retrieved frame may still be biased towards another.

The output u^ is rounded to fp32 for tokens with reason >= 0, -3 or -4 and
is NaN for -1, -2 and -5.

``rotation_pair`` / ``reproject_rotation`` state the fixed-centre case of
Eq. reprojection (the rotation / zoom homography of Sec. 4.3) as its own
depth-free path; see their docstrings for the reading taken.
"""

from __future__ import annotations

import numpy as np

UNDEFINED, BEHIND, OFF_GRID, OCCLUDED, NO_SOURCE = -1, -2, -3, -4, -5
CENTRE_MOVED = -6  # rotation-only path: the source's centre is not the target's


def pooled_depth(depth, p):
    """Mean of each p x p block of a depth map [..., h*p, w*p] -> [..., h, w],
    summed row-major (row a, then column b) then divided by p*p."""
    d = np.asarray(depth, dtype=np.float64)
    acc = None
    for a in range(p):
        for b in range(p):
            blk = d[..., a::p, b::p]
            acc = blk.copy() if acc is None else acc + blk
    return acc / float(p * p)


def token_intrinsics(K, p):
    """(fx, fy, cx, cy) on the token grid: depth-map intrinsics / p."""
    K = np.asarray(K, dtype=np.float64)
    return K[..., 0] / p, K[..., 1] / p, K[..., 2] / p, K[..., 3] / p


def reproject_pair(tgt_depth, tgt_c2w, tgt_K, src_depth, src_c2w, src_K, p, eps):
    """Correspondence of every token of ONE target frame into ONE source frame.

    tgt_depth, src_depth: [h*p, w*p]; c2w: [4, 4]; K: [4] (depth-map px).
    Returns (uv [h*w, 2] float32, idx [h*w] int32), tokens row-major."""
    return _pair(tgt_depth, tgt_c2w, tgt_K, src_depth, src_c2w, src_K, p, eps)[:2]


def _pair(tgt_depth, tgt_c2w, tgt_K, src_depth, src_c2w, src_K, p, eps):
    """``reproject_pair`` plus, per token, [X_s]_z, D_s(u^) (0 off the grid) and
    the on-grid mask, for the visibility diagnostics."""
    zt = pooled_depth(tgt_depth, p)
    zs_map = pooled_depth(src_depth, p)
    h, w = zt.shape
    fxt, fyt, cxt, cyt = token_intrinsics(tgt_K, p)
    fxs, fys, cxs, cys = token_intrinsics(src_K, p)
    Mt = np.asarray(tgt_c2w, dtype=np.float64)
    Ms = np.asarray(src_c2w, dtype=np.float64)
    Rt, ct = Mt[:3, :3], Mt[:3, 3]
    Rs, cs = Ms[:3, :3], Ms[:3, 3]

    ii, jj = np.meshgrid(np.arange(h), np.arange(w), indexing="ij")
    ux = jj.astype(np.float64) + 0.5
    uy = ii.astype(np.float64) + 0.5
    z = zt

    # X_t = z K_t^{-1} u~
    Xt = ((ux - cxt) / fxt) * z
    Yt = ((uy - cyt) / fyt) * z
    Zt = z
    # R_t X_t + c_t - c_s, left to right
    W = [((Rt[r, 0] * Xt + Rt[r, 1] * Yt) + Rt[r, 2] * Zt) + ct[r] - cs[r] for r in range(3)]
    # X_s = R_s^T (...): component r is column r of R_s dotted with W
    Xs, Ys, Zs = [(Rs[0, r] * W[0] + Rs[1, r] * W[1]) + Rs[2, r] * W[2] for r in range(3)]
    # pi(K_s X_s)
    h0 = fxs * Xs + cxs * Zs
    h1 = fys * Ys + cys * Zs
    with np.errstate(divide="ignore", invalid="ignore", over="ignore"):
        uhx = h0 / Zs
        uhy = h1 / Zs

    defined = np.isfinite(z) & (z > 0)
    front = defined & (Zs > 0)
    with np.errstate(invalid="ignore"):
        on_grid = front & (uhx >= 0) & (uhx < w) & (uhy >= 0) & (uhy < h)
    kx = np.where(on_grid, np.floor(np.where(on_grid, uhx, 0.0)), 0).astype(np.int64)
    ky = np.where(on_grid, np.floor(np.where(on_grid, uhy, 0.0)), 0).astype(np.int64)
    Ds = zs_map[ky, kx]
    tol = 1.0 + np.float64(np.float32(eps))
    with np.errstate(invalid="ignore"):
        visible = on_grid & (Zs <= tol * Ds)

    idx = np.where(visible, ky * w + kx, OCCLUDED)
    idx = np.where(on_grid, idx, OFF_GRID)
    idx = np.where(front, idx, BEHIND)
    idx = np.where(defined, idx, UNDEFINED)

    uv = np.stack([uhx, uhy], axis=-1)
    uv[~front] = np.nan
    n = h * w
    return (uv.reshape(n, 2).astype(np.float32), idx.reshape(n).astype(np.int32), Zs.reshape(n),
            np.where(on_grid, Ds, 0.0).reshape(n), on_grid.reshape(n))


def visibility_near_ties(tgt_depth, tgt_c2w, tgt_K, src_depth, src_c2w, src_K, p, eps, src_sel=None, rel=1e-9):
    """Diagnostic of Eq. visibility: the number of (source frame, query token)
    pairs on the source grid whose test is a near tie,
    |[X_s]_z - (1 + eps) D_s(u^)| < rel D_s(u^). Same inputs as ``reproject``.
    A mismatch of the visibility decision between two exact evaluations can
    only occur at such a pair; the parity tests report the count."""
    tgt_depth = np.asarray(tgt_depth)
    Tq = tgt_depth.shape[0]
    S = len(src_sel) if src_sel is not None else np.asarray(src_depth).shape[0]
    tol = 1.0 + np.float64(np.float32(eps))
    count = 0
    for s in range(S):
        f = s if src_sel is None else int(src_sel[s])
        if f < 0:
            continue
        for t in range(Tq):
            _, _, Zs, Ds, on_grid = _pair(tgt_depth[t], tgt_c2w[t], tgt_K[t], src_depth[f], src_c2w[f], src_K[f], p,
                                          eps)
            with np.errstate(invalid="ignore"):
                count += int(np.sum(on_grid & (np.abs(Zs - tol * Ds) < rel * Ds)))
    return count


def reproject(tgt_depth, tgt_c2w, tgt_K, src_depth, src_c2w, src_K, p, eps, src_sel=None):
    """All target frames against all source frames.

    tgt_*: [Tq, ...]; src_*: [S, ...] (or a frame bank indexed by ``src_sel``
    [S], negative = no source). Returns uv [S, Tq*h*w, 2] float32 and idx
    [S, Tq*h*w] int32, the query tokens frame-major then row-major."""
    tgt_depth = np.asarray(tgt_depth)
    Tq = tgt_depth.shape[0]
    h, w = tgt_depth.shape[1] // p, tgt_depth.shape[2] // p
    S = len(src_sel) if src_sel is not None else np.asarray(src_depth).shape[0]
    uv = np.full((S, Tq * h * w, 2), np.nan, np.float32)
    idx = np.full((S, Tq * h * w), NO_SOURCE, np.int32)
    for s in range(S):
        f = s if src_sel is None else int(src_sel[s])
        if f < 0:
            continue
        for t in range(Tq):
            u, i = reproject_pair(tgt_depth[t], tgt_c2w[t], tgt_K[t], src_depth[f], src_c2w[f], src_K[f], p, eps)
            uv[s, t * h * w:(t + 1) * h * w] = u
            idx[s, t * h * w:(t + 1) * h * w] = i
    return uv, idx


def rotation_pair(tgt_c2w, tgt_K, src_c2w, src_K, h, w, p):
    """Correspondence of every token of ONE target frame into ONE source frame
    that shares its camera centre: the rotation / zoom homography of Sec. 4.3.

    With c_s = c_t the depth z_p scales X_s and cancels under pi, so Eq.
    reprojection reduces to u^ = pi(K_s R_s^T R_t K_t^{-1} u~). This path reads
    no depth: the visibility test of Eq. visibility is not applied (with one
    centre there is no parallax, hence no disocclusion), so the codes are the
    key index, -2 (behind the source camera), -3 (off the grid) or
    CENTRE_MOVED (-6) for every token when the two fp32 centres are not equal.

    The matrix is formed once per frame pair, in this order:
        A = R_s^T R_t          A[r][c] = (Rs[0][r] Rt[0][c] + Rs[1][r] Rt[1][c]) + Rs[2][r] Rt[2][c]
        M = K_s A              rows (fx_s A0 + cx_s A2, fy_s A1 + cy_s A2, A2)
        H = M K_t^{-1}         H[r][0] = M[r][0] / fx_t, H[r][1] = M[r][1] / fy_t,
                               H[r][2] = (M[r][2] - H[r][0] cx_t) - H[r][1] cy_t
    then per token v_r = (H[r][0] u_x + H[r][1] u_y) + H[r][2] and
    u^ = (v_0 / v_2, v_1 / v_2), behind iff v_2 <= 0 (v_2 has the sign of
    [X_s]_z for any positive depth). Intrinsics on the token grid as for
    ``reproject_pair``. Returns (uv [h*w, 2] float32, idx [h*w] int32)."""
    Mt32 = np.asarray(tgt_c2w, dtype=np.float32)
    Ms32 = np.asarray(src_c2w, dtype=np.float32)
    n = h * w
    if not bool(np.all(Mt32[:3, 3] == Ms32[:3, 3])):
        return np.full((n, 2), np.nan, np.float32), np.full(n, CENTRE_MOVED, np.int32)
    fxt, fyt, cxt, cyt = (float(x) for x in token_intrinsics(tgt_K, p))
    fxs, fys, cxs, cys = (float(x) for x in token_intrinsics(src_K, p))
    Rt = Mt32[:3, :3].astype(np.float64)
    Rs = Ms32[:3, :3].astype(np.float64)
    A = [[(Rs[0, r] * Rt[0, c] + Rs[1, r] * Rt[1, c]) + Rs[2, r] * Rt[2, c] for c in range(3)] for r in range(3)]
    M = [[fxs * A[0][c] + cxs * A[2][c] for c in range(3)],
         [fys * A[1][c] + cys * A[2][c] for c in range(3)],
         [A[2][c] for c in range(3)]]
    H = []
    for r in range(3):
        h0 = M[r][0] / fxt
        h1 = M[r][1] / fyt
        H.append((h0, h1, (M[r][2] - h0 * cxt) - h1 * cyt))

    ii, jj = np.meshgrid(np.arange(h), np.arange(w), indexing="ij")
    ux = jj.astype(np.float64) + 0.5
    uy = ii.astype(np.float64) + 0.5
    v0, v1, v2 = [(H[r][0] * ux + H[r][1] * uy) + H[r][2] for r in range(3)]
    with np.errstate(divide="ignore", invalid="ignore", over="ignore"):
        uhx = v0 / v2
        uhy = v1 / v2
    front = v2 > 0
    with np.errstate(invalid="ignore"):
        on_grid = front & (uhx >= 0) & (uhx < w) & (uhy >= 0) & (uhy < h)
    kx = np.where(on_grid, np.floor(np.where(on_grid, uhx, 0.0)), 0).astype(np.int64)
    ky = np.where(on_grid, np.floor(np.where(on_grid, uhy, 0.0)), 0).astype(np.int64)
    idx = np.where(on_grid, ky * w + kx, OFF_GRID)
    idx = np.where(front, idx, BEHIND)
    uv = np.stack([uhx, uhy], axis=-1)
    uv[~front] = np.nan
    return uv.reshape(n, 2).astype(np.float32), idx.reshape(n).astype(np.int32)


def reproject_rotation(tgt_c2w, tgt_K, src_c2w, src_K, h, w, p, src_sel=None):
    """``rotation_pair`` for all target frames against all source frames.

    tgt_*: [Tq, ...]; src_*: [S, ...] (or a frame bank indexed by ``src_sel``
    [S], an entry outside the bank = no source, NO_SOURCE). Returns uv
    [S, Tq*h*w, 2] float32 and idx [S, Tq*h*w] int32."""
    tgt_c2w = np.asarray(tgt_c2w)
    Tq = tgt_c2w.shape[0]
    n_bank = np.asarray(src_c2w).shape[0]
    S = len(src_sel) if src_sel is not None else n_bank
    uv = np.full((S, Tq * h * w, 2), np.nan, np.float32)
    idx = np.full((S, Tq * h * w), NO_SOURCE, np.int32)
    for s in range(S):
        f = s if src_sel is None else int(src_sel[s])
        if f < 0 or f >= n_bank:
            continue
        for t in range(Tq):
            u, i = rotation_pair(tgt_c2w[t], tgt_K[t], src_c2w[f], src_K[f], h, w, p)
            uv[s, t * h * w:(t + 1) * h * w] = u
            idx[s, t * h * w:(t + 1) * h * w] = i
    return uv, idx


def boundary_margin(uv, p, h, w):
    """Distance, in depth-map pixels, from each u^ to the nearest token-cell
    boundary line (including the grid edges 0, w and 0, h). NaN -> inf."""
    uv = np.asarray(uv, dtype=np.float64)
    x, y = uv[..., 0], uv[..., 1]
    with np.errstate(invalid="ignore"):
        mx = np.abs(x - np.round(x))
        my = np.abs(y - np.round(y))
    m = np.minimum(mx, my) * p
    return np.where(np.isfinite(m), m, np.inf)
