"""Pins of the rotation-only correspondence oracle (Sec. 4.3: with a fixed
camera centre, Eq. reprojection reduces to the rotation / zoom homography
pi(K_s R_s^T R_t K_t^{-1} u~)).

The pins are independent of the homography's own arithmetic:
* the general Eq. reprojection (``reproject_pair``, depth and all) on
  shared-centre poses and random depth: depth cancels, so u^ must agree to
  rounding and every non-visibility code must agree;
* closed forms: identity (every token onto itself, exactly), a pure zoom
  about the principal points, a pure yaw (u^_x = c_x + f tan(alpha - theta)),
  a half turn (all behind);
* the path's own definitions: a moved centre gives -6 everywhere, an empty
  slot -5.
"""

from __future__ import annotations

import math

import numpy as np
import pytest

from oracle import reprojection as R


def _rot(axis, ang):
    axis = np.asarray(axis, np.float64)
    axis = axis / np.linalg.norm(axis)
    k = np.array([[0, -axis[2], axis[1]], [axis[2], 0, -axis[0]], [-axis[1], axis[0], 0]])
    return np.eye(3) + math.sin(ang) * k + (1 - math.cos(ang)) * (k @ k)


def _pose(Rm, c):
    M = np.eye(4)
    M[:3, :3] = Rm
    M[:3, 3] = c
    return M.astype(np.float32)


def test_identity_maps_every_token_onto_itself():
    rng = np.random.default_rng(5)
    Rm = _rot(rng.normal(size=3), 0.7)
    M = _pose(Rm, [1.0, -2.0, 3.0])
    K = np.array([52.0, 52.0, 52.0, 30.0], np.float32)
    uv, idx = R.rotation_pair(M, K, M, K, 30, 52, 2)
    assert np.array_equal(idx, np.arange(30 * 52, dtype=np.int32))
    jj, ii = np.meshgrid(np.arange(52), np.arange(30))
    want = np.stack([jj.ravel() + 0.5, ii.ravel() + 0.5], -1)
    # A = R^T R is the identity only to rounding (fp32 rotation entries)
    assert np.abs(uv - want).max() < 1e-5


def test_zoom_is_a_scaling_about_the_principal_points():
    Rm = _rot([0.2, 1.0, -0.3], 0.4)
    M = _pose(Rm, [0.5, 0.0, 2.0])
    Kt = np.array([52.0, 48.0, 52.0, 30.0], np.float32)
    Ks = np.array([130.0, 120.0, 50.0, 31.0], np.float32)  # 2.5x zoom, shifted principal point
    h, w, p = 30, 52, 2
    uv, idx = R.rotation_pair(M, Kt, M, Ks, h, w, p)
    fxt, fyt, cxt, cyt = (float(x) / p for x in Kt)
    fxs, fys, cxs, cys = (float(x) / p for x in Ks)
    jj, ii = np.meshgrid(np.arange(w) + 0.5, np.arange(h) + 0.5)
    ex = cxs + (fxs / fxt) * (jj.ravel() - cxt)
    ey = cys + (fys / fyt) * (ii.ravel() - cyt)
    assert np.abs(uv[:, 0] - ex).max() < 1e-4 and np.abs(uv[:, 1] - ey).max() < 1e-4
    inside = (ex >= 0) & (ex < w) & (ey >= 0) & (ey < h)
    margin = np.minimum(np.abs(ex - np.round(ex)), np.abs(ey - np.round(ey))) > 1e-6
    assert np.array_equal(idx[inside & margin], (np.floor(ey) * w + np.floor(ex)).astype(np.int32)[inside & margin])
    assert np.all(idx[~inside & margin] == R.OFF_GRID)


@pytest.mark.parametrize("theta", [0.05, -0.3, 0.6])
def test_pure_yaw_closed_form(theta):
    # source camera yawed by theta about its own y axis: R_s = R_t R_y(theta)
    Rt = _rot([0.1, 0.0, 1.0], 0.25)
    Ry = np.array([[math.cos(theta), 0, math.sin(theta)], [0, 1, 0], [-math.sin(theta), 0, math.cos(theta)]])
    c = [3.0, 1.5, -2.0]
    Mt, Ms = _pose(Rt, c), _pose(Rt @ Ry, c)
    # the poses are stored in fp32, which moves the angle by ~1e-7 rad: far
    # inside the 2e-4 px bar at f = 52
    K = np.array([104.0, 104.0, 104.0, 60.0], np.float32)
    h, w, p = 30, 52, 2
    uv, idx = R.rotation_pair(Mt, K, Ms, K, h, w, p)
    f, cx, cy = 52.0, 52.0, 30.0
    jj, ii = np.meshgrid(np.arange(w) + 0.5, np.arange(h) + 0.5)
    alpha = np.arctan((jj.ravel() - cx) / f)
    dy = (ii.ravel() - cy) / f
    ex = cx + f * np.tan(alpha - theta)
    ey = cy + f * dy * np.cos(alpha) / np.cos(alpha - theta)
    front = np.cos(alpha - theta) > 0
    assert np.all(front)
    assert np.abs(uv[:, 0] - ex).max() < 2e-4 and np.abs(uv[:, 1] - ey).max() < 2e-4


def test_half_turn_puts_every_token_behind():
    Rt = _rot([0.0, 1.0, 0.0], 0.1)
    Ms = _pose(Rt @ _rot([0.0, 1.0, 0.0], math.pi), [0, 0, 0])
    Mt = _pose(Rt, [0, 0, 0])
    K = np.array([16.0, 16.0, 8.0, 8.0], np.float32)
    uv, idx = R.rotation_pair(Mt, K, Ms, K, 8, 8, 2)
    assert np.all(idx == R.BEHIND) and np.all(np.isnan(uv))


def test_agrees_with_the_general_reprojection_where_depth_cancels():
    """Shared centres, random rotations and zooms, random positive depth:
    u^ of Eq. reprojection equals the homography's to rounding, and every
    code that does not come from the depth test agrees."""
    rng = np.random.default_rng(11)
    h, w, p = 30, 52, 2
    n_checked = 0
    for trial in range(12):
        c = rng.normal(size=3) * 5
        Rt = _rot(rng.normal(size=3), rng.uniform(0, math.pi))
        Rs = Rt @ _rot(rng.normal(size=3), rng.uniform(0, 0.8))
        Mt, Ms = _pose(Rt, c), _pose(Rs, c)
        Kt = np.array([104.0, 92.0, 104.0, 60.0], np.float32)
        Ks = (Kt * np.float32(rng.uniform(0.6, 1.8))).astype(np.float32)
        Ks[2:] = Kt[2:] + rng.uniform(-4, 4, 2).astype(np.float32)
        depth_t = rng.uniform(0.5, 50.0, (h * p, w * p)).astype(np.float32)
        depth_s = rng.uniform(0.5, 50.0, (h * p, w * p)).astype(np.float32)
        uv_g, idx_g = R.reproject_pair(depth_t, Mt, Kt, depth_s, Ms, Ks, p, 0.05)
        uv_r, idx_r = R.rotation_pair(Mt, Kt, Ms, Ks, h, w, p)
        front = idx_g != R.BEHIND
        assert np.array_equal(idx_r == R.BEHIND, ~front)
        scale = np.maximum(1.0, np.abs(uv_g[front]).astype(np.float64))
        assert np.all(np.abs(uv_r[front] - uv_g[front]) <= 1e-5 * scale)
        far = front & (R.boundary_margin(uv_g, p, h, w) > 1e-4)
        g, r = idx_g[far], idx_r[far]
        occluded = g == R.OCCLUDED
        assert np.array_equal(g[~occluded], r[~occluded])
        # where the depth test rejected, the homography still names the cell
        cell = (np.floor(uv_g[far][:, 1]) * w + np.floor(uv_g[far][:, 0])).astype(np.int32)
        assert np.array_equal(r[occluded], cell[occluded])
        n_checked += int(far.sum())
    assert n_checked > 12 * h * w // 4


def test_moved_centre_and_empty_slot():
    M = _pose(np.eye(3), [0, 0, 0])
    Mm = _pose(np.eye(3), [0, 0, 1e-3])
    K = np.array([16.0, 16.0, 8.0, 8.0], np.float32)
    uv, idx = R.rotation_pair(M, K, Mm, K, 8, 8, 2)
    assert np.all(idx == R.CENTRE_MOVED) and np.all(np.isnan(uv))
    bank_c2w = np.stack([M, Mm])
    bank_K = np.stack([K, K])
    uv, idx = R.reproject_rotation(M[None], K[None], bank_c2w, bank_K, 8, 8, 2, src_sel=np.array([0, 1, -1, 2]))
    assert np.array_equal(idx[0], np.arange(64, dtype=np.int32))
    assert np.all(idx[1] == R.CENTRE_MOVED)
    assert np.all(idx[2] == R.NO_SOURCE) and np.all(idx[3] == R.NO_SOURCE)
    assert np.all(np.isnan(uv[2:]))
