"""Pins for the reprojection oracle (Sec. 4.3, Eq. reprojection, Eq. visibility).

* hand-derived translation example (tests/golden/reprojection_translation_example.json);
* identity pose with equal depth maps every token to itself;
* translation-only motion over a constant-depth fronto-parallel plane
  matches the closed form u^ = c' + (Z (u - c') - f' dc_xy) / (Z - dc_z);
* rotation/zoom only (c_s = c_t) matches the homography
  pi(K_s R_s^T R_t K_t^{-1} u~), built with numpy.linalg.inv, and is the
  same for two different depth maps (depth cancels, as the paper notes);
* an independent formulation (world point projected by K_s [R_s^T | -R_s^T c_s]
  with the world-to-camera matrix from numpy.linalg.inv) agrees;
* each rejection cause is produced by a scene built to cause it;
* a pure-Python brute force agrees on the 8x8 workload.
"""

import json
import math
import os

import numpy as np
import pytest

from oracle import brute, reprojection as R
from workloads import make_c1
from workloads.synth import axis_angle, pose_from, random_unit


def _rand_rot(rng, max_deg=180.0):
    return axis_angle(random_unit(rng), math.radians(rng.uniform(0, max_deg)))


def _const(h, w, p, Z):
    return np.full((h * p, w * p), Z, np.float32)


def test_golden_translation_example(golden_dir):
    with open(os.path.join(golden_dir, "reprojection_translation_example.json")) as f:
        g = json.load(f)
    h, w, p = g["h"], g["w"], g["p"]
    Kk = np.array(g["K"], np.float32)
    dt = _const(h, w, p, g["Z"])
    uv, idx = R.reproject_pair(dt, pose_from(np.eye(3), g["c_t"]), Kk, dt, pose_from(np.eye(3), g["c_s"]), Kk,
                               p, g["eps"])
    t = g["token_row"] * w + g["token_col"]
    np.testing.assert_allclose(uv[t], g["expected_uv"], atol=1e-6)
    assert idx[t] == g["expected_idx"]


@pytest.mark.parametrize("seed", range(3))
def test_identity_pose_maps_tokens_to_themselves(seed):
    rng = np.random.default_rng(seed)
    h, w, p = 7, 11, 2
    depth = rng.uniform(0.5, 30.0, size=(h * p, w * p)).astype(np.float32)
    c2w = pose_from(_rand_rot(rng), rng.normal(0, 5, 3)).astype(np.float32)
    Kk = np.array([9.0, 8.0, 11.0, 7.0], np.float32)
    # eps > 0: the round trip leaves [X_s]_z within rounding of D_s, on either side
    uv, idx = R.reproject_pair(depth, c2w, Kk, depth, c2w, Kk, p, 1e-6)
    assert (idx == np.arange(h * w)).all()
    ii, jj = np.divmod(np.arange(h * w), w)
    np.testing.assert_allclose(uv[:, 0], jj + 0.5, atol=1e-5)
    np.testing.assert_allclose(uv[:, 1], ii + 0.5, atol=1e-5)


@pytest.mark.parametrize("seed", range(4))
def test_translation_only_closed_form(seed):
    rng = np.random.default_rng(10 + seed)
    h, w, p = 12, 20, 2
    Z = rng.uniform(3.0, 20.0)
    Rm = _rand_rot(rng)
    ct = rng.normal(0, 3, 3)
    dcam = rng.uniform(-0.6, 0.6, 3)  # camera-frame offset of c_s from c_t
    cs = ct + Rm @ dcam
    Kk = np.array([10.0, 12.0, 20.0, 12.0])
    d = _const(h, w, p, Z)
    uv, idx = R.reproject_pair(d, pose_from(Rm, ct), Kk, d, pose_from(Rm, cs), Kk, p, 0.05)
    f = Kk / p
    ii, jj = np.divmod(np.arange(h * w), w)
    ux, uy = jj + 0.5, ii + 0.5
    Zf = float(np.float32(Z))
    ex = f[2] + (Zf * (ux - f[2]) - f[0] * dcam[0]) / (Zf - dcam[2])
    ey = f[3] + (Zf * (uy - f[3]) - f[1] * dcam[1]) / (Zf - dcam[2])
    np.testing.assert_allclose(uv[:, 0], ex, atol=1e-4)
    np.testing.assert_allclose(uv[:, 1], ey, atol=1e-4)
    on = (ex >= 0) & (ex < w) & (ey >= 0) & (ey < h)
    margin = np.minimum(np.abs(ex - np.round(ex)), np.abs(ey - np.round(ey)))
    sure = margin > 1e-4
    # constant source depth Z: visible iff [X_s]_z = Z - dc_z <= (1 + eps) Z
    visible = (Zf - dcam[2]) <= (1.0 + float(np.float32(0.05))) * Zf
    exp_idx = np.where(on, np.floor(ey) * w + np.floor(ex) if visible else -4, -3)
    assert (idx[sure] == exp_idx[sure]).all()


@pytest.mark.parametrize("seed", range(4))
def test_rotation_only_is_depth_independent_homography(seed):
    rng = np.random.default_rng(20 + seed)
    h, w, p = 10, 16, 2
    Rt, Rs = _rand_rot(rng), None
    Rs = axis_angle(random_unit(rng), math.radians(rng.uniform(0, 15))) @ Rt
    c = rng.normal(0, 4, 3)
    Kt = np.array([16.0, 16.0, 16.0, 10.0])
    Ks = np.array([24.0, 22.0, 15.0, 11.0])  # zoom change as well
    d1 = rng.uniform(1, 40, size=(h * p, w * p)).astype(np.float32)
    d2 = rng.uniform(1, 40, size=(h * p, w * p)).astype(np.float32)
    uv1, _ = R.reproject_pair(d1, pose_from(Rt, c), Kt, d1, pose_from(Rs, c), Ks, p, 0.05)
    uv2, _ = R.reproject_pair(d2, pose_from(Rt, c), Kt, d1, pose_from(Rs, c), Ks, p, 0.05)

    def kmat(K):
        return np.array([[K[0] / p, 0, K[2] / p], [0, K[1] / p, K[3] / p], [0, 0, 1.0]])

    Hm = kmat(Ks) @ Rs.T @ Rt @ np.linalg.inv(kmat(Kt))
    ii, jj = np.divmod(np.arange(h * w), w)
    ut = np.stack([jj + 0.5, ii + 0.5, np.ones(h * w)])
    hu = Hm @ ut
    front = hu[2] > 0
    np.testing.assert_allclose(uv1[front, 0], (hu[0] / hu[2])[front], rtol=1e-6, atol=1e-4)
    np.testing.assert_allclose(uv1[front, 1], (hu[1] / hu[2])[front], rtol=1e-6, atol=1e-4)
    np.testing.assert_allclose(uv1[front], uv2[front], rtol=1e-6, atol=1e-4)


@pytest.mark.parametrize("seed", range(4))
def test_world_point_projection_formulation(seed):
    rng = np.random.default_rng(30 + seed)
    h, w, p = 9, 13, 2
    Kt = np.array([13.0, 13.0, 13.0, 9.0])
    Ks = np.array([13.0, 14.0, 12.0, 9.5])
    Mt = pose_from(_rand_rot(rng), rng.normal(0, 3, 3))
    Ms = pose_from(axis_angle(random_unit(rng), math.radians(rng.uniform(0, 10))) @ Mt[:3, :3],
                   Mt[:3, 3] + rng.normal(0, 0.5, 3))
    dt = rng.uniform(2, 20, size=(h * p, w * p)).astype(np.float32)
    uv, idx = R.reproject_pair(dt, Mt, Kt, dt, Ms, Ks, p, 0.05)
    z = R.pooled_depth(dt, p).reshape(-1)
    ii, jj = np.divmod(np.arange(h * w), w)
    Kti = np.linalg.inv(np.array([[Kt[0] / p, 0, Kt[2] / p], [0, Kt[1] / p, Kt[3] / p], [0, 0, 1]]))
    Xt = (Kti @ np.stack([jj + 0.5, ii + 0.5, np.ones(h * w)])) * z
    Xw = Mt[:3, :3] @ Xt + Mt[:3, 3:4]
    w2c = np.linalg.inv(Ms)
    P = np.array([[Ks[0] / p, 0, Ks[2] / p], [0, Ks[1] / p, Ks[3] / p], [0, 0, 1]]) @ w2c[:3, :]
    hp = P @ np.vstack([Xw, np.ones(h * w)])
    front = hp[2] > 0
    np.testing.assert_allclose(uv[front, 0], (hp[0] / hp[2])[front], rtol=1e-6, atol=1e-4)
    np.testing.assert_allclose(uv[front, 1], (hp[1] / hp[2])[front], rtol=1e-6, atol=1e-4)


def test_rejection_causes():
    h, w, p = 6, 8, 2
    Kk = np.array([8.0, 6.0, 8.0, 6.0])
    d = _const(h, w, p, 5.0)
    base = pose_from(np.eye(3), [0, 0, 0])
    # 180 deg yaw: everything behind the source camera
    turned = pose_from(axis_angle(np.array([0, 1.0, 0]), math.pi), [0, 0, 0])
    _, idx = R.reproject_pair(d, base, Kk, d, turned, Kk, p, 0.05)
    assert (idx == R.BEHIND).all()
    # large sideways translation: everything off the grid
    _, idx = R.reproject_pair(d, base, Kk, d, pose_from(np.eye(3), [40.0, 0, 0]), Kk, p, 0.05)
    assert (idx == R.OFF_GRID).all()
    # an occluder 1 m in front of the source camera: everything occluded
    _, idx = R.reproject_pair(d, base, Kk, _const(h, w, p, 1.0), base, Kk, p, 0.05)
    assert (idx == R.OCCLUDED).all()
    # eps tolerance: a source surface 4% nearer than the point is still accepted at eps = 0.05
    _, idx = R.reproject_pair(d, base, Kk, _const(h, w, p, 5.0 / 1.04), base, Kk, p, 0.05)
    assert (idx == np.arange(h * w)).all()
    # undefined depth: NaN, zero and negative
    bad = d.copy()
    bad[0:2, 0:2] = np.nan
    bad[0:2, 2:4] = 0.0
    bad[2:4, 0:2] = -1.0
    uv, idx = R.reproject_pair(bad, base, Kk, d, base, Kk, p, 0.05)
    assert idx[0] == R.UNDEFINED and idx[1] == R.UNDEFINED and idx[w] == R.UNDEFINED
    assert np.isnan(uv[0]).all()
    assert idx[2] == 2


def test_no_source_slot():
    c1 = make_c1()
    uv, idx = R.reproject(c1.tgt_depth, c1.tgt_c2w, c1.tgt_K, c1.src_depth, c1.src_c2w, c1.src_K, 2, 0.05,
                          src_sel=np.array([1, -1]))
    assert (idx[1] == R.NO_SOURCE).all() and np.isnan(uv[1]).all()
    uv2, idx2 = R.reproject(c1.tgt_depth, c1.tgt_c2w, c1.tgt_K, c1.src_depth[1:], c1.src_c2w[1:], c1.src_K[1:],
                            2, 0.05)
    assert (idx[0] == idx2[0]).all()


def test_brute_force_agrees_on_tiny_workload():
    c1 = make_c1()
    uv, idx = R.reproject(c1.tgt_depth, c1.tgt_c2w, c1.tgt_K, c1.src_depth, c1.src_c2w, c1.src_K, c1.p, c1.eps)
    for s in range(c1.S):
        bf = brute.reproject(c1.tgt_depth[0].tolist(), c1.tgt_c2w[0].tolist(), c1.tgt_K[0].tolist(),
                             c1.src_depth[s].tolist(), c1.src_c2w[s].tolist(), c1.src_K[s].tolist(),
                             c1.p, float(np.float32(c1.eps)))
        for t, (ux, uy, i) in enumerate(bf):
            assert idx[s, t] == i
            if ux is not None:
                assert uv[s, t, 0] == np.float32(ux) and uv[s, t, 1] == np.float32(uy)
    # the tiny workload exercises accepted and rejected correspondences
    assert (idx >= 0).mean() > 0.8


def test_pooled_depth_is_block_mean():
    rng = np.random.default_rng(5)
    d = rng.uniform(1, 9, size=(6, 10)).astype(np.float32)
    pd = R.pooled_depth(d, 2)
    np.testing.assert_allclose(pd, d.astype(np.float64).reshape(3, 2, 5, 2).mean(axis=(1, 3)), rtol=1e-15)


def test_boundary_margin():
    m = R.boundary_margin(np.array([[2.5, 3.5], [4.00001, 1.5], [np.nan, np.nan]]), 2, 8, 8)
    np.testing.assert_allclose(m[:2], [1.0, 2e-5], rtol=1e-3)
    assert np.isinf(m[2])


def test_half_open_grid_edges():
    """Cells are half-open: u^_x == w is off the grid, u^_x == 0 is on it.
    Setup of the golden example (f' = c' = 4, Z = 4, R = I), for which
    u^_x = u_x - dc_x holds exactly in binary floating point."""
    h, w, p = 8, 8, 2
    Kk = np.array([8.0, 8.0, 8.0, 8.0], np.float32)
    d = _const(h, w, p, 4.0)
    base = pose_from(np.eye(3), [0.0, 0.0, 0.0])
    uv, idx = R.reproject_pair(d, base, Kk, d, pose_from(np.eye(3), [-0.5, 0.0, 0.0]), Kk, p, 0.05)
    assert uv[7, 0] == 8.0 and idx[7] == R.OFF_GRID          # token col 7 lands on x = w
    assert uv[6, 0] == 7.0 and idx[6] == 7                    # col 6 lands on the last cell's left edge
    uv, idx = R.reproject_pair(d, base, Kk, d, pose_from(np.eye(3), [0.5, 0.0, 0.0]), Kk, p, 0.05)
    assert uv[0, 0] == 0.0 and idx[0] == 0                    # col 0 lands on x = 0: on the grid
    uv, idx = R.reproject_pair(d, base, Kk, d, pose_from(np.eye(3), [0.0, -0.5, 0.0]), Kk, p, 0.05)
    assert uv[7 * w, 1] == 8.0 and idx[7 * w] == R.OFF_GRID  # last row lands on y = h


def test_visibility_near_ties():
    """Eq. visibility's near ties, |[X_s]_z - (1 + eps) D_s| < 1e-9 D_s, counted
    over on-grid pairs. Identity pose over a constant depth of 5 m: [X_s]_z = 5
    for every token. Against a source map of 4 m with eps = 0.25 the test is
    5 <= 1.25 * 4 = 5, an exact tie for all 48 tokens (and all are kept);
    against the same 5 m map, eps = 0 ties every token, eps = 0.05 none; a
    source looking away (every token behind it) has no pair on the grid."""
    h, w, p = 6, 8, 2
    Kk = np.array([[8.0, 8.0, 8.0, 6.0]], np.float32)
    eye = np.eye(4, dtype=np.float32)[None]
    d5, d4 = _const(h, w, p, 5.0)[None], _const(h, w, p, 4.0)[None]
    assert R.visibility_near_ties(d5, eye, Kk, d4, eye, Kk, p, 0.25) == h * w
    _, idx = R.reproject(d5, eye, Kk, d4, eye, Kk, p, 0.25)
    assert np.array_equal(idx[0], np.arange(h * w))
    assert R.visibility_near_ties(d5, eye, Kk, d5, eye, Kk, p, 0.0) == h * w
    assert R.visibility_near_ties(d5, eye, Kk, d5, eye, Kk, p, 0.05) == 0
    back = pose_from(axis_angle(np.array([0.0, 1.0, 0.0]), math.pi), [0.0, 0.0, 0.0]).astype(np.float32)[None]
    assert R.visibility_near_ties(d5, eye, Kk, d5, back, Kk, p, 0.0) == 0
    # two sources, the second an empty slot of a frame bank
    assert R.visibility_near_ties(d5, eye, Kk, d4, eye, Kk, p, 0.25, src_sel=[0, -1]) == h * w
