"""Invariance pins for the oracle: properties the paper's definitions fix
whatever the numbers, chosen to catch mistakes that a hand example or a
brute force written with the same reading could share.

* Retrieval (Sec. 4.2, Eq. retrieval) depends on poses only through centre
  distances and dot products of viewing directions, so moving the whole
  trajectory by one rigid motion leaves the result unchanged. The motions
  used are exact in fp32 (axis permutations, sign flips, integer shifts of
  centres on a 1/1024 grid); a cyclic axis permutation changes the third
  row of R and keeps its third column, so reading v = R e_z from the wrong
  side of R fails.
* Correspondence (Sec. 4.3, Eq. reprojection, Eq. visibility) is a relation
  between two cameras and a depth map, unchanged when both cameras move by
  the same rigid motion (R_s transposed, not inverted numerically or left
  untransposed, is what keeps it so).
* Biased attention (Sec. 4.3, Eq. bias) treats the KV frames as a set:
  permuting them together with their slot entries changes nothing; O is
  linear in V and a convex combination of the V rows.
"""

import math

import numpy as np
import pytest

from oracle import attention as OA, reprojection as OR, retrieval as ORT
from workloads.synth import axis_angle, pose_from, random_unit, ring_bank

# exact rigid motions: (rotation part, integer shift of the centre)
MOTIONS = [
    (np.array([[0, 1, 0], [0, 0, 1], [1, 0, 0]], np.float32), np.array([3, -2, 7], np.float32)),  # cyclic axes
    (np.array([[0, -1, 0], [1, 0, 0], [0, 0, 1]], np.float32), np.array([-5, 1, 0], np.float32)),  # 90 deg about z
    (np.array([[1, 0, 0], [0, 0, -1], [0, 1, 0]], np.float32), np.array([0, 0, 11], np.float32)),  # 90 deg about x
]


def _move(c2w, R0, t):
    out = np.array(c2w, np.float32, copy=True)
    out[..., :3, :3] = np.einsum("ij,...jk->...ik", R0, c2w[..., :3, :3])
    out[..., :3, 3] = np.einsum("ij,...j->...i", R0, c2w[..., :3, 3]) + t
    return out


def _snap_centres(c2w):
    out = np.array(c2w, np.float32, copy=True)
    out[..., :3, 3] = np.round(out[..., :3, 3] * 1024.0) / 1024.0
    return out


@pytest.mark.parametrize("m", range(len(MOTIONS)))
def test_retrieval_invariant_under_rigid_motion(m):
    rng = np.random.default_rng(40 + m)
    bank = ring_bank(rng, 400, radius=6.0)
    # tilt every camera a little so that the third column of R is not the third row
    for j in range(len(bank)):
        bank[j, :3, :3] = (axis_angle(random_unit(rng), math.radians(rng.uniform(0, 25))) @ bank[j, :3, :3]).astype(np.float32)
    bank = _snap_centres(bank)
    query = _snap_centres(bank[[10, 150, 333, 399]] @ pose_from(axis_angle(random_unit(rng), 0.1), [0.05, 0, 0]).astype(np.float32))
    qchunk = np.array([420, 300, 380, 405], np.int32)
    args = dict(E=12.0, w_v=0.5, tau_c=0.15, tau_v=0.7, delta=3, first_candidate=1, k=8)
    i0, s0, c0 = ORT.retrieve(bank, query, qchunk, **args)
    R0, t = MOTIONS[m]
    i1, s1, c1 = ORT.retrieve(_move(bank, R0, t), _move(query, R0, t), qchunk, **args)
    assert (c0 > 2).all()
    assert np.array_equal(c0, c1) and np.array_equal(i0, i1)
    ok = np.isfinite(s0)
    assert np.allclose(s0[ok], s1[ok], rtol=0, atol=1e-12)
    # reading the viewing direction from the third row instead is not invariant
    rowwise = bank.copy()
    rowwise[:, :3, :3] = np.swapaxes(bank[:, :3, :3], 1, 2)
    qrow = query.copy()
    qrow[:, :3, :3] = np.swapaxes(query[:, :3, :3], 1, 2)
    j0, _, _ = ORT.retrieve(rowwise, qrow, qchunk, **args)
    j1, _, _ = ORT.retrieve(_transposed_move(bank, R0, t), _transposed_move(query, R0, t), qchunk, **args)
    if m == 0:
        assert not np.array_equal(j0, j1)


def _transposed_move(c2w, R0, t):
    """The moved poses with R stored transposed: what a reader of rows sees."""
    moved = _move(c2w, R0, t)
    moved[..., :3, :3] = np.swapaxes(moved[..., :3, :3], -1, -2)
    return moved


def _plane_depth(rng, n, Hd, Wd):
    yy, xx = np.mgrid[0:Hd, 0:Wd].astype(np.float64)
    d = np.empty((n, Hd, Wd), np.float32)
    for i in range(n):
        z0 = rng.uniform(4.0, 9.0)
        d[i] = z0 + 0.02 * (xx - Wd / 2) + 0.01 * (yy - Hd / 2)
    return d


@pytest.mark.parametrize("m", range(len(MOTIONS)))
def test_correspondence_invariant_under_rigid_motion(m):
    rng = np.random.default_rng(70 + m)
    h, w, p = 9, 13, 2
    K = np.array([[12.0, 12.0, 13.0, 9.0]], np.float32)
    tgt_c = _snap_centres(pose_from(axis_angle(random_unit(rng), 0.3), [0.5, -0.25, 0.125]).astype(np.float32)[None])
    src_c = _snap_centres(np.stack([tgt_c[0] @ pose_from(axis_angle(random_unit(rng), math.radians(6)),
                                                          rng.uniform(-0.3, 0.3, 3)).astype(np.float32)
                                    for _ in range(3)]))
    td, sd = _plane_depth(rng, 1, h * p, w * p), _plane_depth(rng, 3, h * p, w * p)
    uv0, idx0 = OR.reproject(td, tgt_c, K, sd, src_c, np.repeat(K, 3, 0), p, 0.05)
    R0, t = MOTIONS[m]
    uv1, idx1 = OR.reproject(td, _move(tgt_c, R0, t), K, sd, _move(src_c, R0, t), np.repeat(K, 3, 0), p, 0.05)
    near = OR.boundary_margin(uv0, p, h, w) < 1e-6
    assert (idx0 >= 0).mean() > 0.2
    assert np.array_equal(idx0[~near], idx1[~near])
    both = np.isfinite(uv0) & np.isfinite(uv1)
    assert np.array_equal(np.isfinite(uv0), np.isfinite(uv1))
    assert np.abs(uv0[both].astype(np.float64) - uv1[both]).max() <= 1e-4


def _attention_case(rng, nf=5, h=3, w=4, Lq=7, H=2, D=16, S=3):
    hw = h * w
    slot = np.full(nf, -1, np.int32)
    slot[rng.choice(nf, S, replace=False)] = np.arange(S)
    uv = np.stack([rng.uniform(0, w, (S, Lq)), rng.uniform(0, h, (S, Lq))], -1).astype(np.float32)
    idx = rng.integers(-2, hw, (S, Lq)).astype(np.int32)
    q = rng.standard_normal((Lq, H, D))
    k = rng.standard_normal((nf * hw, H, D))
    v = rng.standard_normal((nf * hw, H, D))
    return q, k, v, slot, uv, idx, h, w


def test_attention_invariant_under_frame_permutation():
    rng = np.random.default_rng(5)
    q, k, v, slot, uv, idx, h, w = _attention_case(rng)
    nf, hw = len(slot), h * w
    O0, L0 = OA.biased_attention(q, k, v, slot, uv, idx, h, w, 0.3, 1.0, 1.5)
    perm = rng.permutation(nf)
    rows = (perm[:, None] * hw + np.arange(hw)[None, :]).reshape(-1)
    O1, L1 = OA.biased_attention(q, k[rows], v[rows], slot[perm], uv, idx, h, w, 0.3, 1.0, 1.5)
    assert np.allclose(O0, O1, rtol=0, atol=1e-12) and np.allclose(L0, L1, rtol=0, atol=1e-12)
    # the bias really is in play: without it the result moves
    O2, _ = OA.biased_attention(q, k, v, np.full(nf, -1, np.int32), uv, idx, h, w, 0.3, 1.0, 1.5)
    assert np.abs(O2 - O0).max() > 1e-3


def test_attention_linear_in_v_and_convex():
    rng = np.random.default_rng(6)
    q, k, v, slot, uv, idx, h, w = _attention_case(rng)
    v2 = rng.standard_normal(v.shape)
    O1, L1 = OA.biased_attention(q, k, v, slot, uv, idx, h, w, 0.3, 1.0, 1.5)
    O2, _ = OA.biased_attention(q, k, v2, slot, uv, idx, h, w, 0.3, 1.0, 1.5)
    O3, L3 = OA.biased_attention(q, k, 2.0 * v - 0.5 * v2, slot, uv, idx, h, w, 0.3, 1.0, 1.5)
    assert np.allclose(O3, 2.0 * O1 - 0.5 * O2, rtol=0, atol=1e-12) and np.array_equal(L1, L3)
    lo, hi = v.min(axis=0), v.max(axis=0)  # [H, D]
    assert (O1 >= lo[None] - 1e-12).all() and (O1 <= hi[None] + 1e-12).all()
