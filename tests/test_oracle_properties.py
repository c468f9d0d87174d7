"""Property tests of the oracle over generated inputs (hypothesis), for
invariants the paper states rather than values it prints.

* Eq. bias: every bias value is <= 0, it is exactly 0 only at a key centre
  equal to u^, and over a biased frame its maximum sits at the key whose
  cell holds u^, i.e. at the correspondence index of Eq. reprojection
  (for u^ away from cell edges). Unbiased frames and rejected rows stay
  exactly 0 (design choices (ii) and (iii)).
* Sec. 4.3: for any two cameras sharing a centre, the depth cancels, so the
  rotation-only homography gives the general Eq. reprojection's u^ and every
  code that the depth test does not decide.
"""

from __future__ import annotations

import math

import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

from oracle import attention as A
from oracle import reprojection as R

SETTINGS = settings(max_examples=40, deadline=None, suppress_health_check=[HealthCheck.too_slow])


@SETTINGS
@given(h=st.integers(1, 9), w=st.integers(1, 11), sigma=st.floats(0.3, 6.0),
       fx=st.floats(0.0, 1.0, exclude_max=True), fy=st.floats(0.0, 1.0, exclude_max=True),
       slots=st.lists(st.integers(-1, 1), min_size=1, max_size=4), rejected=st.booleans())
def test_bias_is_nonpositive_and_peaks_at_the_corresponding_key(h, w, sigma, fx, fy, slots, rejected):
    Lk = len(slots) * h * w
    uh = np.array([[fx * w, fy * h]], np.float32)  # one query row, u^ inside the grid
    code = -4 if rejected else int(math.floor(uh[0, 1])) * w + int(math.floor(uh[0, 0]))
    corr_uv = np.repeat(uh[None], 2, axis=0)  # the same u^ for both source frames
    corr_idx = np.full((2, 1), code, np.int32)
    B = A.bias_block([0], Lk, h, w, np.array(slots), corr_uv, corr_idx, sigma)[0]
    assert np.all(B <= 0.0)
    kc = A.key_centres(Lk, h, w)
    at_centre = (kc[:, 0] == float(uh[0, 0])) & (kc[:, 1] == float(uh[0, 1]))
    for f, s in enumerate(slots):
        cols = slice(f * h * w, (f + 1) * h * w)
        if s < 0 or rejected:
            assert np.all(B[cols] == 0.0)
            continue
        assert np.array_equal(B[cols] == 0.0, at_centre[cols])
        x, y = float(uh[0, 0]), float(uh[0, 1])
        edge = min(x - math.floor(x), math.ceil(x) - x, y - math.floor(y), math.ceil(y) - y)
        if edge > 1e-6 and not (abs(x % 1 - 0.5) < 1e-6 or abs(y % 1 - 0.5) < 1e-6):
            assert int(np.argmax(B[cols])) == code


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


unit = st.tuples(st.floats(-1, 1), st.floats(-1, 1), st.floats(-1, 1)).filter(
    lambda v: 0.1 < math.sqrt(v[0] ** 2 + v[1] ** 2 + v[2] ** 2))


@SETTINGS
@given(axis_t=unit, ang_t=st.floats(0.0, 3.1), axis_d=unit, ang_d=st.floats(0.0, 1.2),
       zoom=st.floats(0.5, 2.0), dcx=st.floats(-5, 5), dcy=st.floats(-5, 5), depth=st.floats(0.5, 50.0),
       centre=st.tuples(st.floats(-30, 30), st.floats(-30, 30), st.floats(-30, 30)))
def test_rotation_only_equals_general_reprojection(axis_t, ang_t, axis_d, ang_d, zoom, dcx, dcy, depth, centre):
    h, w, p = 7, 11, 2
    Rt = _rot(axis_t, ang_t)
    Mt, Ms = _pose(Rt, centre), _pose(Rt @ _rot(axis_d, ang_d), centre)
    Kt = np.array([22.0, 20.0, 11.0, 7.0], np.float32)
    Ks = np.array([22.0 * zoom, 20.0 * zoom, 11.0 + dcx, 7.0 + dcy], np.float32)
    dmap = np.full((h * p, w * p), depth, np.float32)
    uv_g, idx_g = R.reproject_pair(dmap, Mt, Kt, dmap, Ms, Ks, p, 0.05)
    uv_r, idx_r = R.rotation_pair(Mt, Kt, Ms, Ks, h, w, p)
    front = idx_g != R.BEHIND
    assert np.array_equal(idx_r == R.BEHIND, ~front)
    scale = np.maximum(1.0, np.abs(uv_g[front]).astype(np.float64))
    assert np.all(np.abs(uv_r[front] - uv_g[front]) <= 1e-5 * scale)
    far = front & (R.boundary_margin(uv_g, p, h, w) > 1e-4) & (idx_g != R.OCCLUDED)
    assert np.array_equal(idx_r[far], idx_g[far])
