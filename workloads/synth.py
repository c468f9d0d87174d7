"""Scene-synthesis primitives: rotations, camera poses, plane-rendered depth.

Conventions shared with the library's interface (not the method itself):

* a camera pose is a 4x4 row-major camera-to-world matrix ``[R | c; 0 0 0 1]``,
  camera axes OpenCV style (x right, y down, z forward);
* intrinsics are ``(fx, fy, cx, cy)`` in depth-map pixel units, a pixel
  ``(x, y)`` covering ``[x, x+1) x [y, y+1)``;
* depth is planar: the camera-frame z of the surface seen through a pixel
  centre.

The depth renderer intersects pixel-centre rays with a list of world planes
and keeps the nearest hit; it is how the synthetic scenes are *made*, not
part of the path under test.
"""

from __future__ import annotations

import numpy as np

WORLD_UP = np.array([0.0, 0.0, 1.0])


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even (NaN kept)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    # no uint32 overflow for finite or infinite inputs; NaNs are patched below
    with np.errstate(over="ignore"):
        rounded = (u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) >> np.uint32(16)
    out = rounded.astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def fp8e4m3_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> fp8 e4m3 codes (uint8), round to nearest even, saturating at
    +-448 (inputs are finite)."""
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), 448.0)
    _, e = np.frexp(a)  # a = f 2^e, 0.5 <= f < 1: spacing 2^(e - 4), at least 2^-9
    q = np.maximum(e - 4, -9)
    r = np.rint(np.ldexp(a, -q))  # ties to even
    v = np.ldexp(r, q)
    _, e2 = np.frexp(v)
    exp_field = np.where(v >= 2.0**-6, e2 - 1 + 7, 0)
    mant = np.where(v >= 2.0**-6, np.rint((np.ldexp(v, -(e2 - 1)) - 1.0) * 8), np.rint(v / 2.0**-9))
    code = (exp_field.astype(np.int64) << 3) | mant.astype(np.int64)
    return (code | np.where(np.signbit(x), 0x80, 0)).astype(np.uint8)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """fp32 values rounded to the nearest bf16, returned as fp32."""
    bits = bf16_bits(x).astype(np.uint32) << 16
    return bits.view(np.float32).reshape(np.shape(x))


def axis_angle(axis: np.ndarray, angle: float) -> np.ndarray:
    """Rotation matrix of ``angle`` radians about the unit ``axis``."""
    axis = np.asarray(axis, dtype=np.float64)
    axis = axis / np.linalg.norm(axis)
    x, y, z = axis
    k = np.array([[0.0, -z, y], [z, 0.0, -x], [-y, x, 0.0]])
    return np.eye(3) + np.sin(angle) * k + (1.0 - np.cos(angle)) * (k @ k)


def random_unit(rng: np.random.Generator) -> np.ndarray:
    v = rng.normal(size=3)
    return v / np.linalg.norm(v)


def pose_from(R: np.ndarray, c: np.ndarray) -> np.ndarray:
    m = np.eye(4)
    m[:3, :3] = R
    m[:3, 3] = c
    return m


def look_pose(position, yaw: float, pitch: float = 0.0) -> np.ndarray:
    """Camera at ``position`` looking along heading ``yaw`` (radians, world
    z-up), tilted down by ``pitch``; returns the 4x4 camera-to-world pose."""
    f = np.array([np.cos(yaw) * np.cos(pitch), np.sin(yaw) * np.cos(pitch), -np.sin(pitch)])
    r = np.cross(f, WORLD_UP)
    r /= np.linalg.norm(r)
    d = np.cross(f, r)
    R = np.stack([r, d, f], axis=1)
    return pose_from(R, np.asarray(position, dtype=np.float64))


def perturb_pose(rng: np.random.Generator, c2w: np.ndarray, max_deg: float, max_t: float) -> np.ndarray:
    """Rotate by U(0, max_deg) about a uniform random axis and translate by
    U(0, max_t) along a uniform random direction."""
    Rp = axis_angle(random_unit(rng), np.deg2rad(rng.uniform(0.0, max_deg)))
    t = random_unit(rng) * rng.uniform(0.0, max_t)
    return pose_from(Rp @ c2w[:3, :3], c2w[:3, 3] + t)


def pixel_rays(H: int, W: int, K) -> np.ndarray:
    """Camera-frame rays through pixel centres, z component 1: [H, W, 3]."""
    fx, fy, cx, cy = (float(v) for v in K)
    ys, xs = np.meshgrid(np.arange(H) + 0.5, np.arange(W) + 0.5, indexing="ij")
    return np.stack([(xs - cx) / fx, (ys - cy) / fy, np.ones_like(xs)], axis=-1)


def render_planes(c2w: np.ndarray, K, H: int, W: int, planes, zmin: float, zmax: float) -> np.ndarray:
    """Planar depth [H, W] of the nearest of ``planes`` (list of (n, o) with
    unit normal n, plane {X : n.X = o}) seen from ``c2w``; misses -> zmax;
    the result is clamped to [zmin, zmax]."""
    rays = pixel_rays(H, W, K)
    R, c = c2w[:3, :3], c2w[:3, 3]
    dirs = rays @ R.T
    depth = np.full((H, W), np.inf)
    for n, o in planes:
        n = np.asarray(n, dtype=np.float64)
        denom = dirs @ n
        with np.errstate(divide="ignore", invalid="ignore"):
            t = (o - n @ c) / denom
        hit = np.isfinite(t) & (t > 1e-6)
        depth = np.where(hit & (t < depth), t, depth)
    depth[~np.isfinite(depth)] = zmax
    return np.clip(depth, zmin, zmax)


def random_view_plane(rng, c2w, z_lo, z_hi, max_tilt_deg):
    """A random world plane (n, o) seen by camera ``c2w``: its normal lies
    within ``max_tilt_deg`` of the optical axis and it crosses the principal
    ray at camera depth z ~ U(z_lo, z_hi)."""
    tilt = axis_angle(random_unit(rng), np.deg2rad(rng.uniform(0.0, max_tilt_deg)))
    R, c = c2w[:3, :3], c2w[:3, 3]
    n = R @ (tilt @ np.array([0.0, 0.0, -1.0]))
    point = c + R @ np.array([0.0, 0.0, rng.uniform(z_lo, z_hi)])
    return n, float(n @ point)


def noisy_plane_depth(rng, c2w, K, H, W, plane, z_lo, z_hi, noise_std) -> np.ndarray:
    """Depth of one plane seen from ``c2w``, clipped to [z_lo, z_hi], plus
    N(0, noise_std) noise, re-clipped."""
    t = render_planes(c2w, K, H, W, [plane], z_lo, z_hi)
    t = t + rng.normal(0.0, noise_std, size=t.shape)
    return np.clip(t, z_lo, z_hi)


def ring_bank(rng: np.random.Generator, n: int, radius: float, height: float = 1.5,
              yaw_jitter_deg: float = 10.0) -> np.ndarray:
    """n camera-to-world poses [n, 4, 4] fp32 scattered over a disc of the
    given radius at a fixed height (world z up), each looking horizontally
    along the tangent of its circle plus a uniform yaw jitter: look_pose with
    pitch 0, vectorised for large stress banks."""
    rad = radius * np.sqrt(rng.uniform(0.0, 1.0, n))
    phi = rng.uniform(0.0, 2.0 * np.pi, n)
    yaw = phi + 0.5 * np.pi + np.deg2rad(rng.uniform(-yaw_jitter_deg, yaw_jitter_deg, n))
    c, s = np.cos(yaw), np.sin(yaw)
    out = np.zeros((n, 4, 4), np.float32)
    # columns: right = forward x up = (s, -c, 0), down = (0, 0, -1), forward = (c, s, 0)
    out[:, 0, 0], out[:, 1, 0] = s, -c
    out[:, 2, 1] = -1.0
    out[:, 0, 2], out[:, 1, 2] = c, s
    out[:, 0, 3] = rad * np.cos(phi)
    out[:, 1, 3] = rad * np.sin(phi)
    out[:, 2, 3] = height
    out[:, 3, 3] = 1.0
    return out
