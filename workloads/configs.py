"""The five synthetic workloads, shaped like the paper's Wan-1.3B / Wan-14B use.

Shapes borrowed from the paper (Sec. 4.1, Sec. 4.2, Sec. 5.1): F = 3 latent
frames per chunk; a 30x52 token grid for 832x480 video (8x VAE, 2x2 patch);
a 90 degree field of view; revisits within about 2 m and 45 degrees; planar
metric depth. The datasets the paper evaluates on (TartanGround-Revisit,
TartanAir-Revisit) are not available, so seeded synthetic scenes stand in
for them.

Seeds: ``numpy.random.Generator(PCG64(1000 + config_id))``. Q/K/V are
drawn N(0, 1) in fp32; bf16 workloads round them to nearest-even bf16 and
keep the bit patterns (``q_bits`` ...), fp32 workloads keep fp32 values.

    C1  tiny fp32: 1 head, D 64, 8x8 tokens over a 16x16 depth map (p = 2),
        fx = fy = 8, cx = cy = 8; Lq = 64; KV = 2 retrieved + 2 recent frames
        (Lk = 256, slots [0, 1, -1, -1]); a random plane (normal within 30 deg
        of the query's optical axis, crossing it at z in [1, 10] m) seen by
        all three frames, each frame with its own N(0, 0.01) m noise, clipped
        to [1, 10] m; retrieved poses = query pose perturbed <= 5 deg / <= 0.2 m.
    C2  Wan-1.3B plain window: 12 heads, D 128, bf16, 30x52 tokens,
        Lq = 4680 (3 frames), Lk = 18720 (sink + 3 recent chunks), no bias.
    C3  C2 plus 2 retrieved chunks: Lk = 28080, slots 0..5 on KV frames 3..8;
        fx = fy = 52, cx = 52, cy = 30 (90 deg FOV over 104x60 latent px);
        6 stored frames 0.5 m apart moving forward; query frame i = stored
        frame i perturbed <= 5 deg / <= 0.3 m; depth from 4 world planes
        (ground + 3 random walls 4-15 m ahead) shared by all 9 frames,
        [0.5, 50] m; about 70% of (query token, source frame) pairs land on
        the source grid.
    C4  history bank: 200 chunks x 3 frames on a circle of radius 20 m at
        1.5 m height, heading = tangent + U(+-10 deg); walls 5-25 m outside
        the loop plus ground; 8 query chunks on a second lap (n = 200 + 25 q)
        with fresh heading jitter; top-4 retrieval (E = 40 m, tau_c = 0.05,
        tau_v = 45 deg, Delta = 3, first candidate 1, middle frame as the
        chunk pose); reprojection into 12 frames; attention over
        Lk = 37440 (sink + 4 retrieved + 3 recent chunks).
    C5  Wan-14B 720p: 40 heads, D 128, bf16, 45x80 tokens, Lq = 10800,
        Lk = 64800 (sink + 2 retrieved + 3 recent chunks), depth 90x160 from
        ground + 5 walls in [0.5, 80] m, fx = fy = 80, cx = 80, cy = 45; bank
        of 300 chunks on a circle of radius 30 m (E = 60 m), query = stored
        chunk 150 perturbed <= 5 deg / <= 0.3 m, top-2 retrieval.

Method constants the paper leaves open and these workloads fix: sigma = 2
token-grid units, lambda = 1, eps = 0.05 (Sec. 4.3 gives no values);
tau_c * E = 2 m and tau_v = 45 deg reuse the revisit definition of Sec. 5.1;
Delta = 3 excludes the two recent chunks (Sec. 4.2 cache layout).
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

from .synth import (
    bf16_bits,
    look_pose,
    perturb_pose,
    noisy_plane_depth,
    random_view_plane,
    render_planes,
)

CONFIG_NAMES = {
    1: "tiny-fp32-ref",
    2: "wan1.3b-plain-window",
    3: "wan1.3b-loop-closure",
    4: "wan1.3b-history-bank",
    5: "wan14b-720p",
}

F_PER_CHUNK = 3


def _rng(config_id: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(1000 + config_id))


@dataclass
class Retrieval:
    """Inputs of pose retrieval: one representative pose per chunk."""

    bank_c2w: np.ndarray  # [N, 4, 4] fp32, bank entry j is chunk j
    query_c2w: np.ndarray  # [Q, 4, 4] fp32
    query_chunk: np.ndarray  # [Q] int32
    E: float
    w_v: float
    tau_c: float
    tau_v: float  # radians
    delta: int
    first_candidate: int
    k: int
    frames_per_chunk: int = F_PER_CHUNK
    # per-frame bank (the reprojection sources are gathered from it)
    bank_frame_depth: Optional[np.ndarray] = None  # [N*F, H, W] fp32
    bank_frame_c2w: Optional[np.ndarray] = None  # [N*F, 4, 4] fp32
    bank_frame_K: Optional[np.ndarray] = None  # [N*F, 4] fp32
    # per query chunk, its F frames (reprojection targets)
    query_frame_depth: Optional[np.ndarray] = None  # [Q, F, H, W]
    query_frame_c2w: Optional[np.ndarray] = None  # [Q, F, 4, 4]
    query_frame_K: Optional[np.ndarray] = None  # [Q, F, 4]


@dataclass
class Workload:
    config_id: int
    name: str
    dtype: str  # "f32" or "bf16"
    H: int
    D: int
    h: int  # token grid rows
    w: int  # token grid cols
    p: int  # latent px per token side
    Tq: int  # query frames
    Lq: int
    Lk: int
    slot: np.ndarray  # [Lk / (h*w)] int32, -1 or retrieved frame index s
    S: int  # retrieved (source) frames
    softmax_scale: float
    lam: float
    sigma: float
    eps: float
    # fp32 values (f32 workloads) or bf16 bit patterns (bf16 workloads)
    q: np.ndarray = field(repr=False, default=None)  # [Lq, H, D]
    k: np.ndarray = field(repr=False, default=None)  # [Lk, H, D]
    v: np.ndarray = field(repr=False, default=None)  # [Lk, H, D]
    # reprojection inputs when the sources are fixed (C1, C3); None when
    # they come out of retrieval (C4, C5: see ``retrieval``)
    tgt_depth: Optional[np.ndarray] = None  # [Tq, h*p, w*p]
    tgt_c2w: Optional[np.ndarray] = None  # [Tq, 4, 4]
    tgt_K: Optional[np.ndarray] = None  # [Tq, 4]
    src_depth: Optional[np.ndarray] = None  # [S, h*p, w*p]
    src_c2w: Optional[np.ndarray] = None  # [S, 4, 4]
    src_K: Optional[np.ndarray] = None  # [S, 4]
    retrieval: Optional[Retrieval] = None

    @property
    def flops(self) -> float:
        """Algorithmic attention flops: QK^T plus PV, 4 Lq Lk D H."""
        return 4.0 * self.Lq * self.Lk * self.D * self.H

    def values(self, name: str, rows=None) -> np.ndarray:
        """fp32 values of q/k/v (optionally only some token rows)."""
        a = getattr(self, name)
        if rows is not None:
            a = a[rows]
        if self.dtype == "bf16":
            return (a.astype(np.uint32) << 16).view(np.float32)
        return a


def _qkv(rng, Lq, Lk, H, D, dtype):
    out = []
    for L in (Lq, Lk, Lk):
        x = rng.standard_normal((L, H, D), dtype=np.float32)
        out.append(bf16_bits(x) if dtype == "bf16" else x)
    return out


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


# --------------------------------------------------------------------------
# C1: tiny fp32 reference
# --------------------------------------------------------------------------
def make_c1() -> Workload:
    rng = _rng(1)
    h = w = 8
    p = 2
    K = np.array([8.0, 8.0, 8.0, 8.0])
    base = look_pose([0.0, 0.0, 1.5], yaw=rng.uniform(-np.pi, np.pi))
    tgt_c2w = base[None]
    src_c2w = np.stack([perturb_pose(rng, base, 5.0, 0.2) for _ in range(2)])
    plane = random_view_plane(rng, base, 1.0, 10.0, 30.0)
    depths = [noisy_plane_depth(rng, c, K, h * p, w * p, plane, 1.0, 10.0, 0.01)
              for c in [base, src_c2w[0], src_c2w[1]]]
    q, k, v = _qkv(rng, 64, 256, 1, 64, "f32")
    return Workload(
        config_id=1, name=CONFIG_NAMES[1], dtype="f32", H=1, D=64, h=h, w=w, p=p, Tq=1,
        Lq=64, Lk=256, slot=np.array([0, 1, -1, -1], np.int32), S=2,
        softmax_scale=1.0 / math.sqrt(64), lam=1.0, sigma=2.0, eps=0.05,
        q=q, k=k, v=v,
        tgt_depth=_f32(depths[0][None]), tgt_c2w=_f32(tgt_c2w), tgt_K=_f32(K[None]),
        src_depth=_f32(np.stack(depths[1:])), src_c2w=_f32(src_c2w), src_K=_f32(np.stack([K, K])),
    )


# --------------------------------------------------------------------------
# C2: Wan-1.3B plain window (bias off)
# --------------------------------------------------------------------------
def make_c2(dtype: str = "bf16", qkv: bool = True) -> Workload:
    rng = _rng(2)
    h, w = 30, 52
    hw = h * w
    q, k, v = _qkv(rng, 3 * hw, 12 * hw, 12, 128, dtype) if qkv else (None, None, None)
    return Workload(
        config_id=2, name=CONFIG_NAMES[2], dtype=dtype, H=12, D=128, h=h, w=w, p=2, Tq=3,
        Lq=3 * hw, Lk=12 * hw, slot=np.full(12, -1, np.int32), S=0,
        softmax_scale=1.0 / math.sqrt(128), lam=1.0, sigma=2.0, eps=0.05,
        q=q, k=k, v=v,
    )


# --------------------------------------------------------------------------
# C3: Wan-1.3B loop closure with fixed retrieved chunks
# --------------------------------------------------------------------------
def _c3_scene(rng):
    planes = [(np.array([0.0, 0.0, 1.0]), 0.0)]  # ground, camera 1.5 m above
    for _ in range(3):
        yaw = rng.uniform(-0.7, 0.7)
        n = -np.array([np.cos(yaw), np.sin(yaw), 0.0])  # faces the camera
        dist = rng.uniform(4.0, 15.0)
        planes.append((n, -dist))
    return planes


def make_c3_geometry(rng, h=30, w=52, p=2):
    K = np.array([52.0, 52.0, 52.0, 30.0])
    planes = _c3_scene(rng)
    stored = [look_pose([0.5 * i, 0.0, 1.5], yaw=0.0, pitch=0.05) for i in range(6)]
    queries = [perturb_pose(rng, stored[i], 5.0, 0.3) for i in range(3)]
    H, W = h * p, w * p
    src_depth = np.stack([render_planes(c, K, H, W, planes, 0.5, 50.0) for c in stored])
    tgt_depth = np.stack([render_planes(c, K, H, W, planes, 0.5, 50.0) for c in queries])
    return (
        _f32(tgt_depth), _f32(np.stack(queries)), _f32(np.tile(K, (3, 1))),
        _f32(src_depth), _f32(np.stack(stored)), _f32(np.tile(K, (6, 1))),
    )


def make_c3(dtype: str = "bf16", qkv: bool = True) -> Workload:
    rng = _rng(3)
    h, w, p = 30, 52, 2
    hw = h * w
    geo = make_c3_geometry(rng, h, w, p)
    slot = np.full(18, -1, np.int32)
    slot[3:9] = np.arange(6)
    q, k, v = _qkv(rng, 3 * hw, 18 * hw, 12, 128, dtype) if qkv else (None, None, None)
    return Workload(
        config_id=3, name=CONFIG_NAMES[3], dtype=dtype, H=12, D=128, h=h, w=w, p=p, Tq=3,
        Lq=3 * hw, Lk=18 * hw, slot=slot, S=6,
        softmax_scale=1.0 / math.sqrt(128), lam=1.0, sigma=2.0, eps=0.05,
        q=q, k=k, v=v,
        tgt_depth=geo[0], tgt_c2w=geo[1], tgt_K=geo[2],
        src_depth=geo[3], src_c2w=geo[4], src_K=geo[5],
    )


def make_reproj_batch(B: int, distinct: int = 16, seed: int = 3003):
    """B independent C3-shaped reprojection problems (3 target frames, 6
    sources, 60x104 depth), ``distinct`` of them generated and tiled to B.
    Returns the six arrays with a leading batch dimension."""
    rng = np.random.Generator(np.random.PCG64(seed))
    probs = [make_c3_geometry(rng) for _ in range(min(B, distinct))]
    reps = -(-B // len(probs))
    return tuple(np.ascontiguousarray(np.concatenate([np.stack([pr[i] for pr in probs])] * reps)[:B])
                 for i in range(6))


def _fov_K(fov_deg: float, H: int, W: int) -> np.ndarray:
    """Pinhole (fx, fy, cx, cy) in depth-map pixels for a horizontal FOV."""
    f = (W / 2.0) / np.tan(np.deg2rad(fov_deg) / 2.0)
    return np.array([f, f, W / 2.0, H / 2.0])


def make_rotation_batch(B: int, Tq: int = 3, S: int = 6, h: int = 30, w: int = 52, p: int = 2,
                        distinct: int = 16, seed: int = 3006):
    """B shared-centre problems shaped like the paper's panorama-rendered
    revisit clips (Sec. 5: a rotation excursion that yaws away by 90-180
    degrees and returns, or a zoom excursion from a 90 to a 35 degree FOV and
    back). Per problem one camera centre; the S source frames are the
    outward leg, the Tq target frames the return leg near the same headings
    (+-10 degrees yaw, +-3 degrees pitch jitter). Even problems rotate at a
    90 degree FOV, odd ones zoom at a fixed heading. ``distinct`` problems are
    generated and tiled to B. Returns tgt_c2w [B,Tq,4,4], tgt_K [B,Tq,4],
    src_c2w [B,S,4,4], src_K [B,S,4], all fp32."""
    rng = np.random.Generator(np.random.PCG64(seed))
    H, W = h * p, w * p
    probs = []
    for n in range(min(B, distinct)):
        c = rng.uniform(-20.0, 20.0, 3)
        c[2] = rng.uniform(1.0, 3.0)
        yaw0 = rng.uniform(0.0, 2 * np.pi)
        if n % 2 == 0:
            span = np.deg2rad(rng.uniform(90.0, 180.0))
            yaws = yaw0 + span * np.arange(S) / max(S - 1, 1)
            fovs = np.full(S, 90.0)
        else:
            yaws = np.full(S, yaw0)
            fovs = 90.0 - (90.0 - 35.0) * np.arange(S) / max(S - 1, 1)
        src_c2w = np.stack([look_pose(c, yaw=y, pitch=0.05) for y in yaws])
        src_K = np.stack([_fov_K(f, H, W) for f in fovs])
        pick = rng.integers(0, S, Tq)
        tgt_c2w = np.stack([look_pose(c, yaw=yaws[k] + np.deg2rad(rng.uniform(-10, 10)),
                                      pitch=0.05 + np.deg2rad(rng.uniform(-3, 3))) for k in pick])
        tgt_K = np.stack([_fov_K(fovs[k] * rng.uniform(0.95, 1.05), H, W) for k in pick])
        probs.append(tuple(x.astype(np.float32) for x in (tgt_c2w, tgt_K, src_c2w, src_K)))
    reps = -(-B // len(probs))
    return tuple(np.ascontiguousarray(np.concatenate([np.stack([pr[i] for pr in probs])] * reps)[:B])
                 for i in range(4))


# --------------------------------------------------------------------------
# C4 / C5: history bank on a loop + retrieval
# --------------------------------------------------------------------------
def _ring_walls(rng, n_walls, radius, lo, hi):
    planes = [(np.array([0.0, 0.0, 1.0]), 0.0)]
    for _ in range(n_walls):
        th = rng.uniform(0.0, 2 * np.pi)
        n = np.array([np.cos(th), np.sin(th), 0.0])
        planes.append((n, radius + rng.uniform(lo, hi)))
    return planes


def _loop_pose(rng, g, frames_per_lap, radius, jitter_deg):
    th = 2.0 * np.pi * (g % frames_per_lap) / frames_per_lap
    pos = [radius * np.cos(th), radius * np.sin(th), 1.5]
    yaw = th + np.pi / 2 + np.deg2rad(rng.uniform(-jitter_deg, jitter_deg))
    return look_pose(pos, yaw=yaw, pitch=0.08)


def _bank_workload(config_id, rng, *, n_chunks, radius, n_walls, wall_lo, wall_hi, zmax,
                   h, w, p, K, queries, k_top, E, tau_c, tau_v_deg, perturb=None):
    F = F_PER_CHUNK
    frames_per_lap = n_chunks * F
    planes = _ring_walls(rng, n_walls, radius, wall_lo, wall_hi)
    H, W = h * p, w * p
    frame_c2w = np.stack([_loop_pose(rng, g, frames_per_lap, radius, 10.0) for g in range(n_chunks * F)])
    frame_depth = np.stack([render_planes(c, K, H, W, planes, 0.5, zmax) for c in frame_c2w])
    q_c2w, q_depth, q_chunk = [], [], []
    for n, src_chunk in queries:
        if perturb is None:
            poses = [_loop_pose(rng, n * F + f, frames_per_lap, radius, 10.0) for f in range(F)]
        else:
            poses = [perturb_pose(rng, frame_c2w[src_chunk * F + f], *perturb) for f in range(F)]
        q_c2w.append(np.stack(poses))
        q_depth.append(np.stack([render_planes(c, K, H, W, planes, 0.5, zmax) for c in poses]))
        q_chunk.append(n)
    q_c2w = np.stack(q_c2w)
    mid = F // 2
    return Retrieval(
        bank_c2w=_f32(frame_c2w[mid::F]),
        query_c2w=_f32(q_c2w[:, mid]),
        query_chunk=np.asarray(q_chunk, np.int32),
        E=E, w_v=0.5, tau_c=tau_c, tau_v=np.deg2rad(tau_v_deg), delta=3, first_candidate=1, k=k_top,
        bank_frame_depth=_f32(frame_depth), bank_frame_c2w=_f32(frame_c2w),
        bank_frame_K=_f32(np.tile(K, (len(frame_c2w), 1))),
        query_frame_depth=_f32(np.stack(q_depth)), query_frame_c2w=_f32(q_c2w),
        query_frame_K=_f32(np.tile(K, (len(queries), F, 1))),
    )


def make_c4(dtype: str = "bf16", qkv: bool = True) -> Workload:
    rng = _rng(4)
    h, w, p = 30, 52, 2
    hw = h * w
    K = np.array([52.0, 52.0, 52.0, 30.0])
    queries = [(200 + 25 * q, None) for q in range(8)]
    ret = _bank_workload(4, rng, n_chunks=200, radius=20.0, n_walls=16, wall_lo=5.0, wall_hi=25.0,
                         zmax=50.0, h=h, w=w, p=p, K=K, queries=queries, k_top=4,
                         E=40.0, tau_c=0.05, tau_v_deg=45.0)
    slot = np.full(24, -1, np.int32)
    slot[3:15] = np.arange(12)
    q = k = v = None
    if qkv:
        q, k, v = _qkv(rng, 3 * hw, 24 * hw, 12, 128, dtype)
    return Workload(
        config_id=4, name=CONFIG_NAMES[4], dtype=dtype, H=12, D=128, h=h, w=w, p=p, Tq=3,
        Lq=3 * hw, Lk=24 * hw, slot=slot, S=12,
        softmax_scale=1.0 / math.sqrt(128), lam=1.0, sigma=2.0, eps=0.05,
        q=q, k=k, v=v, retrieval=ret,
    )


def make_c5(dtype: str = "bf16", qkv: bool = True) -> Workload:
    rng = _rng(5)
    h, w, p = 45, 80, 2
    hw = h * w
    K = np.array([80.0, 80.0, 80.0, 45.0])
    ret = _bank_workload(5, rng, n_chunks=300, radius=30.0, n_walls=5, wall_lo=5.0, wall_hi=25.0,
                         zmax=80.0, h=h, w=w, p=p, K=K, queries=[(300, 150)], k_top=2,
                         E=60.0, tau_c=2.0 / 60.0, tau_v_deg=45.0, perturb=(5.0, 0.3))
    slot = np.full(18, -1, np.int32)
    slot[3:9] = np.arange(6)
    q = k = v = None
    if qkv:
        q, k, v = _qkv(rng, 3 * hw, 18 * hw, 40, 128, dtype)
    return Workload(
        config_id=5, name=CONFIG_NAMES[5], dtype=dtype, H=40, D=128, h=h, w=w, p=p, Tq=3,
        Lq=3 * hw, Lk=18 * hw, slot=slot, S=6,
        softmax_scale=1.0 / math.sqrt(128), lam=1.0, sigma=2.0, eps=0.05,
        q=q, k=k, v=v, retrieval=ret,
    )


def make_config(config_id: int, dtype: Optional[str] = None, **kw) -> Workload:
    if config_id == 1:
        return make_c1()
    maker = {2: make_c2, 3: make_c3, 4: make_c4, 5: make_c5}[config_id]
    return maker(dtype or "bf16", **kw)
