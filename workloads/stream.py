"""Seeded multi-chunk trajectory for the streaming driver (Sec. 4.2, cache layout).

A camera walks a loop of radius ``radius`` at 1.5 m height, ``chunks_per_lap``
chunks of F = 3 latent frames per lap, heading = tangent + U(+-10 deg), so
chunk n returns to the place of chunk n - chunks_per_lap. With 8 chunks per
lap and a gap of 3 chunks, the first loop closures come at n = 9 (the anchor
chunk 0 is never a candidate). Depth is rendered per frame from a world of
ground plus walls outside the loop, [0.5, 30] m; intrinsics give a 90 degree
field of view. q, k, v of every layer are drawn N(0, 1) per chunk (bf16:
rounded to nearest even, bit patterns kept); they stand in for the network's
projections and carry no structure. Nothing here computes a step of the
method.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List

import numpy as np

from .configs import F_PER_CHUNK, _loop_pose, _ring_walls
from .synth import bf16_bits, render_planes


@dataclass
class StreamChunk:
    depth: np.ndarray  # [F, h*p, w*p] float32, planar metric depth
    c2w: np.ndarray  # [F, 4, 4] float32
    K: np.ndarray  # [F, 4] float32 (fx, fy, cx, cy) in depth pixels
    q: np.ndarray = field(repr=False, default=None)  # [L, F*h*w, H, D] (bf16 bits or float32)
    k: np.ndarray = field(repr=False, default=None)
    v: np.ndarray = field(repr=False, default=None)


@dataclass
class Stream:
    F: int
    h: int
    w: int
    p: int
    H: int
    D: int
    L: int
    dtype: str
    chunks: List[StreamChunk]
    # retrieval (Eq. retrieval): E = loop diameter, tau_c E = 2 m, tau_v = 45 deg, Delta = 3, k = 1
    E: float
    w_v: float = 0.5
    tau_c: float = 0.0
    tau_v: float = math.radians(45.0)
    delta: int = 3
    # correspondence and bias (Sec. 4.3)
    eps: float = 0.05
    lam: float = 1.0
    sigma: float = 2.0
    softmax_scale: float = 0.0
    # temporal band of the rotary embedding
    rope_t_pairs: int = 22
    rope_theta: float = 10000.0


def make_stream(n_chunks: int = 12, h: int = 6, w: int = 8, p: int = 2, H: int = 2, D: int = 128, L: int = 2,
                dtype: str = "bf16", chunks_per_lap: int = 8, radius: float = 4.0, seed: int = 2024,
                qkv: bool = True) -> Stream:
    rng = np.random.Generator(np.random.PCG64(seed))
    F = F_PER_CHUNK
    Hd, Wd = h * p, w * p
    K = np.array([Wd / 2.0, Wd / 2.0, Wd / 2.0, Hd / 2.0])
    planes = _ring_walls(rng, 12, radius, 3.0, 10.0)
    frames_per_lap = chunks_per_lap * F
    T = F * h * w
    chunks = []
    for n in range(n_chunks):
        c2w = np.stack([_loop_pose(rng, n * F + f, frames_per_lap, radius, 10.0) for f in range(F)])
        depth = np.stack([render_planes(c, K, Hd, Wd, planes, 0.5, 30.0) for c in c2w]).astype(np.float32)
        ch = StreamChunk(depth=depth, c2w=c2w.astype(np.float32), K=np.tile(K, (F, 1)).astype(np.float32))
        if qkv:
            draw = [rng.standard_normal((L, T, H, D)).astype(np.float32) for _ in range(3)]
            if dtype == "bf16":
                draw = [bf16_bits(a) for a in draw]
            ch.q, ch.k, ch.v = draw
        chunks.append(ch)
    return Stream(F=F, h=h, w=w, p=p, H=H, D=D, L=L, dtype=dtype, chunks=chunks, E=2.0 * radius,
                  tau_c=2.0 / (2.0 * radius), softmax_scale=1.0 / math.sqrt(D))
