"""Seeded random sweeps through the kernels' parameter space, each case
against the fp64 oracle at the bars of the targeted tests (attention:
1e-4 fp32, 2e-2 / 4e-3 on O / LSE for bf16 and fp8 logits; correspondence:
codes and u^ bit-exact outside the boundary exemption).

Attention: ragged Lq and frame grids from 1 x 1 to 12 x 16 tokens, 1-24 KV
frames, 0-20 retrieved frames (frames beyond the staged ones included),
lambda of either sign and zero, sigma, softmax scale, and forced key-part
counts for the bf16 kernel. Correspondence: batches sized so that both
launch shapes (a thread per token, a thread per (token, source)) occur,
p = 1, 2, 3, depth maps with NaN, zero and negative pixels, with and
without a frame-bank selection, and sources that share a target frame's
camera centre (a camera turning in place) mixed with ones that do not."""

from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import paper_2607_21848_amd as rv
import workloads as W
from oracle import attention as OA, reprojection as OR
from tests.gpu_helpers import dev, host, same_bits_f32
from workloads.synth import axis_angle, fp8e4m3_bits, pose_from, random_unit

pytestmark = pytest.mark.gpu

F32_TOL, LSE_F32_TOL = 1e-4, 1e-4
BF16_TOL, LSE_BF16_TOL = 2e-2, 4e-3
KINDS = ("f32-64", "f32-128", "bf16", "fp8")


@pytest.mark.parametrize("case", range(20))
def test_attention_random_sweep(case):
    rng = np.random.default_rng(9100 + case)
    kind = KINDS[case % 4]
    D = 64 if kind == "f32-64" else 128
    h, w = int(rng.integers(1, 13)), int(rng.integers(1, 17))
    hw = h * w
    nf = int(rng.integers(1, min(24, max(1, 4000 // hw)) + 1))
    Lk, Lq, H = nf * hw, int(rng.integers(1, 400)), int(rng.integers(1, 4))
    S = int(rng.integers(0, 21))
    lam = float(rng.choice([0.0, 0.5, 1.0, 2.0, -0.5]))
    sigma = float(rng.uniform(1.0, 4.0))
    scale = float(rng.uniform(0.5, 1.5)) / math.sqrt(D)
    parts = int(rng.choice([0, 1, 2, 3, 5])) if kind in ("bf16", "fp8") else 0
    slot = np.full(nf, -1, np.int32)
    if S:
        frames = rng.choice(nf, size=min(S, nf), replace=False)
        slot[frames] = rng.permutation(S)[:len(frames)]
    uv = np.stack([rng.uniform(-1, w + 1, (S, Lq)), rng.uniform(-1, h + 1, (S, Lq))], axis=-1).astype(np.float32)
    idx = rng.integers(-5, hw, size=(S, Lq)).astype(np.int32)
    q = rng.standard_normal((Lq, H, D), dtype=np.float32)
    k = rng.standard_normal((Lk, H, D), dtype=np.float32)
    v = rng.standard_normal((Lk, H, D), dtype=np.float32)
    if kind.startswith("f32"):
        tq, tk, tv = dev(q), dev(k), dev(v)
        tol, ltol = F32_TOL, LSE_F32_TOL
    elif kind == "bf16":
        q, k, v = (W.bf16_round(x) for x in (q, k, v))
        tq, tk, tv = (dev(x, torch.bfloat16) for x in (q, k, v))
        tol, ltol = BF16_TOL, LSE_BF16_TOL
    else:
        q8, k8 = fp8e4m3_bits(q), fp8e4m3_bits(k)
        q, k, v = OA.fp8e4m3_values(q8), OA.fp8e4m3_values(k8), W.bf16_round(v)
        tq = torch.from_numpy(q8).cuda().view(torch.float8_e4m3fn)
        tk = torch.from_numpy(k8).cuda().view(torch.float8_e4m3fn)
        tv = dev(v, torch.bfloat16)
        tol, ltol = BF16_TOL, LSE_BF16_TOL
    print(f"case {case}: {kind} Lq={Lq} Lk={Lk} ({nf} frames of {h}x{w}) H={H} S={S} lam={lam} sigma={sigma:.2f} "
          f"scale={scale:.4f} parts={parts}", flush=True)
    o, lse = rv.biased_chunk_attention(tq, tk, tv, dev(slot), dev(uv) if S else None, dev(idx) if S else None,
                                       h=h, w=w, softmax_scale=scale, lam=lam, sigma=sigma, key_parts=parts)
    torch.cuda.synchronize()
    Oo, Lo = OA.biased_attention(q, k, v, slot, uv if S else np.zeros((0, Lq, 2), np.float32),
                                 idx if S else np.zeros((0, Lq), np.int32), h, w, scale, lam, sigma)
    err, lerr = np.abs(host(o) - Oo).max(), np.abs(host(lse) - Lo).max()
    print(f"  max|dO|={err:.3e} max|dLSE|={lerr:.3e}")
    assert np.isfinite(host(o)).all()
    assert err <= tol and lerr <= ltol


def _scene(rng, n, h, w, p):
    """n depth maps [n, h p, w p]: a tilted plane 2-20 m away plus 1% noise,
    with a few NaN, zero and negative pixels; intrinsics of a 60-100 degree
    field of view centred on the map."""
    Hd, Wd = h * p, w * p
    yy, xx = np.mgrid[0:Hd, 0:Wd].astype(np.float64)
    d = np.empty((n, Hd, Wd), np.float32)
    K = np.empty((n, 4), np.float32)
    for i in range(n):
        z0 = rng.uniform(2.0, 20.0)
        gx, gy = rng.uniform(-0.3, 0.3, 2) * z0 / max(Wd, Hd)
        d[i] = (z0 + gx * (xx - Wd / 2) + gy * (yy - Hd / 2)) * (1.0 + 0.01 * rng.standard_normal((Hd, Wd)))
        bad = rng.random((Hd, Wd))
        d[i][bad < 0.01] = np.nan
        d[i][(bad >= 0.01) & (bad < 0.02)] = 0.0
        d[i][(bad >= 0.02) & (bad < 0.025)] = -1.0
        f = (Wd / 2) / math.tan(math.radians(rng.uniform(30.0, 50.0)))
        K[i] = (f, f * rng.uniform(0.9, 1.1), Wd / 2 + rng.uniform(-1, 1), Hd / 2 + rng.uniform(-1, 1))
    return d, K


def _poses(rng, n, base):
    out = np.empty((n, 4, 4), np.float32)
    for i in range(n):
        R = axis_angle(random_unit(rng), math.radians(rng.uniform(0.0, 12.0))) @ base[:3, :3]
        c = base[:3, 3] + random_unit(rng) * rng.uniform(0.0, 0.4)
        out[i] = pose_from(R, c)
    return out


# (B, Tq, S, h, w, p, bank, shared centres): large cases run a thread per token, small ones a thread
# per (token, source)
SWEEP_REPROJ = [
    (40, 3, 6, 30, 40, 2, False, False), (48, 3, 8, 33, 27, 1, True, False), (1, 1, 1, 1, 1, 1, False, False),
    (3, 2, 5, 7, 11, 3, True, False), (1, 3, 12, 30, 52, 2, True, True), (2, 1, 64, 5, 6, 2, False, True),
    (64, 3, 4, 25, 30, 3, False, True), (5, 1, 3, 40, 1, 2, True, True), (7, 3, 2, 1, 40, 1, False, False),
    (90, 3, 6, 17, 29, 2, True, True),
]


@pytest.mark.parametrize("case", range(len(SWEEP_REPROJ)))
def test_reprojection_random_sweep(case):
    B, Tq, S, h, w, p, bank, shared = SWEEP_REPROJ[case]
    rng = np.random.default_rng(9300 + case)
    eps = float(rng.choice([0.0, 0.05, 0.2]))
    base = pose_from(axis_angle(random_unit(rng), rng.uniform(0, math.pi)), rng.normal(size=3))
    td, tk = _scene(rng, B * Tq, h, w, p)
    tc = _poses(rng, B * Tq, base)
    n_src = B * S if not bank else int(rng.integers(max(1, S // 2), 3 * S + 2))
    sd, sk = _scene(rng, n_src, h, w, p)
    sc = _poses(rng, n_src, base)
    sel = rng.integers(-2, n_src + 2, size=(B, S)).astype(np.int32) if bank else None
    if shared:  # sources at the centre of one of their problem's target frames (turning in place)
        if bank:
            for b in range(B):
                if 0 <= sel[b, 0] < n_src:
                    sc[sel[b, 0], :3, 3] = tc[b * Tq + int(rng.integers(0, Tq)), :3, 3]
        else:
            for f in range(0, n_src, 2):
                sc[f, :3, 3] = tc[(f // S) * Tq + int(rng.integers(0, Tq)), :3, 3]
    Hd, Wd = h * p, w * p
    tgt = (td.reshape(B, Tq, Hd, Wd), tc.reshape(B, Tq, 4, 4), tk.reshape(B, Tq, 4))
    print(f"case {case}: B={B} Tq={Tq} S={S} grid {h}x{w} p={p} bank={bank} shared centres={shared} eps={eps}",
          flush=True)
    if bank:
        guv, gidx = rv.reproject_correspondence(*[dev(a) for a in tgt], dev(sd), dev(sc), dev(sk), p=p, eps=eps,
                                                src_sel=dev(sel))
    else:
        src = (sd.reshape(B, S, Hd, Wd), sc.reshape(B, S, 4, 4), sk.reshape(B, S, 4))
        guv, gidx = rv.reproject_correspondence(*[dev(a) for a in tgt], *[dev(a) for a in src], p=p, eps=eps)
    guv, gidx = host(guv), host(gidx)
    checked = range(B) if B <= 8 else sorted({0, 1, B // 2, B - 1, *rng.choice(B, 4, replace=False).tolist()})
    for b in checked:
        if bank:
            sel_b = np.where((sel[b] >= 0) & (sel[b] < n_src), sel[b], -1)
            ouv, oidx = OR.reproject(tgt[0][b], tgt[1][b], tgt[2][b], sd, sc, sk, p, eps, src_sel=sel_b)
        else:
            ouv, oidx = OR.reproject(tgt[0][b], tgt[1][b], tgt[2][b], src[0][b], src[1][b], src[2][b], p, eps)
        exempt = OR.boundary_margin(ouv, p, h, w) < 1e-4
        bad_idx = (gidx[b] != oidx) & ~exempt
        bad_uv = ~same_bits_f32(guv[b], ouv).all(axis=-1) & ~exempt
        print(f"  problem {b}: valid={np.mean(oidx >= 0):.3f} exempt={int(exempt.sum())} "
              f"idx_mismatch={int(bad_idx.sum())} uv_mismatch={int(bad_uv.sum())}")
        assert not bad_idx.any() and not bad_uv.any()
