"""The seeded input generators: reproducible, in range, shaped as stated."""

import numpy as np
import torch

import workloads as W
from oracle import reprojection as R
from workloads.synth import bf16_bits, look_pose, render_planes


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 100000),
                        np.array([0.0, -0.0, np.inf, -np.inf, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8], np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bf16_bits(x), ref)


def test_c1_reproducible_and_in_range():
    a, b = W.make_c1(), W.make_c1()
    for name in ("q", "k", "v", "tgt_depth", "src_depth", "tgt_c2w", "src_c2w"):
        assert np.array_equal(getattr(a, name), getattr(b, name))
    assert a.q.shape == (64, 1, 64) and a.k.shape == (256, 1, 64)
    for d in (a.tgt_depth, a.src_depth):
        assert d.min() >= 1.0 and d.max() <= 10.0
    assert a.tgt_depth.shape == (1, 16, 16)


def test_c3_shapes_and_inbounds_fraction():
    c3 = W.make_c3()
    assert c3.q.dtype == np.uint16 and c3.q.shape == (4680, 12, 128)
    assert c3.k.shape == (28080, 12, 128)
    assert c3.slot.tolist() == [-1] * 3 + list(range(6)) + [-1] * 9
    assert c3.src_depth.shape == (6, 60, 104)
    assert c3.src_depth.min() >= 0.5 and c3.src_depth.max() <= 50.0
    _, idx = R.reproject(c3.tgt_depth, c3.tgt_c2w, c3.tgt_K, c3.src_depth, c3.src_c2w, c3.src_K, c3.p, c3.eps)
    on_grid = ((idx >= 0) | (idx == R.OCCLUDED)).mean()
    assert 0.6 < on_grid < 0.8


def test_bank_workloads_geometry():
    c4 = W.make_c4(qkv=False)
    r = c4.retrieval
    assert r.bank_c2w.shape == (200, 4, 4) and r.bank_frame_depth.shape == (600, 60, 104)
    assert r.query_frame_depth.shape == (8, 3, 60, 104)
    # bank entry j is the middle frame of chunk j
    assert np.array_equal(r.bank_c2w[5], r.bank_frame_c2w[16])
    # the camera stays on the circle of radius 20 m at 1.5 m height
    c = r.bank_frame_c2w[:, :3, 3]
    np.testing.assert_allclose(np.hypot(c[:, 0], c[:, 1]), 20.0, rtol=1e-6)
    np.testing.assert_allclose(c[:, 2], 1.5)
    c5 = W.make_c5(qkv=False)
    assert c5.retrieval.bank_frame_depth.shape == (900, 90, 160)
    assert c5.Lk == 64800 and c5.Lq == 10800


def test_renderer_fronto_parallel_plane():
    # camera at the origin looking along +x; wall x = 7 -> planar depth 7 everywhere
    c2w = look_pose([0.0, 0.0, 0.0], yaw=0.0)
    d = render_planes(c2w, [4.0, 4.0, 4.0, 3.0], 6, 8, [(np.array([1.0, 0, 0]), 7.0)], 0.5, 50.0)
    np.testing.assert_allclose(d, 7.0, rtol=1e-12)


def test_reproj_batch_tiles_distinct_problems():
    arrs = W.make_reproj_batch(40, distinct=8)
    assert arrs[0].shape == (40, 3, 60, 104) and arrs[3].shape == (40, 6, 60, 104)
    assert np.array_equal(arrs[0][3], arrs[0][11])
    assert not np.array_equal(arrs[0][3], arrs[0][4])


def test_fp8e4m3_encoding_matches_torch():
    import torch
    from workloads.synth import fp8e4m3_bits
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.standard_normal(50000).astype(np.float32) * s for s in (1.0, 0.01, 30.0)] +
                       [np.array([0.0, -0.0, 448.0, -448.0, 2.0**-9, 2.0**-10, 3 * 2.0**-10, -1e-5], np.float32)])
    want = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(fp8e4m3_bits(x), want)


def test_rotation_batch_reproducible_and_shared_centres():
    a, b = W.make_rotation_batch(20), W.make_rotation_batch(20)
    for x, y in zip(a, b):
        assert x.dtype == np.float32 and np.array_equal(x, y)
    tc, tk, sc, sk = a
    assert tc.shape == (20, 3, 4, 4) and tk.shape == (20, 3, 4) and sc.shape == (20, 6, 4, 4) and sk.shape == (20, 6, 4)
    # one camera centre per problem, exactly (in fp32)
    centres = np.concatenate([tc[:, :, :3, 3], sc[:, :, :3, 3]], axis=1)
    assert np.array_equal(centres, np.broadcast_to(centres[:, :1], centres.shape))
    # 16 distinct problems tiled to 20
    assert np.array_equal(tc[16:], tc[:4]) and not np.array_equal(tc[1], tc[0])
    # horizontal FOV of the sources: 90 degrees for rotation clips, 90 down to 35 for zoom clips
    fov = np.degrees(2 * np.arctan((104 / 2) / sk[..., 0].astype(np.float64)))
    assert np.allclose(fov[0::2], 90.0, atol=1e-3)
    assert np.allclose(fov[1::2, 0], 90.0, atol=1e-3) and np.allclose(fov[1::2, -1], 35.0, atol=1e-3)
    # the oracle finds the mix of outcomes the recipe states
    _, idx = R.reproject_rotation(tc[0], tk[0], sc[0], sk[0], 30, 52, 2)
    assert (idx >= 0).mean() > 0.3 and (idx == R.CENTRE_MOVED).sum() == 0
