"""Pins for the biased-attention oracle (Sec. 4.3, Eq. bias; design choices (ii), (iii)).

* lambda = 0 equals PyTorch's scaled_dot_product_attention in float64;
* every query whose correspondences were all rejected gets exactly the
  plain attention row (exact fallback);
* rows of the softmax sum to one: a constant V comes back unchanged;
* with Q = 0 the weights are exp(lambda B) on biased columns and 1 elsewhere
  (the multiplicative reading of the bias), checked with one-hot V against
  hand-computed ratios on a non-square grid;
* Lk = 1 returns that key's value;
* a pure-Python brute force agrees on the tiny workload.
"""

import math

import numpy as np
import pytest
import torch

from oracle import attention as A, brute, reprojection as R
from workloads import make_c1


def _rand(rng, *shape):
    return rng.standard_normal(shape)


def test_lambda_zero_is_plain_sdpa():
    rng = np.random.default_rng(0)
    Lq, Lk, H, D = 40, 96, 3, 16
    q, k, v = _rand(rng, Lq, H, D), _rand(rng, Lk, H, D), _rand(rng, Lk, H, D)
    slot = np.array([0, -1, 1, -1, 0, -1], np.int32)  # hw = 16
    uv = rng.uniform(0, 4, size=(2, Lq, 2))
    idx = rng.integers(-4, 16, size=(2, Lq))
    O, lse = A.biased_attention(q, k, v, slot, uv, idx, 4, 4, 0.25, 0.0, 2.0)
    tq = torch.from_numpy(q).permute(1, 0, 2)
    tk = torch.from_numpy(k).permute(1, 0, 2)
    tv = torch.from_numpy(v).permute(1, 0, 2)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, scale=0.25).permute(1, 0, 2).numpy()
    np.testing.assert_allclose(O, ref, atol=1e-12)
    ref_lse = torch.logsumexp(torch.einsum("hqd,hkd->hqk", tq, tk) * 0.25, dim=-1).numpy()
    np.testing.assert_allclose(lse, ref_lse, atol=1e-12)


def test_rejected_rows_fall_back_exactly():
    rng = np.random.default_rng(1)
    Lq, Lk, H, D = 16, 64, 2, 8
    q, k, v = _rand(rng, Lq, H, D), _rand(rng, Lk, H, D), _rand(rng, Lk, H, D)
    slot = np.array([0, 1, -1, -1], np.int32)
    uv = rng.uniform(0, 4, size=(2, Lq, 2))
    idx = rng.integers(0, 16, size=(2, Lq))
    idx[:, 5] = -3
    idx[:, 9] = [-4, -1]
    O, lse = A.biased_attention(q, k, v, slot, uv, idx, 4, 4, 0.3, 1.5, 1.0)
    O0, lse0 = A.biased_attention(q, k, v, slot, uv, idx, 4, 4, 0.3, 0.0, 1.0)
    assert np.array_equal(O[[5, 9]], O0[[5, 9]])
    assert np.array_equal(lse[:, [5, 9]], lse0[:, [5, 9]])
    assert not np.allclose(O[0], O0[0])


def test_rows_sum_to_one():
    rng = np.random.default_rng(2)
    Lq, Lk, H, D = 12, 48, 1, 4
    q, k = _rand(rng, Lq, H, D) * 3, _rand(rng, Lk, H, D) * 3
    v = np.full((Lk, H, D), 2.75)
    slot = np.array([0, -1, 1], np.int32)
    uv = rng.uniform(0, 4, size=(2, Lq, 2))
    idx = rng.integers(0, 16, size=(2, Lq))
    O, _ = A.biased_attention(q, k, v, slot, uv, idx, 4, 4, 1.0, 3.0, 0.7)
    np.testing.assert_allclose(O, 2.75, atol=1e-12)


def test_zero_query_weights_are_gaussian_on_grid():
    """Q = 0, one retrieved frame on a 3x5 grid, V = identity: O is the weight
    vector. u^ at the centre of key (x=2, y=1) = index 7."""
    h, w = 3, 5
    Lk = h * w
    lam, sigma = 1.0, 2.0
    q = np.zeros((1, 1, Lk))
    k = _rand(np.random.default_rng(3), Lk, 1, Lk)
    v = np.eye(Lk)[:, None, :]
    uv = np.array([[[2.5, 1.5]]])
    O, lse = A.biased_attention(q, k, v, np.array([0]), uv, np.array([[7]]), h, w, 1.0, lam, sigma)
    P = O[0, 0]
    c = lam / (2 * sigma ** 2)
    assert P.argmax() == 7
    np.testing.assert_allclose(P[7] / P[8], math.exp(c * 1), rtol=1e-12)   # one step in x
    np.testing.assert_allclose(P[7] / P[2], math.exp(c * 1), rtol=1e-12)   # one step in y
    np.testing.assert_allclose(P[7] / P[0], math.exp(c * 5), rtol=1e-12)   # (2, 1) away
    np.testing.assert_allclose(P[7] / P[14], math.exp(c * 5), rtol=1e-12)  # (2, 1) away
    np.testing.assert_allclose(P[7] / P[10], math.exp(c * 5), rtol=1e-12)  # (x0, y2): (2, 1) away
    # exact multiplicative form and LSE: sum_k exp(lam B_k)
    tot = sum(math.exp(-c * ((x + 0.5 - 2.5) ** 2 + (y + 0.5 - 1.5) ** 2)) for y in range(h) for x in range(w))
    np.testing.assert_allclose(lse[0, 0], math.log(tot), rtol=1e-12)


def test_zero_query_off_centre_asymmetric():
    """Non-square grid and an off-centre u^ catch an x/y swap or a missing
    half-cell offset."""
    h, w = 2, 7
    lam, sigma = 0.75, 1.25  # exactly representable in fp32, as the interface carries them
    v = np.eye(3 * h * w)[:, None, :]
    q = np.zeros((1, 1, 3 * h * w))
    k = np.zeros((3 * h * w, 1, 3 * h * w))
    slot = np.array([-1, 0, -1])
    uv = np.array([[[5.2, 0.3]]])
    O, _ = A.biased_attention(q, k, v, slot, uv, np.array([[5]]), h, w, 1.0, lam, sigma)
    P = O[0, 0]
    wts = np.ones(3 * h * w)
    for t in range(h * w):
        ky, kx = divmod(t, w)
        wts[h * w + t] = math.exp(-lam * ((kx + 0.5 - 5.2) ** 2 + (ky + 0.5 - 0.3) ** 2) / (2 * sigma ** 2))
    np.testing.assert_allclose(P, wts / wts.sum(), rtol=1e-12)


def test_single_key_returns_its_value():
    rng = np.random.default_rng(4)
    q, k, v = _rand(rng, 5, 2, 8), _rand(rng, 1, 2, 8), _rand(rng, 1, 2, 8)
    O, _ = A.biased_attention(q, k, v, np.array([-1]), None, None, 1, 1, 0.35, 1.0, 2.0)
    np.testing.assert_allclose(O, np.broadcast_to(v[0], O.shape), atol=1e-14)


def test_row_sampling_matches_full():
    rng = np.random.default_rng(6)
    Lq, Lk, H, D = 30, 80, 2, 8
    q, k, v = _rand(rng, Lq, H, D), _rand(rng, Lk, H, D), _rand(rng, Lk, H, D)
    slot = np.array([0, -1, 1, -1, -1], np.int32)
    uv = rng.uniform(0, 4, size=(2, Lq, 2))
    idx = rng.integers(-2, 16, size=(2, Lq))
    O, lse = A.biased_attention(q, k, v, slot, uv, idx, 4, 4, 0.3, 1.0, 2.0, block=7)
    rows = np.array([3, 17, 29])
    Os, lses = A.biased_attention(q, k, v, slot, uv, idx, 4, 4, 0.3, 1.0, 2.0, rows=rows, heads=[1])
    np.testing.assert_allclose(Os[:, 0], O[rows, 1], atol=1e-13)
    np.testing.assert_allclose(lses[0], lse[1, rows], atol=1e-13)


def test_brute_force_agrees_on_tiny_workload():
    c1 = make_c1()
    uv, idx = R.reproject(c1.tgt_depth, c1.tgt_c2w, c1.tgt_K, c1.src_depth, c1.src_c2w, c1.src_K, c1.p, c1.eps)
    O, lse = A.biased_attention(c1.q, c1.k, c1.v, c1.slot, uv, idx, c1.h, c1.w, c1.softmax_scale, c1.lam, c1.sigma)
    hw = c1.h * c1.w
    keys = c1.k[:, 0, :].astype(np.float64).tolist()
    vals = c1.v[:, 0, :].astype(np.float64).tolist()
    scale = float(np.float32(c1.softmax_scale))
    for r in range(0, c1.Lq, 3):
        info = []
        for key in range(c1.Lk):
            s = int(c1.slot[key // hw])
            if s >= 0 and idx[s, r] >= 0:
                ky, kx = divmod(key % hw, c1.w)
                info.append((kx, ky, float(uv[s, r, 0]), float(uv[s, r, 1])))
            else:
                info.append(None)
        out, l = brute.attention_row(c1.q[r, 0].astype(np.float64).tolist(), keys, vals, info, scale,
                                     c1.lam, c1.sigma)
        np.testing.assert_allclose(O[r, 0], out, atol=1e-12)
        assert abs(lse[0, r] - l) < 1e-12


def test_fp8e4m3_decoding_matches_torch_on_every_code():
    """The oracle's e4m3 decoding (fp8-logit attention inputs) against torch's
    float8_e4m3fn for all 256 codes, plus hand values."""
    import torch
    from oracle.attention import fp8e4m3_values
    codes = np.arange(256, dtype=np.uint8)
    got = fp8e4m3_values(codes)
    want = torch.from_numpy(codes).view(torch.float8_e4m3fn).float().numpy().astype(np.float64)
    assert np.array_equal(np.isnan(got), np.isnan(want))
    assert np.array_equal(got[~np.isnan(got)], want[~np.isnan(want)])
    assert fp8e4m3_values(np.array([0x38, 0x7E, 0x01, 0xC4, 0x08]), ).tolist() == [1.0, 448.0, 2.0**-9, -3.0, 2.0**-6]
