"""GPU parity: the HIP path (through the C interface) against the fp64 oracle.

Bars (written here, not derived from the kernels):
* retrieval: chunk ids, counts and frame selections bit-exact; scores equal
  to the oracle's fp64 score rounded to fp32, bit for bit;
* reprojection: codes and u^ (fp32) bit-exact, except tokens whose u^ lies
  within 1e-4 depth-map pixels of a token-cell boundary, which are counted
  (expected: none, since both sides evaluate the same IEEE double
  expressions);
* attention: max |O - O_oracle| <= 1e-4 for fp32 inputs and <= 2e-2 for
  bf16 inputs (fp32 accumulation), |LSE - LSE_oracle| <= 1e-4 (fp32) and
  <= 4e-3 (bf16). The bf16 LSE bar follows from the arithmetic: the row sum
  adds the probabilities as rounded to bf16 for P V, each off by at most the
  bf16 unit roundoff 2^-8, so LSE can be off by up to ln(1 + 2^-8) = 3.9e-3
  (the logits themselves see exact bf16 inputs and fp32 bias factors, ~1e-5).
  These bars cannot see a subtle bias-geometry error (a half-cell u^ shift
  moves O by ~5e-4 here). The fp32 runs pin the fp32 kernel, which evaluates
  the bias per logit; the bf16 / fp8 kernel's own bias tables are pinned by
  tests/test_gpu_bias_geometry.py, whose case makes the bias the only input
  of the logits and whose bar is relative.
"""

from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import paper_2607_21848_amd as rv
import workloads as W
from oracle import attention as OA, reprojection as OR, retrieval as ORT
from tests.gpu_helpers import dev, dev_bf16, host, qkv_dev, sample_rows, same_bits_f32

pytestmark = pytest.mark.gpu

F32_TOL, BF16_TOL = 1e-4, 2e-2
LSE_F32_TOL, LSE_BF16_TOL = 1e-4, 4e-3


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rv.lib()
    yield
    torch.cuda.synchronize()


# --------------------------------------------------------------------------
# retrieval
# --------------------------------------------------------------------------
def _gpu_retrieve(r, F=None, k=None):
    idx, sc, cnt, sel = rv.retrieve_chunks(dev(r.bank_c2w), dev(r.query_c2w), dev(r.query_chunk), E=r.E, w_v=r.w_v,
                                           tau_c=r.tau_c, tau_v=r.tau_v, delta=r.delta,
                                           first_candidate=r.first_candidate, k=k or r.k, frames_per_chunk=F)
    return host(idx), host(sc), host(cnt), (host(sel) if sel is not None else None)


def _check_retrieval(r, k=None):
    k = k or r.k
    oi, osc, oc = ORT.retrieve(r.bank_c2w, r.query_c2w, r.query_chunk, r.E, r.w_v, r.tau_c, r.tau_v, r.delta,
                               r.first_candidate, k)
    gi, gsc, gc, gsel = _gpu_retrieve(r, F=3, k=k)
    ties, margins = ORT.near_ties(r.bank_c2w, r.query_c2w, r.query_chunk, r.E, r.w_v, r.tau_c, r.tau_v, r.delta,
                                  r.first_candidate, k)
    print(f"retrieval: Q={len(oc)} k={k} counts={oc.tolist()} near_ties={ties} gate_margins={margins}")
    assert np.array_equal(gc, oc)
    assert np.array_equal(gi, oi)
    assert np.array_equal(gsc.view(np.uint32), osc.astype(np.float32).view(np.uint32))
    assert np.array_equal(gsel, ORT.frame_selection(oi, oc, 3))


def test_retrieval_history_bank_c4():
    _check_retrieval(W.make_c4(qkv=False).retrieval)


def test_retrieval_history_bank_c5():
    _check_retrieval(W.make_c5(qkv=False).retrieval)


@pytest.mark.parametrize("k", [1, 5, 32])
def test_retrieval_k_range(k):
    _check_retrieval(W.make_c4(qkv=False).retrieval, k=k)


def test_retrieval_random_banks_and_edges():
    from workloads.synth import axis_angle, pose_from, random_unit
    rng = np.random.default_rng(7)
    for N in (0, 1, 63, 64, 65, 1000, 5000):
        bank = np.stack([pose_from(axis_angle(random_unit(rng), rng.uniform(0, 0.8)), rng.normal(0, 1.5, 3))
                         for _ in range(max(N, 1))])[:N].astype(np.float32).reshape(N, 4, 4)
        Q = 9
        qpose = np.stack([pose_from(axis_angle(random_unit(rng), rng.uniform(0, 0.8)), rng.normal(0, 1.5, 3))
                          for _ in range(Q)]).astype(np.float32)
        qchunk = rng.integers(0, N + 10, size=Q).astype(np.int32)
        r = W.configs.Retrieval(bank_c2w=bank, query_c2w=qpose, query_chunk=qchunk, E=5.0, w_v=0.5, tau_c=0.4,
                                tau_v=0.9, delta=3, first_candidate=1, k=6)
        _check_retrieval(r)


def test_retrieval_duplicates_tie_by_index():
    bank = np.tile(np.eye(4, dtype=np.float32), (100, 1, 1))
    r = W.configs.Retrieval(bank_c2w=bank, query_c2w=np.eye(4, dtype=np.float32)[None],
                            query_chunk=np.array([103], np.int32), E=1.0, w_v=0.5, tau_c=0.1, tau_v=0.5, delta=3,
                            first_candidate=2, k=8)
    gi, gsc, gc, _ = _gpu_retrieve(r)
    assert gc[0] == 8 and gi[0].tolist() == list(range(2, 10)) and (gsc[0] == 0).all()


@pytest.mark.parametrize("N,k", [(8193, 4), (20000, 32), (100003, 4)])
def test_retrieval_segmented_banks(N, k):
    """Banks above 8192 entries take the segmented scan (one wave per 1024
    entries, then a merge): same results as the oracle, bit for bit."""
    from workloads.synth import ring_bank
    rng = np.random.default_rng(N)
    bank = ring_bank(rng, N, radius=6.0)
    q = ring_bank(rng, 5, radius=6.0)
    qchunk = np.array([N + 10, N // 2, 5, N - 1, 3 * N // 4], np.int32)
    r = W.configs.Retrieval(bank_c2w=bank, query_c2w=q, query_chunk=qchunk, E=12.0, w_v=0.5, tau_c=0.1,
                            tau_v=0.8, delta=3, first_candidate=1, k=k)
    _check_retrieval(r)


def test_retrieval_segmented_ties_cross_segments():
    """Equal scores in every segment: the merge keeps the smallest indices."""
    bank = np.tile(np.eye(4, dtype=np.float32), (20000, 1, 1))
    r = W.configs.Retrieval(bank_c2w=bank, query_c2w=np.eye(4, dtype=np.float32)[None],
                            query_chunk=np.array([30000], np.int32), E=1.0, w_v=0.5, tau_c=0.1, tau_v=0.5,
                            delta=3, first_candidate=4000, k=32)
    gi, gsc, gc, _ = _gpu_retrieve(r)
    assert gc[0] == 32 and gi[0].tolist() == list(range(4000, 4032)) and (gsc[0] == 0).all()


def test_retrieval_stress_bank_512mib():
    """The 2^23-entry (512 MiB) stress bank of the retrieval bandwidth figure,
    one query, top-4: identical to the oracle."""
    from workloads.synth import ring_bank
    rng = np.random.default_rng(23)
    N = 1 << 23
    bank = ring_bank(rng, N, radius=20.0)
    q = ring_bank(rng, 1, radius=20.0)
    r = W.configs.Retrieval(bank_c2w=bank, query_c2w=q, query_chunk=np.array([N + 5], np.int32), E=40.0,
                            w_v=0.5, tau_c=0.05, tau_v=float(np.pi / 4), delta=3, first_candidate=1, k=4)
    _check_retrieval(r)


# --------------------------------------------------------------------------
# reprojection
# --------------------------------------------------------------------------
def _compare_reprojection(ouv, oidx, guv, gidx, p, h, w, label):
    exempt = OR.boundary_margin(ouv, p, h, w) < 1e-4
    bad_idx = (gidx != oidx) & ~exempt
    bad_uv = ~same_bits_f32(guv, ouv).all(axis=-1) & ~exempt
    print(f"reprojection {label}: pairs={oidx.size} valid={np.mean(oidx >= 0):.3f} "
          f"on_grid={np.mean((oidx >= 0) | (oidx == -4)):.3f} boundary_exempt={int(exempt.sum())} "
          f"idx_mismatch={int(bad_idx.sum())} uv_mismatch={int(bad_uv.sum())}")
    assert not bad_idx.any()
    assert not bad_uv.any()


@pytest.mark.parametrize("cfg", [1, 3])
def test_reprojection_fixed_sources(cfg):
    wl = W.make_c1() if cfg == 1 else W.make_c3()
    ouv, oidx = OR.reproject(wl.tgt_depth, wl.tgt_c2w, wl.tgt_K, wl.src_depth, wl.src_c2w, wl.src_K, wl.p, wl.eps)
    guv, gidx = rv.reproject_correspondence(dev(wl.tgt_depth), dev(wl.tgt_c2w), dev(wl.tgt_K), dev(wl.src_depth),
                                            dev(wl.src_c2w), dev(wl.src_K), p=wl.p, eps=wl.eps)
    ties = OR.visibility_near_ties(wl.tgt_depth, wl.tgt_c2w, wl.tgt_K, wl.src_depth, wl.src_c2w, wl.src_K, wl.p,
                                   wl.eps)
    print(f"C{cfg}: visibility near ties (|[X_s]_z - (1 + eps) D_s| < 1e-9 D_s): {ties}")
    _compare_reprojection(ouv, oidx, host(guv), host(gidx), wl.p, wl.h, wl.w, f"C{cfg}")


@pytest.mark.parametrize("cfg", [4, 5])
def test_retrieval_then_reprojection_on_device(cfg):
    """Retrieval output feeds reprojection on the device (no host round trip)."""
    wl = W.make_config(cfg, qkv=False)
    r = wl.retrieval
    oi, osc, oc = ORT.retrieve(r.bank_c2w, r.query_c2w, r.query_chunk, r.E, r.w_v, r.tau_c, r.tau_v, r.delta,
                               r.first_candidate, r.k)
    osel = ORT.frame_selection(oi, oc, 3)
    gidx_c, _, _, gsel = rv.retrieve_chunks(dev(r.bank_c2w), dev(r.query_c2w), dev(r.query_chunk), E=r.E,
                                            w_v=r.w_v, tau_c=r.tau_c, tau_v=r.tau_v, delta=r.delta,
                                            first_candidate=r.first_candidate, k=r.k, frames_per_chunk=3)
    bank = (dev(r.bank_frame_depth), dev(r.bank_frame_c2w), dev(r.bank_frame_K))
    guv, gidx = rv.reproject_correspondence(dev(r.query_frame_depth), dev(r.query_frame_c2w), dev(r.query_frame_K),
                                            *bank, p=wl.p, eps=wl.eps, src_sel=gsel)
    guv, gidx = host(guv), host(gidx)
    for qi in range(len(oc)):
        ouv, oidx = OR.reproject(r.query_frame_depth[qi], r.query_frame_c2w[qi], r.query_frame_K[qi],
                                 r.bank_frame_depth, r.bank_frame_c2w, r.bank_frame_K, wl.p, wl.eps,
                                 src_sel=osel[qi])
        ties = OR.visibility_near_ties(r.query_frame_depth[qi], r.query_frame_c2w[qi], r.query_frame_K[qi],
                                       r.bank_frame_depth, r.bank_frame_c2w, r.bank_frame_K, wl.p, wl.eps,
                                       src_sel=osel[qi])
        print(f"C{cfg} query {qi}: visibility near ties: {ties}")
        _compare_reprojection(ouv, oidx, guv[qi], gidx[qi], wl.p, wl.h, wl.w, f"C{cfg} query {qi}")


def test_reprojection_batched_and_no_source():
    arrs = W.make_reproj_batch(6, distinct=3)
    tgt = [dev(a) for a in arrs[:3]]
    guv, gidx = rv.reproject_correspondence(*tgt, *[dev(a) for a in arrs[3:]], p=2, eps=0.05)
    guv, gidx = host(guv), host(gidx)
    for b in range(6):
        ouv, oidx = OR.reproject(arrs[0][b], arrs[1][b], arrs[2][b], arrs[3][b], arrs[4][b], arrs[5][b], 2, 0.05)
        _compare_reprojection(ouv, oidx, guv[b], gidx[b], 2, 30, 52, f"batch {b}")
    # a frame bank with selections, including empty and out-of-range slots
    bank_d = arrs[3].reshape(-1, 60, 104)
    bank_c = arrs[4].reshape(-1, 4, 4)
    bank_k = arrs[5].reshape(-1, 4)
    sel = np.array([[0, 5, -1, 7, 35, 36], [3, -7, 2, 1000, 0, 9]], np.int32)
    guv, gidx = rv.reproject_correspondence(*[dev(a[:2]) for a in arrs[:3]], dev(bank_d), dev(bank_c),
                                            dev(bank_k), p=2, eps=0.05, src_sel=dev(sel))
    guv, gidx = host(guv), host(gidx)
    for b in range(2):
        sel_b = np.where((sel[b] >= 0) & (sel[b] < len(bank_d)), sel[b], -1)
        ouv, oidx = OR.reproject(arrs[0][b], arrs[1][b], arrs[2][b], bank_d, bank_c, bank_k, 2, 0.05,
                                 src_sel=sel_b)
        _compare_reprojection(ouv, oidx, guv[b], gidx[b], 2, 30, 52, f"bank {b}")
    assert (gidx[0, 2] == -5).all() and (gidx[1, 1] == -5).all() and (gidx[1, 3] == -5).all()


def test_reprojection_outside_the_shared_reciprocal_range():
    """The quotients of Eq. reprojection share one reciprocal of [X_s]_z only
    where every frame value and the target depth lie in the range where that
    equals IEEE division; elsewhere the kernel divides. Both paths, bit-exact
    against the oracle: problem 0 in range; problem 1 with a band of target
    depths at 1e-13 m and another at 1e13 m (defined, out of range: their waves
    divide); problem 2 with a source centre 1e21 m away and problem 3 with a
    source principal point of -0 (their blocks divide)."""
    arrs = [a.copy() for a in W.make_reproj_batch(4, distinct=2)]
    tgt_d, tgt_c, tgt_k, src_d, src_c, src_k = arrs
    tgt_d[1, 0, 10:14, :] = 1e-13
    tgt_d[1, 1, 30:34, :] = 1e13
    src_c[2, 3, 0, 3] = 1e21
    src_k[3, 4, 2] = -0.0
    for B in (4, 1):
        guv, gidx = rv.reproject_correspondence(*[dev(a[:B]) for a in arrs], p=2, eps=0.05)
        guv, gidx = host(guv), host(gidx)
        for b in range(B):
            ouv, oidx = OR.reproject(*[a[b] for a in arrs], 2, 0.05)
            _compare_reprojection(ouv, oidx, guv[b], gidx[b], 2, 30, 52, f"range case {b} (batch {B})")
    assert (gidx[0] >= 0).mean() > 0.4


def test_reprojection_per_token_and_per_source_launches_agree():
    """A launch of 32 problems runs one thread per token (looping over the
    sources); a launch of one problem, too small to fill the GPU that way,
    runs one thread per (token, source). Both give the same bits, and the
    oracle's on sampled problems."""
    B = 32
    arrs = W.make_reproj_batch(B, distinct=4)
    guv, gidx = rv.reproject_correspondence(*[dev(a) for a in arrs], p=2, eps=0.05)
    guv, gidx = host(guv), host(gidx)
    for b in range(B):
        suv, sidx = rv.reproject_correspondence(*[dev(a[b:b + 1]) for a in arrs], p=2, eps=0.05)
        assert np.array_equal(host(sidx)[0], gidx[b])
        assert np.array_equal(host(suv)[0].view(np.uint32), guv[b].view(np.uint32))
    for b in (0, 3, 31):
        ouv, oidx = OR.reproject(*[a[b] for a in arrs], 2, 0.05)
        _compare_reprojection(ouv, oidx, guv[b], gidx[b], 2, 30, 52, f"batch-32 problem {b}")
    # the same with source frames selected from a shared bank (empty and out-of-range slots included)
    bank = [dev(a.reshape(-1, *a.shape[2:])) for a in arrs[3:]]
    n_bank = B * arrs[3].shape[1]
    rng = np.random.Generator(np.random.PCG64(77))
    sel = rng.integers(-2, n_bank + 3, size=(B, 6)).astype(np.int32)
    tgt = [dev(a) for a in arrs[:3]]
    guv, gidx = rv.reproject_correspondence(*tgt, *bank, p=2, eps=0.05, src_sel=dev(sel))
    guv, gidx = host(guv), host(gidx)
    for b in range(B):
        suv, sidx = rv.reproject_correspondence(*[t[b:b + 1] for t in tgt], *bank, p=2, eps=0.05,
                                                src_sel=dev(sel[b:b + 1]))
        assert np.array_equal(host(sidx)[0], gidx[b])
        assert np.array_equal(host(suv)[0].view(np.uint32), guv[b].view(np.uint32))
    bank_h = [a.reshape(-1, *a.shape[2:]) for a in arrs[3:]]
    for b in (1, 30):
        sel_b = np.where((sel[b] >= 0) & (sel[b] < n_bank), sel[b], -1)
        ouv, oidx = OR.reproject(arrs[0][b], arrs[1][b], arrs[2][b], *bank_h, 2, 0.05, src_sel=sel_b)
        _compare_reprojection(ouv, oidx, guv[b], gidx[b], 2, 30, 52, f"batch-32 bank problem {b}")


@pytest.mark.parametrize("B", [1, 32])
def test_reprojection_fixed_centre_sources(B):
    """Cameras that turn in place: every source of a problem shares the
    centre of its target frame 0 (c_t - c_s is exactly zero, where Eq.
    reprojection reduces to a homography, Sec. 4.3), and in every other
    problem frame 1 shares it too; one problem (a thread per (token, source))
    and 32 (a thread per token), bit-exact against the oracle."""
    arrs = [a.copy() for a in W.make_reproj_batch(B, distinct=4)]
    tgt_d, tgt_c, tgt_k, src_d, src_c, src_k = arrs
    S = src_c.shape[1]
    src_c[:, :, :3, 3] = tgt_c[:, 0:1, :3, 3]
    tgt_c[:, 1, :3, 3] = np.where(np.arange(B)[:, None] % 2 == 0, tgt_c[:, 0, :3, 3], tgt_c[:, 1, :3, 3])
    guv, gidx = rv.reproject_correspondence(*[dev(a) for a in arrs], p=2, eps=0.05)
    guv, gidx = host(guv), host(gidx)
    for b in sorted({0, B // 2, B - 1}):
        ouv, oidx = OR.reproject(*[a[b] for a in arrs], 2, 0.05)
        _compare_reprojection(ouv, oidx, guv[b], gidx[b], 2, 30, 52, f"fixed centre, problem {b}")
        assert (oidx >= 0).mean() > 0.3


def test_pooled_depth_and_reprojection_on_pooled_maps():
    """pool_token_depth bit-exact against the oracle's pooling rounded to fp32
    (NaN, inf, zero and negative pixels included); reprojection with p = 1 on
    pooled maps and token-grid intrinsics bit-exact against the oracle on the
    same maps; and, on maps whose 2 x 2 blocks are constant (exact pooling),
    bit-identical to the full-resolution call with p = 2."""
    arrs = W.make_reproj_batch(4, distinct=2)
    tgt_d, tgt_c, tgt_k, src_d, src_c, src_k = arrs
    B, Tq, Hd, Wd = tgt_d.shape
    S = src_d.shape[1]
    noisy = tgt_d.copy()
    noisy[0, 0, :4, :4] = [[np.nan, 1.0, 0.0, -2.0], [np.inf, 3.0, 5.0, 5.0], [1e-30, 1e30, 7.0, 7.0], [2.0, 2.0, 7.0, 7.0]]
    pooled = host(rv.pool_token_depth(dev(noisy.reshape(-1, Hd, Wd)), 2)).reshape(B, Tq, Hd // 2, Wd // 2)
    want = OR.pooled_depth(noisy, 2).astype(np.float32)
    assert np.array_equal(np.isnan(pooled), np.isnan(want))
    ok = ~np.isnan(want)
    assert np.array_equal(pooled[ok].view(np.uint32), want[ok].view(np.uint32))
    # p = 1 on pooled maps against the oracle on the same maps
    ptgt = OR.pooled_depth(tgt_d, 2).astype(np.float32)
    psrc = OR.pooled_depth(src_d, 2).astype(np.float32)
    ktok_t = (tgt_k.astype(np.float64) / 2).astype(np.float32)
    ktok_s = (src_k.astype(np.float64) / 2).astype(np.float32)
    guv, gidx = rv.reproject_correspondence(dev(ptgt), dev(tgt_c), dev(ktok_t), dev(psrc), dev(src_c), dev(ktok_s),
                                            p=1, eps=0.05)
    guv, gidx = host(guv), host(gidx)
    for b in range(B):
        ouv, oidx = OR.reproject(ptgt[b], tgt_c[b], ktok_t[b], psrc[b], src_c[b], ktok_s[b], 1, 0.05)
        _compare_reprojection(ouv, oidx, guv[b], gidx[b], 1, 30, 52, f"pooled {b}")
    # exactly poolable maps: the pooled call equals the full-resolution call bit for bit
    blk_t = np.repeat(np.repeat(ptgt, 2, axis=2), 2, axis=3)
    blk_s = np.repeat(np.repeat(psrc, 2, axis=2), 2, axis=3)
    fuv, fidx = rv.reproject_correspondence(dev(blk_t), dev(tgt_c), dev(tgt_k), dev(blk_s), dev(src_c), dev(src_k),
                                            p=2, eps=0.05)
    assert np.array_equal(host(fidx), gidx)
    assert np.array_equal(host(fuv).view(np.uint32), guv.view(np.uint32))
    assert S == 6 and (gidx >= 0).mean() > 0.4


def test_reprojection_rejection_codes():
    h, w, p = 6, 8, 2
    Kk = np.array([[8.0, 6.0, 8.0, 6.0]], np.float32)
    d = np.full((1, h * p, w * p), 5.0, np.float32)
    d[0, 0:2, 0:2] = np.nan
    d[0, 0:2, 2:4] = 0.0
    eye = np.eye(4, dtype=np.float32)[None]
    turned = eye.copy()
    turned[0, 0, 0] = turned[0, 2, 2] = -1.0
    far = eye.copy()
    far[0, 0, 3] = 40.0
    occl = np.full((1, h * p, w * p), 1.0, np.float32)
    for src_d, src_c, exp in ((d, turned, -2), (d, far, -3), (occl, eye, -4)):
        guv, gidx = rv.reproject_correspondence(dev(d), dev(eye), dev(Kk), dev(src_d), dev(src_c), dev(Kk),
                                                p=p, eps=0.05)
        ouv, oidx = OR.reproject(d, eye, Kk, src_d, src_c, Kk, p, 0.05)
        assert np.array_equal(host(gidx), oidx)
        assert host(gidx)[0, 0] == -1 and host(gidx)[0, 1] == -1
        assert (host(gidx)[0, 2:w] == exp).all()


# --------------------------------------------------------------------------
# attention
# --------------------------------------------------------------------------
def _attn_gpu(wl, q, k, v, uv, idx, lam=None):
    S = 0 if uv is None else uv.shape[0]
    return rv.biased_chunk_attention(q, k, v, dev(wl.slot), dev(uv) if S else None, dev(idx) if S else None,
                                     h=wl.h, w=wl.w, softmax_scale=wl.softmax_scale,
                                     lam=wl.lam if lam is None else lam, sigma=wl.sigma)


def _oracle_corr(wl):
    if wl.S == 0:
        return None, None
    if wl.retrieval is None:
        return OR.reproject(wl.tgt_depth, wl.tgt_c2w, wl.tgt_K, wl.src_depth, wl.src_c2w, wl.src_K, wl.p, wl.eps)
    r = wl.retrieval
    qi = 1 if wl.config_id == 4 else 0
    oi, _, oc = ORT.retrieve(r.bank_c2w, r.query_c2w[qi:qi + 1], r.query_chunk[qi:qi + 1], r.E, r.w_v, r.tau_c,
                             r.tau_v, r.delta, r.first_candidate, r.k)
    sel = ORT.frame_selection(oi, oc, 3)[0]
    return OR.reproject(r.query_frame_depth[qi], r.query_frame_c2w[qi], r.query_frame_K[qi], r.bank_frame_depth,
                        r.bank_frame_c2w, r.bank_frame_K, wl.p, wl.eps, src_sel=sel)


def _check_attention(wl, rows, heads, tol, lse_tol, label):
    uv, idx = _oracle_corr(wl)
    q, k, v = qkv_dev(wl)
    o, lse = _attn_gpu(wl, q, k, v, uv, idx)
    torch.cuda.synchronize()
    o, lse = host(o), host(lse)
    qv, kv, vv = wl.values("q"), wl.values("k"), wl.values("v")
    Oo, Lo = OA.biased_attention(qv, kv, vv, wl.slot, uv, idx, wl.h, wl.w, wl.softmax_scale, wl.lam, wl.sigma,
                                 rows=rows, heads=heads)
    err = np.abs(o[rows][:, heads] - Oo).max()
    lerr = np.abs(lse[heads][:, rows] - Lo).max()
    shift = 0.0
    if uv is not None:
        O0, _ = OA.biased_attention(qv, kv, vv, wl.slot, None, None, wl.h, wl.w, wl.softmax_scale, 0.0, wl.sigma,
                                    rows=rows[:16], heads=heads[:2])
        shift = np.abs(O0 - Oo[:16, :2]).max()
    print(f"attention {label}: rows={len(rows)} heads={len(heads)} max|dO|={err:.3e} (tol {tol}) "
          f"max|dLSE|={lerr:.3e} (tol {lse_tol}) bias moves O by {shift:.3e}")
    assert np.isfinite(o).all()
    assert err <= tol
    assert lerr <= lse_tol


def test_attention_tiny_fp32_full():
    wl = W.make_c1()
    _check_attention(wl, np.arange(wl.Lq), np.arange(wl.H), F32_TOL, LSE_F32_TOL, "C1 fp32")


@pytest.mark.parametrize("cfg", [2, 3, 4])
def test_attention_wan13b_bf16(cfg):
    wl = W.make_config(cfg, "bf16")
    _check_attention(wl, sample_rows(wl.Lq, 48, cfg), np.arange(wl.H), BF16_TOL, LSE_BF16_TOL, f"C{cfg} bf16")


@pytest.mark.parametrize("cfg", [2, 3, 4])
def test_attention_wan13b_fp32(cfg):
    wl = W.make_config(cfg, "f32")
    _check_attention(wl, sample_rows(wl.Lq, 32, cfg), np.arange(wl.H), F32_TOL, LSE_F32_TOL, f"C{cfg} fp32")


def test_attention_history_bank_bf16_every_row_of_one_head():
    """Every query row of the last head at the history-bank shape, in the
    launch configuration the bench times (automatic key split)."""
    wl = W.make_config(4, "bf16")
    _check_attention(wl, np.arange(wl.Lq), np.array([wl.H - 1]), BF16_TOL, LSE_BF16_TOL, "C4 bf16 all rows, head 11")


def test_attention_wan14b_bf16():
    """Every one of the 40 heads (the work units map to XCDs by head), on
    sampled rows."""
    wl = W.make_c5("bf16")
    _check_attention(wl, sample_rows(wl.Lq, 16, 5), np.arange(wl.H), BF16_TOL, LSE_BF16_TOL, "C5 bf16")


def test_attention_wan14b_fp32():
    wl = W.make_c5("f32")
    _check_attention(wl, sample_rows(wl.Lq, 16, 5), np.arange(wl.H), F32_TOL, LSE_F32_TOL, "C5 fp32")


def _synthetic(rng, Lq, Lk, H, D, h, w, S, dtype):
    nf = Lk // (h * w)
    slot = np.full(nf, -1, np.int32)
    frames = rng.choice(nf, size=min(S, nf), replace=False)
    slot[frames] = np.arange(len(frames))
    uv = np.stack([rng.uniform(-1, w + 1, (S, Lq)), rng.uniform(-1, h + 1, (S, Lq))], axis=-1).astype(np.float32)
    idx = rng.integers(-4, h * w, size=(S, Lq)).astype(np.int32)
    q = rng.standard_normal((Lq, H, D), dtype=np.float32)
    k = rng.standard_normal((Lk, H, D), dtype=np.float32)
    v = rng.standard_normal((Lk, H, D), dtype=np.float32)
    if dtype == "bf16":
        q, k, v = (W.bf16_round(x) for x in (q, k, v))
    return q, k, v, slot, uv, idx


@pytest.mark.parametrize("dtype,D", [("f32", 64), ("f32", 128), ("bf16", 128)])
@pytest.mark.parametrize("shape", [(1, 20, 1, 4, 5, 2), (100, 60, 2, 3, 4, 3), (129, 300, 3, 6, 5, 4),
                                   (257, 1560, 2, 30, 52, 1), (300, 4 * 70, 1, 7, 10, 2)])
def test_attention_ragged_shapes(dtype, D, shape):
    """Query counts and key counts that are not multiples of the tiles,
    frames smaller than a key tile (several frames per tile) and larger."""
    Lq, Lk, H, h, w, S = shape
    rng = np.random.default_rng(Lq * 7 + Lk)
    q, k, v, slot, uv, idx = _synthetic(rng, Lq, Lk, H, D, h, w, S, dtype)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    o, lse = rv.biased_chunk_attention(dev(q, tdt), dev(k, tdt), dev(v, tdt), dev(slot), dev(uv), dev(idx), h=h, w=w,
                                       softmax_scale=1.0 / math.sqrt(D), lam=1.0, sigma=2.0)
    Oo, Lo = OA.biased_attention(q, k, v, slot, uv, idx, h, w, 1.0 / math.sqrt(D), 1.0, 2.0)
    err = np.abs(host(o) - Oo).max()
    lerr = np.abs(host(lse) - Lo).max()
    tol, ltol = (F32_TOL, LSE_F32_TOL) if dtype == "f32" else (BF16_TOL, LSE_BF16_TOL)
    print(f"ragged {shape} {dtype} D={D}: max|dO|={err:.3e} max|dLSE|={lerr:.3e}")
    assert err <= tol and lerr <= ltol


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_attention_exact_fallbacks(dtype):
    """lambda = 0, an all-(-1) slot table and all-rejected correspondences
    give bit-identical outputs (design choice (iii))."""
    rng = np.random.default_rng(11)
    Lq, Lk, H, D, h, w, S = 200, 6 * 40, 2, 128, 5, 8, 3
    q, k, v, slot, uv, idx = _synthetic(rng, Lq, Lk, H, D, h, w, S, dtype)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    tq, tk, tv = dev(q, tdt), dev(k, tdt), dev(v, tdt)
    kw = dict(h=h, w=w, softmax_scale=1.0 / math.sqrt(D), sigma=2.0)
    o_lam0, l_lam0 = rv.biased_chunk_attention(tq, tk, tv, dev(slot), dev(uv), dev(idx), lam=0.0, **kw)
    o_noslot, l_noslot = rv.biased_chunk_attention(tq, tk, tv, dev(np.full_like(slot, -1)), dev(uv), dev(idx),
                                                   lam=1.0, **kw)
    o_rej, l_rej = rv.biased_chunk_attention(tq, tk, tv, dev(slot), dev(uv), dev(np.full_like(idx, -3)), lam=1.0,
                                             **kw)
    o_off, l_off = rv.biased_chunk_attention(tq, tk, tv, dev(slot), None, None, lam=1.0, **kw)
    for o_, l_ in ((o_noslot, l_noslot), (o_rej, l_rej), (o_off, l_off)):
        assert torch.equal(o_, o_lam0) and torch.equal(l_, l_lam0)
    o_b, _ = rv.biased_chunk_attention(tq, tk, tv, dev(slot), dev(uv), dev(idx), lam=1.0, **kw)
    assert not torch.equal(o_b, o_lam0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_attention_constant_values_and_single_key(dtype):
    rng = np.random.default_rng(12)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    Lq, H, D = 77, 3, 128
    q = dev(rng.standard_normal((Lq, H, D), dtype=np.float32) * 2, tdt)
    k = dev(rng.standard_normal((1, H, D), dtype=np.float32), tdt)
    v = dev(rng.standard_normal((1, H, D), dtype=np.float32), tdt)
    o, lse = rv.biased_chunk_attention(q, k, v, dev(np.array([-1], np.int32)), None, None, h=1, w=1,
                                       softmax_scale=0.1, lam=1.0, sigma=2.0)
    # one key: its weight is 1 up to the rounding of the max subtraction
    assert (o.float() - v.float().expand(Lq, H, D)).abs().max().item() <= 1e-6
    Lk = 4 * 390
    k = dev(rng.standard_normal((Lk, H, D), dtype=np.float32), tdt)
    v = torch.full((Lk, H, D), 0.75, dtype=tdt, device="cuda:0")
    slot = np.array([0, -1, 1, -1], np.int32)
    uv = np.stack([rng.uniform(0, 30, (2, Lq)), rng.uniform(0, 13, (2, Lq))], -1).astype(np.float32)
    o, _ = rv.biased_chunk_attention(q, k, v, dev(slot), dev(uv), dev(np.zeros((2, Lq), np.int32)), h=13, w=30,
                                     softmax_scale=0.1, lam=1.0, sigma=2.0)
    # fp32: Lk-term fp32 sums of p and p * 0.75 (a few ulps); bf16: p rounded to bf16 in P V only
    assert (o.float() - 0.75).abs().max().item() <= (4e-6 if dtype == "f32" else 4e-3)


_SPLIT_CASE = {}


def _split_case():
    """Lq = 300 (three query tiles, the last ragged), Lk = 40 frames of 7 x 10
    tokens (87.5 key tiles), two heads: 6 items of 88 key tiles."""
    if not _SPLIT_CASE:
        rng = np.random.default_rng(21)
        Lq, Lk, H, D, h, w, S = 300, 40 * 70, 2, 128, 7, 10, 3
        q, k, v, slot, uv, idx = _synthetic(rng, Lq, Lk, H, D, h, w, S, "bf16")
        Oo, Lo = OA.biased_attention(q, k, v, slot, uv, idx, h, w, 1.0 / math.sqrt(D), 1.0, 2.0)
        _SPLIT_CASE.update(dict(args=(q, k, v, slot, uv, idx), hw=(h, w), D=D, ref=(Oo, Lo)))
    return _SPLIT_CASE


@pytest.mark.parametrize("parts", [1, 2, 3, 7, 64])
def test_attention_bf16_key_parts(parts):
    """The bf16 key split at forced part counts on 88 key tiles: 1 (no
    merge), 2 and 3 (parts that start inside KV frames; the last part holds
    the ragged key tile), 7, and 64 (parts of one or two tiles)."""
    c = _split_case()
    q, k, v, slot, uv, idx = c["args"]
    h, w = c["hw"]
    Oo, Lo = c["ref"]
    o, lse = rv.biased_chunk_attention(dev(q, torch.bfloat16), dev(k, torch.bfloat16), dev(v, torch.bfloat16),
                                       dev(slot), dev(uv), dev(idx), h=h, w=w,
                                       softmax_scale=1.0 / math.sqrt(c["D"]), lam=1.0, sigma=2.0, key_parts=parts)
    torch.cuda.synchronize()
    err = np.abs(host(o) - Oo).max()
    lerr = np.abs(host(lse) - Lo).max()
    print(f"bf16 keys in {parts} parts: max|dO|={err:.3e} max|dLSE|={lerr:.3e}")
    assert np.isfinite(host(o)).all()
    assert err <= BF16_TOL and lerr <= LSE_BF16_TOL


def test_empty_query_chunk_is_noop():
    q = torch.empty((0, 2, 128), dtype=torch.bfloat16, device="cuda:0")
    k = torch.zeros((40, 2, 128), dtype=torch.bfloat16, device="cuda:0")
    o, lse = rv.biased_chunk_attention(q, k, k, dev(np.full(2, -1, np.int32)), None, None, h=4, w=5,
                                       softmax_scale=0.1, lam=1.0, sigma=2.0)
    assert o.shape == (0, 2, 128) and lse.shape == (2, 0)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_attention_beyond_staged_frames_and_widest_grid(dtype):
    """Bias edges of the bf16 kernel: 20 retrieved frames (correspondences of
    frames 16.. are loaded on demand, the first 16 come from LDS), and a token
    grid 256 wide (the largest its per-column bias table holds)."""
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    tol, ltol = (F32_TOL, LSE_F32_TOL) if dtype == "f32" else (BF16_TOL, LSE_BF16_TOL)
    for (Lq, nf, H, h, w, S) in ((150, 24, 2, 4, 5, 20), (130, 4, 1, 2, 256, 2)):
        rng = np.random.default_rng(nf * 31 + w)
        Lk = nf * h * w
        q, k, v, slot, uv, idx = _synthetic(rng, Lq, Lk, H, 128, h, w, S, dtype)
        slot = np.full(nf, -1, np.int32)
        slot[nf - S:] = np.arange(S)  # the retrieved frames last, frames >= 16 included
        o, lse = rv.biased_chunk_attention(dev(q, tdt), dev(k, tdt), dev(v, tdt), dev(slot), dev(uv), dev(idx), h=h,
                                           w=w, softmax_scale=1.0 / math.sqrt(128), lam=1.0, sigma=2.0)
        Oo, Lo = OA.biased_attention(q, k, v, slot, uv, idx, h, w, 1.0 / math.sqrt(128), 1.0, 2.0)
        err, lerr = np.abs(host(o) - Oo).max(), np.abs(host(lse) - Lo).max()
        print(f"{dtype} S={S} grid {h}x{w}: max|dO|={err:.3e} max|dLSE|={lerr:.3e}")
        assert err <= tol and lerr <= ltol


@pytest.mark.parametrize("dtype,key_parts", [("f32", 0), ("bf16", 0), ("bf16", 4)])
def test_attention_most_kv_frames(dtype, key_parts):
    """1024 KV frames, the most the slot table holds, on a 2 x 2 token grid:
    every 32-key tile then crosses eight frames, and the retrieved frames
    (24 of them, past the 16 staged in LDS) include the first and the last."""
    Lq, nf, H, h, w, S = 70, 1024, 2, 2, 2, 24
    rng = np.random.default_rng(1024)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    tol, ltol = (F32_TOL, LSE_F32_TOL) if dtype == "f32" else (BF16_TOL, LSE_BF16_TOL)
    q, k, v, _, uv, idx = _synthetic(rng, Lq, nf * h * w, H, 128, h, w, S, dtype)
    slot = np.full(nf, -1, np.int32)
    frames = np.concatenate([[0, nf - 1], rng.choice(np.arange(1, nf - 1), size=S - 2, replace=False)])
    slot[frames] = rng.permutation(S)
    o, lse = rv.biased_chunk_attention(dev(q, tdt), dev(k, tdt), dev(v, tdt), dev(slot), dev(uv), dev(idx), h=h, w=w,
                                       softmax_scale=1.0 / math.sqrt(128), lam=1.0, sigma=1.0, key_parts=key_parts)
    Oo, Lo = OA.biased_attention(q, k, v, slot, uv, idx, h, w, 1.0 / math.sqrt(128), 1.0, 1.0)
    O0, _ = OA.biased_attention(q, k, v, slot, None, None, h, w, 1.0 / math.sqrt(128), 0.0, 1.0)
    err, lerr = np.abs(host(o) - Oo).max(), np.abs(host(lse) - Lo).max()
    print(f"{dtype} {nf} frames, key_parts={key_parts}: max|dO|={err:.3e} max|dLSE|={lerr:.3e} "
          f"(bias moves O by {np.abs(Oo - O0).max():.2e})")
    assert err <= tol and lerr <= ltol
