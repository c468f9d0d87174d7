"""The Python binding rejects malformed device arguments before any launch:
caller-supplied outputs of the wrong shape or dtype, a KV-frame slot table
whose length is not the number of KV frames, and malformed poses or
selections for the rotation-only call (the kernels would read or write past
those buffers)."""

from __future__ import annotations

import pytest
import torch

import paper_2607_21848_amd as rv

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _retrieval_inputs(N=12, Q=2):
    eye = torch.eye(4, dtype=torch.float32, device=DEV)
    bank = eye.repeat(N, 1, 1).contiguous()
    qp = eye.repeat(Q, 1, 1).contiguous()
    qc = torch.full((Q,), N + 3, dtype=torch.int32, device=DEV)
    kw = dict(E=10.0, w_v=0.5, tau_c=0.2, tau_v=0.785, delta=3, first_candidate=1, k=4)
    return bank, qp, qc, kw


def _outs(Q, k, F=None, idx_shape=None, score_dtype=torch.float32):
    idx = torch.empty(idx_shape or (Q, k), dtype=torch.int32, device=DEV)
    score = torch.empty((Q, k), dtype=score_dtype, device=DEV)
    count = torch.empty((Q,), dtype=torch.int32, device=DEV)
    sel = torch.empty((Q, k * F), dtype=torch.int32, device=DEV) if F else None
    return idx, score, count, sel


def test_retrieval_rejects_malformed_outputs():
    bank, qp, qc, kw = _retrieval_inputs()
    with pytest.raises(ValueError):
        rv.retrieve_chunks(bank, qp, qc, **kw, out=_outs(2, 4, idx_shape=(2, 3)))
    with pytest.raises(TypeError):
        rv.retrieve_chunks(bank, qp, qc, **kw, out=_outs(2, 4, score_dtype=torch.float64))
    with pytest.raises(ValueError):  # a frame selection buffer without frames_per_chunk
        rv.retrieve_chunks(bank, qp, qc, **kw, out=_outs(2, 4, F=3))
    with pytest.raises(ValueError):  # frames_per_chunk without a frame selection buffer
        rv.retrieve_chunks(bank, qp, qc, **kw, frames_per_chunk=3, out=_outs(2, 4))
    # well-formed outputs are accepted and filled
    idx, score, count, sel = rv.retrieve_chunks(bank, qp, qc, **kw, frames_per_chunk=3, out=_outs(2, 4, F=3))
    torch.cuda.synchronize()
    assert count.tolist() == [4, 4] and sel.shape == (2, 12)


def test_attention_rejects_slot_table_of_wrong_length():
    Lq, Lk, H, D, h, w = 8, 40, 1, 128, 4, 5
    q = torch.zeros((Lq, H, D), dtype=torch.bfloat16, device=DEV)
    k = torch.zeros((Lk, H, D), dtype=torch.bfloat16, device=DEV)
    kw = dict(h=h, w=w, softmax_scale=0.1, lam=1.0, sigma=2.0)
    for n in (1, 3):  # Lk / (h w) = 2 frames
        with pytest.raises(ValueError):
            rv.biased_chunk_attention(q, k, k, torch.full((n,), -1, dtype=torch.int32, device=DEV), None, None, **kw)
    with pytest.raises(ValueError):  # Lk not a whole number of frames
        rv.biased_chunk_attention(q, k[:30], k[:30], torch.full((2,), -1, dtype=torch.int32, device=DEV), None, None,
                                  **kw)


def test_rotation_binding_checks_and_unbatched_form():
    """reproject_rotation: malformed poses, intrinsics, selections or outputs
    raise before any launch; unbatched inputs give unbatched outputs equal to
    the batched call's first problem."""
    eye = torch.eye(4, dtype=torch.float32, device=DEV)
    tc = eye.repeat(2, 3, 1, 1).contiguous()  # [B=2, Tq=3, 4, 4]
    tk = torch.tensor([20.0, 20.0, 13.0, 9.0], device=DEV).repeat(2, 3, 1).contiguous()
    sc, sk = tc[:, :2].contiguous(), tk[:, :2].contiguous()  # S = 2
    kw = dict(h=9, w=13, p=2)
    with pytest.raises(TypeError):
        rv.reproject_rotation(tc.double(), tk, sc, sk, **kw)
    with pytest.raises(ValueError):
        rv.reproject_rotation(tc, tk[:, :2].contiguous(), sc, sk, **kw)
    with pytest.raises(ValueError):  # non-contiguous poses
        rv.reproject_rotation(tc.transpose(2, 3), tk, sc, sk, **kw)
    with pytest.raises(ValueError):  # a frame bank with a selection of the wrong batch
        rv.reproject_rotation(tc, tk, sc.reshape(4, 4, 4), sk.reshape(4, 4), **kw,
                              src_sel=torch.zeros((3, 2), dtype=torch.int32, device=DEV))
    with pytest.raises(ValueError):
        rv.reproject_rotation(tc, tk, sc, sk, **kw, out=(torch.empty((2, 2, 351, 2), device=DEV),
                                                        torch.empty((2, 2, 350), dtype=torch.int32, device=DEV)))
    with pytest.raises(TypeError):
        rv.reproject_rotation(tc, tk, sc, sk, **kw, out=(torch.empty((2, 2, 351, 2), device=DEV),
                                                        torch.empty((2, 2, 351), device=DEV)))
    uv, idx = rv.reproject_rotation(tc, tk, sc, sk, **kw)
    uv1, idx1 = rv.reproject_rotation(tc[0], tk[0], sc[0], sk[0], **kw)
    torch.cuda.synchronize()
    assert idx1.shape == (2, 351) and torch.equal(idx1, idx[0])
    assert torch.equal(uv1.view(torch.int32), uv[0].view(torch.int32))
    # identity poses: every token of each of the 3 frames maps onto itself
    assert torch.equal(idx[1, 0], torch.arange(117, dtype=torch.int32, device=DEV).repeat(3))


def test_rotation_offset_output_views():
    """reproject_rotation stores a token pair's u^ as one 16-byte store and its
    codes as one 8-byte store only where those addresses are so aligned.
    Outputs that start one element into larger buffers (u^ 8-byte but not
    16-byte aligned, codes 4-byte but not 8-byte aligned) take single stores
    and give the same bits as aligned outputs."""
    import numpy as np
    import workloads as W
    tc, tk, sc, sk = (torch.from_numpy(np.ascontiguousarray(a)).to(DEV) for a in W.make_rotation_batch(3, seed=5))
    kw = dict(h=30, w=52, p=2)
    B, S, Lq = 3, 6, 3 * 30 * 52
    print("reproject_rotation: offset output views", flush=True)
    uv, idx = rv.reproject_rotation(tc, tk, sc, sk, **kw)
    uv_buf = torch.full((B * S * Lq * 2 + 2,), 7.0, device=DEV)
    idx_buf = torch.full((B * S * Lq + 1,), 7, dtype=torch.int32, device=DEV)
    ouv, oidx = uv_buf[2:].view(B, S, Lq, 2), idx_buf[1:].view(B, S, Lq)
    assert ouv.data_ptr() % 16 == 8 and oidx.data_ptr() % 8 == 4
    rv.reproject_rotation(tc, tk, sc, sk, **kw, out=(ouv, oidx))
    torch.cuda.synchronize()
    assert torch.equal(oidx, idx)
    assert torch.equal(ouv.view(torch.int32), uv.view(torch.int32))
    assert uv_buf[:2].eq(7.0).all() and idx_buf[:1].eq(7).all()  # nothing written before the views
