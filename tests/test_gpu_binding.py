"""The Python binding rejects malformed device arguments before any launch:
caller-supplied outputs of the wrong shape or dtype, and a KV-frame slot
table whose length is not the number of KV frames (the kernels would read
or write past those buffers)."""

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
