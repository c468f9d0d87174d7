"""The stage path (pose retrieval -> correspondence -> biased attention) at
the history-bank shape, captured in one HIP graph and replayed.

Nothing on the path synchronises with the host or allocates (the attention's
key-split workspace is the caller's), so the three calls capture as kernel
nodes with no eager warm-up on the capture stream. Every replay, with eager
work of the library's on the default stream between replays, must reproduce
the eager results bit for bit: retrieval ids, scores, counts and frame
selection, the correspondence map, and attention output and LSE. The
rotation-only correspondence call is captured and replayed the same way."""

from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2607_21848_amd as rv
import workloads as W

pytestmark = pytest.mark.gpu


def test_stage_path_replays_in_a_graph():
    dev = torch.device("cuda:0")
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    tb = lambda bits: torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)
    wl = W.make_c4("bf16")
    r = wl.retrieval
    qs = slice(1, 2)
    bank = (t(r.bank_frame_depth), t(r.bank_frame_c2w), t(r.bank_frame_K))
    bank_c2w, q_c2w, q_chunk = t(r.bank_c2w), t(r.query_c2w[qs]), t(r.query_chunk[qs])
    tgt = (t(r.query_frame_depth[qs]), t(r.query_frame_c2w[qs]), t(r.query_frame_K[qs]))
    q, k, v, slot = tb(wl.q), tb(wl.k), tb(wl.v), t(wl.slot)

    nbytes = rv.attention_workspace_size(torch.bfloat16, wl.Lq, wl.Lk, wl.H, wl.D)
    assert nbytes > 0  # the history-bank shape splits its keys

    def outputs():
        return dict(ridx=torch.empty((1, r.k), dtype=torch.int32, device=dev),
                    rscore=torch.empty((1, r.k), dtype=torch.float32, device=dev),
                    rcount=torch.empty((1,), dtype=torch.int32, device=dev),
                    rsel=torch.empty((1, r.k * 3), dtype=torch.int32, device=dev),
                    cuv=torch.empty((1, wl.S, wl.Lq, 2), dtype=torch.float32, device=dev),
                    cidx=torch.empty((1, wl.S, wl.Lq), dtype=torch.int32, device=dev),
                    o=torch.empty_like(q), lse=torch.empty((wl.H, wl.Lq), dtype=torch.float32, device=dev),
                    ws=torch.empty(nbytes, dtype=torch.uint8, device=dev))

    def step(b):
        rv.retrieve_chunks(bank_c2w, q_c2w, q_chunk, E=r.E, w_v=r.w_v, tau_c=r.tau_c, tau_v=r.tau_v, delta=r.delta,
                           first_candidate=r.first_candidate, k=r.k, frames_per_chunk=3,
                           out=(b["ridx"], b["rscore"], b["rcount"], b["rsel"]))
        rv.reproject_correspondence(*tgt, *bank, p=wl.p, eps=wl.eps, src_sel=b["rsel"], out=(b["cuv"], b["cidx"]))
        rv.biased_chunk_attention(q, k, v, slot, b["cuv"][0], b["cidx"][0], h=wl.h, w=wl.w,
                                  softmax_scale=wl.softmax_scale, lam=wl.lam, sigma=wl.sigma, out=(b["o"], b["lse"]),
                                  workspace=b["ws"])

    cap = torch.cuda.Stream(dev)
    ref, buf, other = outputs(), outputs(), outputs()
    torch.cuda.synchronize()
    # captured first: nothing of the library's has run on the capture stream before
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=cap):
        step(buf)
    step(ref)  # eager, on the default stream
    torch.cuda.synchronize()
    assert int(ref["rcount"].item()) == r.k
    for rep in range(3):
        for x in buf.values():
            x.zero_()
        step(other)  # eager work of the library's on the default stream between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for name in ref:
            if name != "ws":
                assert torch.equal(buf[name], ref[name]), f"replay {rep}: {name} differs from the eager result"
        assert torch.equal(other["o"], ref["o"])
    print(f"graph of the stage path replayed 3 times, bit-identical to eager; retrieval {ref['ridx'].tolist()}")


def test_rotation_only_correspondence_replays_in_a_graph():
    """reproject_rotation allocates nothing and synchronises with nothing, so
    it captures as one kernel node; every replay reproduces the eager map."""
    dev = torch.device("cuda:0")
    args = [torch.from_numpy(np.ascontiguousarray(a)).to(dev) for a in W.make_rotation_batch(64)]
    shape = dict(h=30, w=52, p=2)

    def outputs():
        return (torch.empty((64, 6, 4680, 2), dtype=torch.float32, device=dev),
                torch.empty((64, 6, 4680), dtype=torch.int32, device=dev))

    cap = torch.cuda.Stream(dev)
    ref, buf, other = outputs(), outputs(), outputs()
    cap.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(cap):
        rv.reproject_rotation(*args, **shape, out=ref)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=cap):
        rv.reproject_rotation(*args, **shape, out=buf)
    for rep in range(3):
        for x in buf:
            x.zero_()
        rv.reproject_rotation(*args, **shape, out=other)  # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(buf[1], ref[1]), f"replay {rep}: codes differ from the eager result"
        assert torch.equal(buf[0].view(torch.int32), ref[0].view(torch.int32)), f"replay {rep}: u^ differs"
    assert (ref[1] >= 0).float().mean().item() > 0.4
