"""Concurrent use of the library: two host threads, each with its own HIP
stream and its own workspace, run bf16 attention with the key split (its
partial results in the workspace) and a segmented retrieval (candidates in
the same workspace, after the attention on that stream) at the same time,
several rounds each. Every result must equal the one computed alone: the
library keeps no state that two streams could share."""

from __future__ import annotations

import math
import threading

import numpy as np
import pytest
import torch

import paper_2607_21848_amd as rv
from workloads.synth import ring_bank

pytestmark = pytest.mark.gpu


def _attention_case(seed, Lq=900, nf=8, h=10, w=12, H=3):
    g = torch.Generator(device="cuda:0")
    g.manual_seed(seed)
    Lk = nf * h * w
    q, k, v = (torch.randn((n, H, 128), generator=g, device="cuda:0").bfloat16() for n in (Lq, Lk, Lk))
    slot = torch.full((nf,), -1, dtype=torch.int32, device="cuda:0")
    slot[2:5] = torch.arange(3, dtype=torch.int32, device="cuda:0")
    uv = torch.rand((3, Lq, 2), generator=g, device="cuda:0") * torch.tensor([float(w), float(h)], device="cuda:0")
    idx = torch.randint(-2, h * w, (3, Lq), generator=g, device="cuda:0", dtype=torch.int32)
    return (q, k, v, slot, uv, idx), dict(h=h, w=w, softmax_scale=1 / math.sqrt(128), lam=1.0, sigma=2.0)


def _retrieval_case(seed, N=40000):
    rng = np.random.default_rng(seed)
    bank = torch.from_numpy(ring_bank(rng, N, radius=6.0)).cuda()
    q = torch.from_numpy(ring_bank(rng, 3, radius=6.0)).cuda()
    qc = torch.tensor([N + 5, N // 3, N - 1], dtype=torch.int32, device="cuda:0")
    return (bank, q, qc), dict(E=12.0, w_v=0.5, tau_c=0.1, tau_v=0.8, delta=3, first_candidate=1, k=16)


def test_two_threads_two_streams():
    cases = [(_attention_case(s), _retrieval_case(s)) for s in (1, 2)]
    # alone, on the default stream
    ref = []
    for (aa, akw), (ra, rkw) in cases:
        o, lse = rv.biased_chunk_attention(*aa, **akw, key_parts=4)
        ri, rs, rc, _ = rv.retrieve_chunks(*ra, **rkw)
        torch.cuda.synchronize()
        ref.append((o.clone(), lse.clone(), ri.clone(), rs.clone(), rc.clone()))
    errors = []

    def worker(t):
        try:
            (aa, akw), (ra, rkw) = cases[t]
            q, k = aa[0], aa[1]
            nbytes = max(rv.attention_workspace_size(q.dtype, q.shape[0], k.shape[0], q.shape[1], q.shape[2], 4),
                         rv.retrieve_workspace_size(ra[0].shape[0], ra[1].shape[0], rkw["k"]))
            assert nbytes > 0
            ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s):
                for _ in range(4):
                    o, lse = rv.biased_chunk_attention(*aa, **akw, key_parts=4, workspace=ws)
                    ri, rs, rc, _ = rv.retrieve_chunks(*ra, **rkw, workspace=ws)
                    s.synchronize()
                    got = (o, lse, ri, rs, rc)
                    for name, x, y in zip(("o", "lse", "idx", "score", "count"), got, ref[t]):
                        if not torch.equal(x, y):
                            errors.append(f"thread {t}: {name} differs from the result computed alone")
        except Exception as e:  # reported below
            errors.append(f"thread {t}: {e!r}")

    threads = [threading.Thread(target=worker, args=(t,)) for t in (0, 1)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    torch.cuda.synchronize()
    assert not errors, errors
