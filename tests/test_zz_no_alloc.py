"""biased_chunk_attention_noalloc, the entry point for callers that cannot
allocate (its bf16 key split keeps partial results in the library's
per-device scratch array), against biased_chunk_attention with a workspace
on the same inputs. Three calls in a row, each on a smaller input than the
one before, so a call that read the previous call's partial results would
show: a shape whose automatic split needs more than the 128 MiB scratch
(cut to the parts that fit), the history-bank shape with 4 key parts, and a
small shape with the automatic split. Each must equal the workspace entry
point with the same number of parts bit for bit (the same kernels; the
parity bar for bf16 is 2e-2 on O and 4e-3 on LSE, and bit equality is
stricter). An explicit split that does not fit is refused before launch."""

from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import paper_2607_21848_amd as rv

pytestmark = pytest.mark.gpu

SCRATCH_BYTES = 128 << 20
PART_BYTES = (128 * 128 + 2 * 128) * 4  # one (item, part) of partial results


def _case(seed, Lq, nf, H, S, h=30, w=52):
    g = torch.Generator(device="cuda:0")
    g.manual_seed(seed)
    Lk = nf * h * w
    q, k, v = (torch.randn((n, H, 128), generator=g, device="cuda:0").bfloat16() for n in (Lq, Lk, Lk))
    slot = torch.full((nf,), -1, dtype=torch.int32, device="cuda:0")
    slot[1:1 + S] = torch.arange(S, dtype=torch.int32, device="cuda:0")
    uv = torch.rand((S, Lq, 2), generator=g, device="cuda:0") * torch.tensor([float(w), float(h)], device="cuda:0")
    idx = torch.randint(-2, h * w, (S, Lq), generator=g, device="cuda:0", dtype=torch.int32)
    return (q, k, v, slot, uv, idx), dict(h=h, w=w, softmax_scale=1 / math.sqrt(128), lam=1.0, sigma=2.0)


def _parts_that_fit(q, k, key_parts):
    """The key parts the no-allocation entry point uses for this call."""
    Lq, H, D = q.shape
    items = (Lq + 127) // 128 * H
    nbytes = rv.attention_workspace_size(torch.bfloat16, Lq, k.shape[0], H, D, key_parts)
    parts = max(1, nbytes // (items * PART_BYTES))
    while parts > 1 and items * parts * PART_BYTES > SCRATCH_BYTES:
        parts -= 1
    return parts


def test_noalloc_matches_the_workspace_entry_point():
    cases = [
        ("Lq 9360, Lk 37440, 24 heads, automatic split", _case(1, 9360, 24, 24, 12), 0),
        ("history-bank shape, 4 key parts", _case(2, 4680, 24, 12, 12), 4),
        ("Lq 1000, Lk 12480, 3 heads, automatic split", _case(3, 1000, 8, 3, 4), 0),
    ]
    used = []
    for label, (args, kw), key_parts in cases:
        q, k = args[0], args[1]
        parts = _parts_that_fit(q, k, key_parts)
        used.append(parts)
        print(f"noalloc: {label}: {parts} key parts", flush=True)
        o_na, lse_na = rv.biased_chunk_attention(*args, **kw, key_parts=key_parts, noalloc=True)
        o_ws, lse_ws = rv.biased_chunk_attention(*args, **kw, key_parts=parts)
        torch.cuda.synchronize()
        d_o = (o_na.float() - o_ws.float()).abs().max().item()
        d_l = (lse_na - lse_ws).abs().max().item()
        print(f"  max |dO| = {d_o:.3e}, max |dLSE| = {d_l:.3e}")
        assert torch.isfinite(o_na.float()).all()
        assert torch.equal(o_na, o_ws) and torch.equal(lse_na, lse_ws), label
    # the first case's automatic split (2 parts on 256 compute units) was cut to fit; the second kept its 4
    assert used[0] == 1 and used[1] == 4


def test_noalloc_refuses_a_split_beyond_its_scratch():
    (q, k, v, slot, uv, idx), kw = _case(4, 4680, 24, 12, 12)
    with pytest.raises(rv.RevisitError) as e:
        rv.biased_chunk_attention(q, k, v, slot, uv, idx, **kw, key_parts=64, noalloc=True)
    assert e.value.status == 2 and "scratch" in str(e.value)
