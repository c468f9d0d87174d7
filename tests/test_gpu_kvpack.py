"""GPU parity of cache packing (Sec. 4.2, cache packing) against the fp64 oracle.

Bar (written here): values and every key element outside the temporal band
are copied bit for bit; rotated key elements are bit-exact in bf16 and
within 1 ulp in fp32. Both sides evaluate the rotation in double precision
in the same order and round once; they differ only through the last bit of
cos, sin and pow of the two math libraries, which can move an fp32 result
across a rounding boundary (about 1 element in 10^9) but practically never
a bf16 one. The exception is a position shift of about 10^9 frames, where
a 1-ulp difference in omega_i moves the angle by up to |delta| omega_i 2^-52
(~4e-7 rad): there the bar is 1 ulp plus |delta| omega_i 2^-51 times the
pair's norm. Slots whose selection is empty or out of range, and rows
outside the slots, must keep their previous contents bit for bit.
"""

from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2607_21848_amd as rv
import workloads as W
from oracle import kvpack as OK
from tests.gpu_helpers import dev, host
from workloads.synth import bf16_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rv.lib()
    yield
    torch.cuda.synchronize()


def _to_dev(a: np.ndarray) -> torch.Tensor:
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _to_host(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def _ordered(a: np.ndarray) -> np.ndarray:
    """Integers ordered like the floats they encode (bf16 or fp32 bit patterns)."""
    if a.dtype == np.uint16:
        i = a.astype(np.int64)
        return np.where(i & 0x8000, 0x8000 - i, i)
    i = a.view(np.uint32).astype(np.int64)
    return np.where(i & 0x80000000, 0x80000000 - i, i)


def _check(got: np.ndarray, want: np.ndarray, n_t: int, exact: bool):
    """got/want: [..., D] cache arrays (uint16 bits or float32)."""
    gb = got.view(np.uint16) if got.dtype == np.uint16 else got.view(np.uint32)
    wb = want.view(np.uint16) if want.dtype == np.uint16 else want.view(np.uint32)
    # outside the temporal band: bit for bit
    assert np.array_equal(gb[..., 2 * n_t:], wb[..., 2 * n_t:])
    if n_t == 0:
        return 0
    g, w = got[..., :2 * n_t], want[..., :2 * n_t]
    d = np.abs(_ordered(np.ascontiguousarray(g)) - _ordered(np.ascontiguousarray(w)))
    n_diff = int(np.count_nonzero(d))
    assert int(d.max(initial=0)) <= 1, f"max ulp distance {int(d.max())}"
    if exact:
        assert n_diff == 0, f"{n_diff} rotated elements differ by 1 ulp"
    return n_diff


def _random_case(rng, dtype, L, n_store, F, h, w, H, D, rows):
    T = F * h * w
    k = rng.standard_normal((L, n_store, T, H, D)).astype(np.float32)
    v = rng.standard_normal((L, n_store, T, H, D)).astype(np.float32)
    if dtype == "bf16":
        sk, sv = bf16_bits(k), bf16_bits(v)
        ck = np.full((L, rows, H, D), 0x7FA1, np.uint16)  # NaN sentinels: any unwanted write shows
        cv = np.full((L, rows, H, D), 0xFFA2, np.uint16)
    else:
        sk, sv = k, v
        ck = np.full((L, rows, H, D), np.float32(-3.5))
        cv = np.full((L, rows, H, D), np.float32(7.25))
    return sk, sv, ck, cv


def _run(sk, sv, pos, sel, dst_pos, ck, cv, row0, F, h, w, n_t, theta):
    gk, gv = _to_dev(ck), _to_dev(cv)
    rv.pack_retrieved_kv(_to_dev(sk), _to_dev(sv), dev(np.asarray(sel, np.int32)), gk, gv, F=F, h=h, w=w,
                         dst_pos=dst_pos, dst_row0=row0, rope_t_pairs=n_t, rope_theta=theta,
                         store_pos=None if pos is None else dev(np.asarray(pos, np.int32)))
    torch.cuda.synchronize()
    return _to_host(gk), _to_host(gv)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("D,n_t", [(128, 22), (64, 11), (8, 4), (128, 64), (128, 0), (24, 5)])
def test_pack_small(dtype, D, n_t):
    rng = np.random.default_rng(D * 100 + n_t)
    L, n_store, F, h, w, H = 2, 6, 2, 3, 5, 3
    T = F * h * w
    sel = [4, -1, 0, 4, 6, 2]  # repeat, empty, out of range
    rows = 3 + len(sel) * T + 5
    sk, sv, ck, cv = _random_case(rng, dtype, L, n_store, F, h, w, H, D, rows)
    pos = rng.integers(-40, 400, n_store)
    args = (sk, sv, pos, sel, 17, ck, cv, 3, F, h, w, n_t, 10000.0)
    gk, gv = _run(*args)
    wk, wv = OK.pack_retrieved_kv(sk, sv, pos, sel, 17, ck, cv, 3, F, n_t, 10000.0)
    assert gv.tobytes() == wv.tobytes()
    _check(gk, wk, n_t, exact=dtype == "bf16")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_pack_ragged_blocks_and_default_positions(dtype):
    # chunk images of 7*11*2*H*D elements: not a multiple of one block's 16 KiB
    rng = np.random.default_rng(21)
    L, n_store, F, h, w, H, D, n_t = 3, 9, 2, 7, 11, 5, 72, 13
    T = F * h * w
    sel = [8, 3, 0]
    rows = len(sel) * T + 1
    sk, sv, ck, cv = _random_case(rng, dtype, L, n_store, F, h, w, H, D, rows)
    gk, gv = _run(sk, sv, None, sel, 6, ck, cv, 1, F, h, w, n_t, 500.0)
    wk, wv = OK.pack_retrieved_kv(sk, sv, None, sel, 6, ck, cv, 1, F, n_t, 500.0)
    assert gv.tobytes() == wv.tobytes()
    _check(gk, wk, n_t, exact=dtype == "bf16")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_pack_position_edges(dtype):
    rng = np.random.default_rng(5)
    L, n_store, F, h, w, H, D, n_t = 1, 4, 3, 2, 4, 2, 128, 22
    T = F * h * w
    sk, sv, ck, cv = _random_case(rng, dtype, L, n_store, F, h, w, H, D, 4 * T)
    # delta = 0 for every slot: the keys come back unchanged
    pos = np.array([0, 3, 6, 9])
    gk, _ = _run(sk, sv, pos, [0, 1, 2, 3], 0, ck, cv, 0, F, h, w, n_t, 10000.0)
    assert gk.reshape(-1).tobytes() == sk[:, [0, 1, 2, 3]].reshape(-1).tobytes()
    # negative and very large shifts
    sel = [3, 0, 2, 1]
    p = np.array([7000, -3, 12, 99999])
    gk, gv = _run(sk, sv, p, sel, -5000, ck, cv, 0, F, h, w, n_t, 10000.0)
    wk, wv = OK.pack_retrieved_kv(sk, sv, p, sel, -5000, ck, cv, 0, F, n_t, 10000.0)
    assert gv.tobytes() == wv.tobytes()
    _check(gk, wk, n_t, exact=dtype == "bf16")
    # shifts of ~2e9 frames: the angle bound of the module docstring
    dst, p = 2_000_000_000, np.array([-100_000_000, 5, 0, 1])
    gk, gv = _run(sk, sv, p, sel, dst, ck, cv, 0, F, h, w, n_t, 10000.0)
    wk, wv = OK.pack_retrieved_kv(sk, sv, p, sel, dst, ck, cv, 0, F, n_t, 10000.0)
    assert gv.tobytes() == wv.tobytes()
    as64 = (lambda a: OK.bf16_to_f64(a)) if dtype == "bf16" else (lambda a: a.astype(np.float64))
    g, wv64 = as64(gk)[..., :2 * n_t], as64(wk)[..., :2 * n_t]
    omega = OK.rope_frequencies(n_t, 10000.0)
    slack = np.zeros_like(g)
    for s_, j in enumerate(sel):
        src = as64(sk[:, j])[..., :2 * n_t]
        norm = np.hypot(src[..., 0::2], src[..., 1::2])
        bound = abs(dst + s_ * F - int(p[j])) * omega * 2.0**-51 * norm
        slack[:, s_ * T:(s_ + 1) * T, :, 0::2] = bound
        slack[:, s_ * T:(s_ + 1) * T, :, 1::2] = bound
    ulp = (np.spacing(np.abs(wv64).astype(np.float32)).astype(np.float64) * 2**16 if dtype == "bf16"
           else np.spacing(np.abs(wv64).astype(np.float32)).astype(np.float64))
    assert np.all(np.abs(g - wv64) <= ulp + slack)
    assert np.array_equal((gk.view(np.uint16) if dtype == "bf16" else gk.view(np.uint32))[..., 2 * n_t:],
                          (wk.view(np.uint16) if dtype == "bf16" else wk.view(np.uint32))[..., 2 * n_t:])


def test_pack_empty_selections_leave_cache_alone():
    rng = np.random.default_rng(8)
    L, n_store, F, h, w, H, D = 2, 3, 1, 4, 4, 2, 64
    T = F * h * w
    sk, sv, ck, cv = _random_case(rng, "bf16", L, n_store, F, h, w, H, D, 3 * T)
    gk, gv = _run(sk, sv, None, [-1, 3, -7], 0, ck, cv, 0, F, h, w, 8, 10000.0)
    assert gk.tobytes() == ck.tobytes() and gv.tobytes() == cv.tobytes()
    gk, gv = _run(sk[:, :0], sv[:, :0], None, [0, 1], 0, ck, cv, T, F, h, w, 8, 10000.0)  # n_store = 0
    assert gk.tobytes() == ck.tobytes() and gv.tobytes() == cv.tobytes()


def test_pack_history_bank_retrieval_on_device():
    """The Wan-1.3B history-bank chunk: the retrieval's out_idx drives the gather
    of 4 chunks (3 frames of 30 x 52 tokens, 12 heads, D 128, bf16) from a
    200-chunk store, one layer, into the slots after the anchor chunk; the
    retrieved slots end where the recent window begins."""
    wl = W.make_config(4, "bf16", qkv=False)
    r = wl.retrieval
    idx, _, cnt, _ = rv.retrieve_chunks(dev(r.bank_c2w), dev(r.query_c2w), dev(r.query_chunk), E=r.E, w_v=r.w_v,
                                        tau_c=r.tau_c, tau_v=r.tau_v, delta=r.delta,
                                        first_candidate=r.first_candidate, k=r.k)
    q = 1  # query chunk 225, a full top-4 retrieval
    sel_dev = idx[q].contiguous()
    sel = host(sel_dev)
    assert int(host(cnt)[q]) == 4
    F, h, w, H, D, n_t, theta = 3, 30, 52, 12, 128, 22, 10000.0
    T = F * h * w
    n_store = int(r.bank_c2w.shape[0])
    rng = np.random.default_rng(1004)
    store_k = torch.zeros((1, n_store, T, H, D), dtype=torch.bfloat16, device="cuda")
    store_v = torch.zeros_like(store_k)
    host_k, host_v = {}, {}
    for j in sel.tolist():
        host_k[j] = bf16_bits(rng.standard_normal((T, H, D)).astype(np.float32))
        host_v[j] = bf16_bits(rng.standard_normal((T, H, D)).astype(np.float32))
        store_k[0, j] = _to_dev(host_k[j])
        store_v[0, j] = _to_dev(host_v[j])
    rows = 8 * T  # anchor | 4 retrieved | recent (3 chunks)
    cache_k = torch.full((1, rows, H, D), 1.0, dtype=torch.bfloat16, device="cuda")
    cache_v = torch.full_like(cache_k, 2.0)
    q_chunk = int(r.query_chunk[q])
    rv.pack_retrieved_kv(store_k, store_v, sel_dev, cache_k, cache_v, F=F, h=h, w=w, dst_pos=F, dst_row0=T,
                         rope_t_pairs=n_t, rope_theta=theta)
    torch.cuda.synchronize()
    gk, gv = _to_host(cache_k), _to_host(cache_v)
    # oracle over the four selected chunks only (the store is zero elsewhere)
    mini_k = np.stack([host_k[j] for j in sel.tolist()])[None]
    mini_v = np.stack([host_v[j] for j in sel.tolist()])[None]
    ck0 = np.full((1, rows, H, D), 0x3F80, np.uint16)
    cv0 = np.full((1, rows, H, D), 0x4000, np.uint16)
    wk, wv = OK.pack_retrieved_kv(mini_k, mini_v, F * sel, [0, 1, 2, 3], F, ck0, cv0, T, F, n_t, theta)
    assert gv.tobytes() == wv.tobytes()
    _check(gk, wk, n_t, exact=True)
    assert q_chunk > int(sel.max())  # every retrieved chunk is older than the query chunk
