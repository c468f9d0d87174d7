"""The C interface without a GPU: the library loads, exports every function
include/revisit.h declares, and rejects bad arguments with the documented
status before touching the device."""

import ctypes
import math
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "revisit.h")


@pytest.fixture(scope="module")
def L():
    from paper_2607_21848_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        pytest.fail("librevisit.so is not built: run `python -m paper_2607_21848_amd.build`")
    return _lib.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_three_stages():
    names = declared_functions()
    for n in ("retrieve_chunks", "reproject_correspondence", "reproject_rotation", "biased_chunk_attention",
              "pack_retrieved_kv",
              "rc_status_string", "rc_last_error", "rc_retrieve_workspace_size", "rc_attention_workspace_size"):
        assert n in names


def test_every_declared_symbol_is_exported(L):
    for name in declared_functions():
        assert hasattr(L, name), name


def test_binding_matches_exports(L):
    from paper_2607_21848_amd import _lib
    assert set(_lib.EXPORTED) == set(declared_functions())


def test_status_strings(L):
    from paper_2607_21848_amd import _lib
    assert _lib.status_string(0) == "ok"
    assert _lib.status_string(4) == "bad parameter"
    assert _lib.status_string(99) == "unknown status"


NULL = None
FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first


def _retrieve(L, **kw):
    a = dict(bank=FAKE, n_bank=10, query=FAKE, qchunk=FAKE, n_query=1, E=1.0, w_v=0.5, tau_c=0.1, tau_v=0.5,
             delta=3, first=1, k=4, idx=FAKE, score=NULL, count=FAKE, F=0, sel=NULL, ws=NULL, ws_bytes=0)
    a.update(kw)
    return L.retrieve_chunks(a["bank"], a["n_bank"], a["query"], a["qchunk"], a["n_query"], a["E"], a["w_v"],
                             a["tau_c"], a["tau_v"], a["delta"], a["first"], a["k"], a["idx"], a["score"],
                             a["count"], a["F"], a["sel"], a["ws"], a["ws_bytes"], NULL)


@pytest.mark.parametrize("kw,status", [
    (dict(k=0), 4), (dict(k=33), 4), (dict(E=0.0), 4), (dict(E=float("nan")), 4), (dict(tau_c=float("inf")), 4),
    (dict(n_bank=-1), 2), (dict(n_bank=(1 << 30) + 1), 2), (dict(n_query=-2), 2), (dict(query=NULL), 1),
    (dict(count=NULL), 1), (dict(bank=ctypes.c_void_p(0x1004)), 2),
    (dict(sel=FAKE, F=0), 4),
    # a bank above 8192 entries needs a workspace: none, too small, NULL, misaligned
    (dict(n_bank=20000), 2), (dict(n_bank=20000, ws=FAKE, ws_bytes=95), 2), (dict(n_bank=20000, ws_bytes=96), 1),
    (dict(n_bank=20000, ws=ctypes.c_void_p(0x1008), ws_bytes=96), 2),
])
def test_retrieve_rejects(L, kw, status):
    from paper_2607_21848_amd import _lib
    assert _retrieve(L, **kw) == status
    assert len(_lib.last_error()) > 0


def test_retrieve_empty_query_is_ok(L):
    assert _retrieve(L, n_query=0, query=NULL, qchunk=NULL, idx=NULL, count=NULL) == 0


def _reproject(L, **kw):
    a = dict(td=FAKE, tc=FAKE, tk=FAKE, sd=FAKE, sc=FAKE, sk=FAKE, sel=NULL, n_src=0, B=1, Tq=3, S=6, h=30, w=52,
             p=2, eps=0.05, uv=FAKE, idx=FAKE)
    a.update(kw)
    return L.reproject_correspondence(a["td"], a["tc"], a["tk"], a["sd"], a["sc"], a["sk"], a["sel"], a["n_src"],
                                      a["B"], a["Tq"], a["S"], a["h"], a["w"], a["p"], a["eps"], a["uv"], a["idx"],
                                      NULL)


@pytest.mark.parametrize("kw,status", [
    (dict(h=0), 2), (dict(p=0), 2), (dict(B=-1), 2), (dict(eps=-0.1), 4), (dict(eps=float("nan")), 4),
    (dict(td=NULL), 1), (dict(uv=NULL), 1), (dict(sd=NULL), 1), (dict(sel=FAKE, n_src=-1), 2),
    (dict(h=1 << 20, w=1 << 20), 2), (dict(S=65), 2),
])
def test_reproject_rejects(L, kw, status):
    assert _reproject(L, **kw) == status


def test_reproject_empty_is_ok(L):
    assert _reproject(L, S=0, td=NULL, uv=NULL) == 0
    assert _reproject(L, B=0, td=NULL, uv=NULL) == 0


def _rotation(L, **kw):
    a = dict(tc=FAKE, tk=FAKE, sc=FAKE, sk=FAKE, sel=NULL, n_src=0, B=1, Tq=3, S=6, h=30, w=52, p=2, uv=FAKE,
             idx=FAKE)
    a.update(kw)
    return L.reproject_rotation(a["tc"], a["tk"], a["sc"], a["sk"], a["sel"], a["n_src"], a["B"], a["Tq"], a["S"],
                                a["h"], a["w"], a["p"], a["uv"], a["idx"], NULL)


@pytest.mark.parametrize("kw,status", [
    (dict(h=0), 2), (dict(w=-3), 2), (dict(p=0), 2), (dict(B=-1), 2), (dict(Tq=-1), 2), (dict(S=65), 2),
    (dict(tc=NULL), 1), (dict(tk=NULL), 1), (dict(uv=NULL), 1), (dict(idx=NULL), 1), (dict(sc=NULL), 1),
    (dict(sel=FAKE, n_src=-1), 2), (dict(h=1 << 15, w=1 << 14), 2), (dict(B=1 << 20, h=64, w=64), 2),
    (dict(uv=ctypes.c_void_p(0x1004)), 2),
])
def test_rotation_rejects(L, kw, status):
    from paper_2607_21848_amd import _lib
    assert _rotation(L, **kw) == status
    assert "reproject_rotation" in _lib.last_error()


def test_rotation_empty_is_ok(L):
    assert _rotation(L, S=0, tc=NULL, uv=NULL) == 0
    assert _rotation(L, B=0, tc=NULL, uv=NULL) == 0
    # a bank with no frames needs no source pointers (every slot is empty)
    assert _rotation(L, B=0, sel=FAKE, n_src=0, sc=NULL, sk=NULL) == 0


def _attention(L, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, o=FAKE, lse=NULL, dtype=1, Lq=4680, Lk=28080, H=12, D=128, h=30, w=52,
             slot=FAKE, uv=FAKE, idx=FAKE, S=6, scale=1 / math.sqrt(128), lam=1.0, sigma=2.0, parts=3, ws=NULL,
             ws_bytes=0)
    a.update(kw)
    return L.biased_chunk_attention(a["q"], a["k"], a["v"], a["o"], a["lse"], a["dtype"], a["Lq"], a["Lk"], a["H"],
                                    a["D"], a["h"], a["w"], a["slot"], a["uv"], a["idx"], a["S"], a["scale"],
                                    a["lam"], a["sigma"], a["parts"], a["ws"], a["ws_bytes"], NULL)


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=7), 3), (dict(D=64), 3), (dict(dtype=2, D=96), 3), (dict(Lk=28081), 2), (dict(Lk=0), 2),
    (dict(H=0), 2), (dict(Lq=-1), 2), (dict(sigma=0.0), 4), (dict(scale=-1.0), 4), (dict(lam=float("inf")), 4),
    (dict(sigma=1e-30), 4), (dict(q=NULL), 1), (dict(o=NULL), 1), (dict(uv=NULL), 1), (dict(slot=NULL), 1),
    (dict(Lk=1025 * 1560), 2), (dict(h=300, w=4, Lk=1200 * 8), 2), (dict(dtype=3, h=4, w=257, Lk=1028 * 8), 2),
    (dict(parts=-1), 4), (dict(parts=65), 4),
    # 3 key parts of 444 items need 444 * 3 * 66560 bytes: none, one byte short, NULL, misaligned
    (dict(), 2), (dict(ws=FAKE, ws_bytes=444 * 3 * 66560 - 1), 2), (dict(ws_bytes=444 * 3 * 66560), 1),
    (dict(ws=ctypes.c_void_p(0x1004), ws_bytes=444 * 3 * 66560), 2),
])
def test_attention_rejects(L, kw, status):
    assert _attention(L, **kw) == status


def test_attention_bias_pointers_optional_when_off(L):
    # S = 0 or lambda = 0 with NULL map pointers passes validation; Lq = 0 then returns before any launch
    assert _attention(L, Lq=0, S=0, uv=NULL, idx=NULL, slot=NULL) == 0
    assert _attention(L, Lq=0, lam=0.0, uv=NULL, idx=NULL, slot=NULL) == 0


def _ws_size(L, fn, *args):
    n = ctypes.c_size_t(12345)
    st = getattr(L, fn)(*args, ctypes.byref(n))
    return st, n.value


@pytest.mark.parametrize("args,status,nbytes", [
    ((1, 4680, 37440, 12, 128, 4), 0, 444 * 4 * 66560), ((1, 4680, 37440, 12, 128, 1), 0, 0),
    ((3, 4680, 37440, 12, 128, 2), 0, 444 * 2 * 66560), ((2, 4680, 37440, 12, 128, 8), 0, 0),
    ((1, 0, 37440, 12, 128, 8), 0, 0), ((1, 4680, 64, 12, 128, 8), 0, 444 * 2 * 66560),
    ((1, 4680, 37440, 12, 128, -1), 4, 0), ((1, 4680, 37440, 12, 128, 65), 4, 0), ((1, 4680, 37440, 12, 64, 4), 3, 0),
    ((9, 4680, 37440, 12, 128, 4), 3, 0), ((1, -1, 37440, 12, 128, 4), 2, 0), ((1, 4680, 0, 12, 128, 4), 2, 0),
])
def test_attention_workspace_size(L, args, status, nbytes):
    """Fixed key parts need no device: items * parts * (128 x 128 + 2 x 128) floats,
    nothing for one part or fp32, parts clamped to the number of 32-key tiles."""
    assert _ws_size(L, "rc_attention_workspace_size", *args) == (status, nbytes)


@pytest.mark.parametrize("args,status,nbytes", [
    ((8192, 5, 4), 0, 0), ((8193, 5, 4), 0, 5 * 1 * 4 * 12), ((1 << 23, 1, 32), 0, 512 * 32 * 12),
    ((0, 1, 1), 0, 0), ((-1, 1, 1), 2, 0), ((10, 1, 0), 4, 0), ((10, 1, 33), 4, 0), ((1 << 30, 1 << 20, 32), 2, 0),
])
def test_retrieve_workspace_size(L, args, status, nbytes):
    assert _ws_size(L, "rc_retrieve_workspace_size", *args) == (status, nbytes)


def test_workspace_size_null_out(L):
    assert L.rc_attention_workspace_size(1, 10, 10, 1, 128, 1, None) == 1
    assert L.rc_retrieve_workspace_size(10, 1, 1, None) == 1


def _pack(L, **kw):
    a = dict(sk=FAKE, sv=FAKE, pos=NULL, n_store=200, sel=FAKE, n_sel=4, dst_pos=3, ck=FAKE, cv=FAKE, row0=4680,
             rows=37440, layers=30, dtype=1, F=3, h=30, w=52, H=12, D=128, nt=22, theta=10000.0)
    a.update(kw)
    return L.pack_retrieved_kv(a["sk"], a["sv"], a["pos"], a["n_store"], a["sel"], a["n_sel"], a["dst_pos"], a["ck"],
                               a["cv"], a["row0"], a["rows"], a["layers"], a["dtype"], a["F"], a["h"], a["w"], a["H"],
                               a["D"], a["nt"], a["theta"], NULL)


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=3), 3), (dict(D=60), 3), (dict(D=0), 3), (dict(D=520), 3),
    (dict(F=0), 2), (dict(H=0), 2), (dict(n_store=-1), 2), (dict(n_sel=-1), 2), (dict(layers=-1), 2), (dict(row0=-1), 2),
    (dict(row0=18721), 2), (dict(n_sel=8), 2), (dict(rows=1 << 30, layers=1 << 14), 2),
    (dict(nt=-1), 4), (dict(nt=65), 4), (dict(theta=0.0), 4), (dict(theta=float("nan")), 4),
    (dict(sk=NULL), 1), (dict(cv=NULL), 1), (dict(sel=NULL), 1),
    (dict(ck=ctypes.c_void_p(0x1008)), 2), (dict(pos=ctypes.c_void_p(0x1002)), 2),
])
def test_pack_rejects(L, kw, status):
    from paper_2607_21848_amd import _lib
    assert _pack(L, **kw) == status
    assert len(_lib.last_error()) > 0


def test_pack_nothing_to_do_is_ok(L):
    assert _pack(L, n_sel=0, sel=NULL, ck=NULL, cv=NULL) == 0
    assert _pack(L, layers=0, sel=NULL) == 0
    # rope_theta is not looked at without temporal pairs
    assert _pack(L, n_sel=0, nt=0, theta=0.0) == 0


def _stream_cfg(**kw):
    from paper_2607_21848_amd import _lib
    a = dict(F=3, h=30, w=52, p=2, H=12, D=128, layers=30, dtype=1, capacity=16, max_chunks=100, E=40.0, w_v=0.5,
             tau_c=0.05, tau_v=0.785, delta=3, eps=0.05, lam=1.0, sigma=2.0, softmax_scale=0.088, rope_t_pairs=22,
             rope_theta=10000.0)
    a.update(kw)
    return _lib.StreamConfig(**a)


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=5), 3), (dict(D=64), 3), (dict(dtype=2, D=96), 3), (dict(F=0), 2), (dict(F=65), 2), (dict(h=0), 2),
    (dict(layers=0), 2), (dict(capacity=4), 2), (dict(max_chunks=0), 2), (dict(E=0.0), 4),
    (dict(sigma=float("nan")), 4), (dict(eps=-1.0), 4), (dict(softmax_scale=0.0), 4), (dict(rope_t_pairs=65), 4),
    (dict(rope_theta=-1.0), 4), (dict(w=257), 2), (dict(H=65536), 2), (dict(layers=70000), 2),
    (dict(capacity=1 << 20, F=64, h=256, w=256), 2), (dict(layers=65536, H=65535), 2),
])
def test_stream_create_rejects(L, kw, status):
    h = ctypes.c_void_p(0x1234)
    assert L.rc_stream_create(ctypes.byref(_stream_cfg(**kw)), ctypes.byref(h)) == status
    assert not h.value  # *out cleared on failure


def test_stream_null_arguments(L):
    h = ctypes.c_void_p(0)
    assert L.rc_stream_create(None, ctypes.byref(h)) == 1
    assert L.rc_stream_step(None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, NULL, NULL) == 1
    assert L.rc_stream_view(None, None) == 1
    assert L.rc_stream_destroy(None) == 0


@pytest.mark.parametrize("args,status", [
    ((FAKE, -1, 30, 52, 2, FAKE), 2), ((FAKE, 3, 0, 52, 2, FAKE), 2), ((FAKE, 3, 30, 52, 0, FAKE), 2),
    ((NULL, 3, 30, 52, 2, FAKE), 1), ((FAKE, 3, 30, 52, 2, NULL), 1), ((ctypes.c_void_p(0x1002), 3, 30, 52, 2, FAKE), 2),
    ((NULL, 0, 30, 52, 2, NULL), 0),
])
def test_pool_token_depth_rejects(L, args, status):
    assert L.pool_token_depth(*args, NULL) == status


def _attention_noalloc(L, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, o=FAKE, lse=NULL, dtype=1, Lq=4680, Lk=37440, H=12, D=128, h=30, w=52,
             slot=FAKE, uv=FAKE, idx=FAKE, S=12, scale=1 / math.sqrt(128), lam=1.0, sigma=2.0, parts=64)
    a.update(kw)
    return L.biased_chunk_attention_noalloc(a["q"], a["k"], a["v"], a["o"], a["lse"], a["dtype"], a["Lq"], a["Lk"],
                                            a["H"], a["D"], a["h"], a["w"], a["slot"], a["uv"], a["idx"], a["S"],
                                            a["scale"], a["lam"], a["sigma"], a["parts"], NULL)


@pytest.mark.parametrize("kw,status", [
    # 444 items x 64 parts x 66560 bytes of partial results: more than the 128 MiB scratch
    (dict(), 2), (dict(parts=3, Lq=9360, H=24), 2),
    (dict(dtype=7), 3), (dict(sigma=0.0), 4), (dict(parts=65), 4), (dict(q=NULL), 1), (dict(Lk=37441), 2),
])
def test_attention_noalloc_rejects(L, kw, status):
    from paper_2607_21848_amd import _lib
    assert _attention_noalloc(L, **kw) == status
    assert "biased_chunk_attention_noalloc" in _lib.last_error()


def test_attention_noalloc_nothing_to_do(L):
    assert _attention_noalloc(L, Lq=0) == 0
