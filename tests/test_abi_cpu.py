"""The C ABI on the CPU: the library loads, exports what include/bpc.h
declares, sizes its workspaces, and rejects bad arguments on the host.

Every call here fails argument checking by construction (the pointers are
fake), so nothing is ever enqueued on a device.
"""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bpc.h")
LIB = os.path.join(ROOT, "paper_2608_04405_amd", "libbpc.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libbpc.so not built")

OK, EINVAL, EUNSUP, EALIGN, EWS, EHIP = 0, -1, -2, -3, -4, -5
FAKE = 0x10000  # 16-byte aligned, never dereferenced: every call below fails validation first


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(bpc_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    L = ctypes.CDLL(LIB)
    L.bpc_status_string.restype = ctypes.c_char_p
    L.bpc_last_error.restype = ctypes.c_char_p
    L.bpc_decode_workspace_bytes.restype = ctypes.c_size_t
    L.bpc_build_workspace_bytes.restype = ctypes.c_size_t
    return L


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert {"bpc_build_hash", "bpc_hash_keys", "bpc_decode_attention"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    for code, word in ((OK, b"ok"), (EINVAL, b"invalid"), (EUNSUP, b"unsupported"), (EALIGN, b"misaligned"),
                       (EWS, b"workspace"), (EHIP, b"HIP")):
        assert word in lib.bpc_status_string(code)
    assert lib.bpc_version() >= 100


def test_workspace_sizes(lib):
    ws = lib.bpc_decode_workspace_bytes
    assert ws(16, 32, 8, 131072, 128, 64, 2622) > 0
    assert ws(16, 32, 8, 131072, 128, 64, 2622) % 256 == 0
    assert ws(1, 8, 8, 4096, 128, 32, 82) < ws(1, 8, 8, 40000, 128, 32, 82)
    assert ws(1, 8, 8, 4096, 64, 32, 82) == 0  # D != 128
    assert ws(1, 8, 8, 4096, 128, 48, 82) == 0  # bad L
    assert ws(1, 8, 8, 4096, 128, 32, 0) == 0  # k < 1
    assert ws(1, 8, 8, 4096, 128, 32, 4097) == 0  # k > N
    assert ws(1, 6, 4, 4096, 128, 32, 8) == 0  # Hq % Hkv
    b = lib.bpc_build_workspace_bytes(2, 8, 1000, 128, 64)
    # one fp64 partial sum per 128-key chunk, (b, h) and coordinate, P and G
    # widened to fp64; no N x D residual
    assert b >= 2 * 8 * ((1000 + 127) // 128) * 128 * 8 + 2 * 8 * 64 * 128 * 8 + 64 * 128 * 8
    assert b < 2 * 8 * 1000 * 128 * 8 // 4
    # with the residual checkpoint: 1 KiB more per key, padded to 128-key chunks
    lib.bpc_build_checkpoint_workspace_bytes.restype = ctypes.c_size_t
    bc = lib.bpc_build_checkpoint_workspace_bytes(2, 8, 1000, 128, 64)
    assert bc - b >= 2 * 8 * 1024 * 128 * 8 and (bc - b) % 256 == 0 and bc < b + 2 * 8 * 1024 * 128 * 8 + 256
    assert lib.bpc_build_checkpoint_workspace_bytes(2, 8, 1000, 64, 64) == 0  # D != 128


_i64 = ctypes.c_int64


def _decode(lib, **kw):
    a = dict(q=FAKE, K=FAKE, sKb=8 * 4096 * 128, sKh=4096 * 128, sKn=128, V=FAKE, sVb=8 * 4096 * 128,
             sVh=4096 * 128, sVn=128, codes=FAKE, sCb=8 * 4096, sCh=4096, P=FAKE, sPb=8 * 32 * 128, sPh=32 * 128,
             B=1, Hq=8, Hkv=8, N=4096, D=128, L=32, k=82, sm=0.088, out=FAKE, idx=None, score=None, qcode=None,
             ws=FAKE, ws_bytes=0, stream=None)
    a.update(kw)
    f = lib.bpc_decode_attention
    f.restype = ctypes.c_int
    return f(ctypes.c_void_p(a["q"]), ctypes.c_void_p(a["K"]), _i64(a["sKb"]), _i64(a["sKh"]), _i64(a["sKn"]),
             ctypes.c_void_p(a["V"]), _i64(a["sVb"]), _i64(a["sVh"]), _i64(a["sVn"]), ctypes.c_void_p(a["codes"]),
             _i64(a["sCb"]), _i64(a["sCh"]), ctypes.c_void_p(a["P"]), _i64(a["sPb"]), _i64(a["sPh"]), a["B"],
             a["Hq"], a["Hkv"], a["N"], a["D"], a["L"], a["k"], ctypes.c_float(a["sm"]), ctypes.c_void_p(a["out"]),
             ctypes.c_void_p(a["idx"]), ctypes.c_void_p(a["score"]), ctypes.c_void_p(a["qcode"]),
             ctypes.c_void_p(a["ws"]), ctypes.c_size_t(a["ws_bytes"]), ctypes.c_void_p(a["stream"]))


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), EINVAL),
    (dict(out=None), EINVAL),
    (dict(K=None), EINVAL),
    (dict(codes=None), EINVAL),
    (dict(P=None), EINVAL),
    (dict(B=0), EINVAL),
    (dict(N=0), EINVAL),
    (dict(Hq=12), EINVAL),          # not a multiple of Hkv
    (dict(Hq=24), EUNSUP),          # group of 3
    (dict(Hq=8 * 32), EUNSUP),      # group of 32
    (dict(k=0), EINVAL),
    (dict(k=4097), EINVAL),
    (dict(D=64), EUNSUP),
    (dict(L=48), EUNSUP),
    (dict(sm=0.0), EINVAL),
    (dict(sm=float("nan")), EINVAL),
    (dict(sKn=100), EINVAL),
    (dict(sKn=132), EALIGN),
    (dict(K=FAKE + 8), EALIGN),
    (dict(q=FAKE + 2), EALIGN),
    (dict(idx=FAKE + 4), EALIGN),
    (dict(sPh=32 * 128 + 2), EALIGN),
    (dict(ws=None), EWS),
    (dict(ws_bytes=1024), EWS),     # too small
])
def test_decode_rejects(lib, kw, code):
    assert _decode(lib, **kw) == code
    assert lib.bpc_last_error() != b""


def test_decode_rejects_misaligned_workspace(lib):
    need = lib.bpc_decode_workspace_bytes(1, 8, 8, 4096, 128, 32, 82)
    assert _decode(lib, ws=FAKE + 16, ws_bytes=need) == EALIGN


def _hash(lib, **kw):
    a = dict(K=FAKE, sKb=0, sKh=4096 * 128, sKn=128, B=1, Hkv=8, N=4096, D=128, L=64, P=FAKE, sPb=0, sPh=0,
             codes=FAKE, sCb=8 * 4096 * 2, sCh=4096 * 2, err=None, frag=None, stream=None)
    a.update(kw)
    f = lib.bpc_hash_keys
    f.restype = ctypes.c_int
    return f(ctypes.c_void_p(a["K"]), _i64(a["sKb"]), _i64(a["sKh"]), _i64(a["sKn"]), a["B"], a["Hkv"], a["N"],
             a["D"], a["L"], ctypes.c_void_p(a["P"]), _i64(a["sPb"]), _i64(a["sPh"]), ctypes.c_void_p(a["codes"]),
             _i64(a["sCb"]), _i64(a["sCh"]), ctypes.c_void_p(a["err"]), ctypes.c_void_p(a["frag"]),
             ctypes.c_void_p(a["stream"]))


@pytest.mark.parametrize("kw,code", [
    (dict(K=None), EINVAL), (dict(P=None), EINVAL), (dict(codes=None), EINVAL), (dict(N=-1), EINVAL),
    (dict(L=96), EUNSUP), (dict(D=256), EUNSUP), (dict(sCh=4096 * 2 + 1), EALIGN), (dict(P=FAKE + 4), EALIGN),
    (dict(err=FAKE + 4), EALIGN), (dict(sPb=-4), EINVAL),
])
def test_hash_rejects(lib, kw, code):
    assert _hash(lib, **kw) == code


def _hash_mm(lib, **kw):
    a = dict(K=FAKE, sKb=0, sKh=4096 * 128, sKn=128, B=1, Hkv=8, N=4096, D=128, L=64, P=FAKE, sPb=0, sPh=0,
             codes=FAKE, sCb=8 * 4096 * 2, sCh=4096 * 2, frag=None, fall=None, stream=None)
    a.update(kw)
    f = lib.bpc_hash_keys_mm
    f.restype = ctypes.c_int
    return f(ctypes.c_void_p(a["K"]), _i64(a["sKb"]), _i64(a["sKh"]), _i64(a["sKn"]), a["B"], a["Hkv"], a["N"],
             a["D"], a["L"], ctypes.c_void_p(a["P"]), _i64(a["sPb"]), _i64(a["sPh"]), ctypes.c_void_p(a["codes"]),
             _i64(a["sCb"]), _i64(a["sCh"]), ctypes.c_void_p(a["frag"]), ctypes.c_void_p(a["fall"]),
             ctypes.c_void_p(a["stream"]))


@pytest.mark.parametrize("kw,code", [
    (dict(K=None), EINVAL), (dict(P=None), EINVAL), (dict(codes=None), EINVAL), (dict(N=0), EINVAL),
    (dict(B=0), EINVAL), (dict(L=96), EUNSUP), (dict(D=64), EUNSUP), (dict(sCh=4096 * 2 + 1), EALIGN),
    (dict(P=FAKE + 4), EALIGN), (dict(K=FAKE + 2), EALIGN), (dict(sKn=100), EINVAL), (dict(sPh=-4), EINVAL),
])
def test_hash_mm_rejects(lib, kw, code):
    assert _hash_mm(lib, **kw) == code


def _build(lib, **kw):
    a = dict(K=FAKE, sKb=0, sKh=4096 * 128, sKn=128, B=1, Hkv=8, N=4096, D=128, L=32, G=FAKE, P=FAKE,
             codes=FAKE, sCb=8 * 4096, sCh=4096, err=None, frag=None, ws=FAKE, ws_bytes=0, stream=None)
    a.update(kw)
    f = lib.bpc_build_hash
    f.restype = ctypes.c_int
    return f(ctypes.c_void_p(a["K"]), _i64(a["sKb"]), _i64(a["sKh"]), _i64(a["sKn"]), a["B"], a["Hkv"], a["N"],
             a["D"], a["L"], ctypes.c_void_p(a["G"]), ctypes.c_void_p(a["P"]), ctypes.c_void_p(a["codes"]),
             _i64(a["sCb"]), _i64(a["sCh"]), ctypes.c_void_p(a["err"]), ctypes.c_void_p(a["frag"]),
             ctypes.c_void_p(a["ws"]), ctypes.c_size_t(a["ws_bytes"]), ctypes.c_void_p(a["stream"]))


@pytest.mark.parametrize("kw,code", [
    (dict(G=None), EINVAL), (dict(P=None), EINVAL), (dict(codes=None), EINVAL), (dict(L=16), EUNSUP),
    (dict(ws=None), EWS), (dict(ws_bytes=100), EWS), (dict(G=FAKE + 8), EALIGN),
])
def test_build_rejects(lib, kw, code):
    assert _build(lib, **kw) == code


def _select_hard(lib, **kw):
    a = dict(err=FAKE, sEb=8 * 4096, sEh=4096, B=1, Hkv=8, N=4096, m=9, out=FAKE, stream=None)
    a.update(kw)
    f = lib.bpc_select_hard
    f.restype = ctypes.c_int
    return f(ctypes.c_void_p(a["err"]), _i64(a["sEb"]), _i64(a["sEh"]), a["B"], a["Hkv"], a["N"], a["m"],
             ctypes.c_void_p(a["out"]), ctypes.c_void_p(a["stream"]))


@pytest.mark.parametrize("kw,code", [
    (dict(err=None), EINVAL),
    (dict(out=None), EINVAL),
    (dict(B=0), EINVAL),
    (dict(m=-1), EINVAL),
    (dict(m=4097), EINVAL),
    (dict(sEh=-1), EINVAL),
    (dict(err=FAKE + 2), EALIGN),
    (dict(out=FAKE + 1), EALIGN),
])
def test_select_hard_rejects(lib, kw, code):
    assert _select_hard(lib, **kw) == code
    assert lib.bpc_last_error() != b""


def test_select_hard_empty_set_launches_nothing(lib):
    # m = 0 selects nothing: success without touching the (fake) pointers
    assert _select_hard(lib, m=0, err=None, out=None) == OK


def _decode_eas(lib, **kw):
    a = dict(q=FAKE, K=FAKE, sKb=8 * 4096 * 128, sKh=4096 * 128, sKn=128, V=FAKE, sVb=8 * 4096 * 128,
             sVh=4096 * 128, sVn=128, codes=FAKE, sCb=8 * 4096, sCh=4096, P=FAKE, sPb=8 * 32 * 128, sPh=32 * 128,
             B=1, Hq=8, Hkv=8, N=4096, D=128, L=32, k=74, sm=0.088, serr=FAKE, sSb=8 * 8, sSh=8, m=8, out=FAKE,
             idx=None, added=None, ws=FAKE, ws_bytes=0, stream=None)
    a.update(kw)
    f = lib.bpc_decode_attention_eas
    f.restype = ctypes.c_int
    return f(ctypes.c_void_p(a["q"]), ctypes.c_void_p(a["K"]), _i64(a["sKb"]), _i64(a["sKh"]), _i64(a["sKn"]),
             ctypes.c_void_p(a["V"]), _i64(a["sVb"]), _i64(a["sVh"]), _i64(a["sVn"]), ctypes.c_void_p(a["codes"]),
             _i64(a["sCb"]), _i64(a["sCh"]), ctypes.c_void_p(a["P"]), _i64(a["sPb"]), _i64(a["sPh"]), a["B"],
             a["Hq"], a["Hkv"], a["N"], a["D"], a["L"], a["k"], ctypes.c_float(a["sm"]), ctypes.c_void_p(a["serr"]),
             _i64(a["sSb"]), _i64(a["sSh"]), a["m"], ctypes.c_void_p(a["out"]), ctypes.c_void_p(a["idx"]),
             ctypes.c_void_p(a["added"]), ctypes.c_void_p(a["ws"]), ctypes.c_size_t(a["ws_bytes"]),
             ctypes.c_void_p(a["stream"]))


@pytest.mark.parametrize("kw,code", [
    (dict(serr=None), EINVAL),       # m > 0 needs the hard set
    (dict(m=-1), EINVAL),
    (dict(m=4097), EINVAL),
    (dict(sSh=-8), EINVAL),
    (dict(added=FAKE + 4), EALIGN),
    (dict(k=0), EINVAL),
    (dict(q=None), EINVAL),
    (dict(ws_bytes=1024), EWS),
])
def test_decode_eas_rejects(lib, kw, code):
    assert _decode_eas(lib, **kw) == code
    assert lib.bpc_last_error() != b""


def _append(lib, **kw):
    a = dict(kn=FAKE, sKnb=8 * 128, sKnh=128, sKnt=128, vn=FAKE, sVnb=8 * 128, sVnh=128, sVnt=128, K=FAKE,
             sKb=8 * 4096 * 128, sKh=4096 * 128, sKn=128, V=FAKE, sVb=8 * 4096 * 128, sVh=4096 * 128, sVn=128,
             codes=FAKE, sCb=8 * 4096 * 2, sCh=4096 * 2, P=FAKE, sPb=8 * 64 * 128, sPh=64 * 128, B=1, Hkv=8,
             Ncap=4096, pos=4095, T=1, D=128, L=64, err=None, frag=None, stream=None)
    a.update(kw)
    f = lib.bpc_append_kv
    f.restype = ctypes.c_int
    v = ctypes.c_void_p
    return f(v(a["kn"]), _i64(a["sKnb"]), _i64(a["sKnh"]), _i64(a["sKnt"]), v(a["vn"]), _i64(a["sVnb"]),
             _i64(a["sVnh"]), _i64(a["sVnt"]), v(a["K"]), _i64(a["sKb"]), _i64(a["sKh"]), _i64(a["sKn"]), v(a["V"]),
             _i64(a["sVb"]), _i64(a["sVh"]), _i64(a["sVn"]), v(a["codes"]), _i64(a["sCb"]), _i64(a["sCh"]),
             v(a["P"]), _i64(a["sPb"]), _i64(a["sPh"]), a["B"], a["Hkv"], a["Ncap"], a["pos"], a["T"], a["D"],
             a["L"], v(a["err"]), v(a["frag"]), v(a["stream"]))


@pytest.mark.parametrize("kw,code", [
    (dict(pos=4096), EINVAL),        # past the cache
    (dict(pos=4090, T=7), EINVAL),
    (dict(pos=-1), EINVAL),
    (dict(T=0), EINVAL),
    (dict(kn=None), EINVAL),
    (dict(vn=None), EINVAL),
    (dict(V=None), EINVAL),
    (dict(codes=None), EINVAL),
    (dict(P=None), EINVAL),
    (dict(D=64), EUNSUP),
    (dict(L=16), EUNSUP),
    (dict(sCh=4097), EALIGN),        # not a multiple of the code words
    (dict(kn=FAKE + 8), EALIGN),
    (dict(err=FAKE + 4), EALIGN),
])
def test_append_rejects(lib, kw, code):
    assert _append(lib, **kw) == code
    assert lib.bpc_last_error() != b""


def test_dense_workspace_and_rejects(lib):
    ws = lib.bpc_dense_workspace_bytes
    ws.restype = ctypes.c_size_t
    assert ws(16, 32, 8, 131072, 128) == 16 * 8 * 8 * 4 * 130 * 4
    assert ws(1, 8, 8, 4096, 64) == 0
    f = lib.bpc_dense_attention
    f.restype = ctypes.c_int

    def call(**kw):
        a = dict(q=FAKE, K=FAKE, V=FAKE, B=1, Hq=8, Hkv=8, N=4096, D=128, sm=0.088, out=FAKE, ws=FAKE, wsb=0)
        a.update(kw)
        v = ctypes.c_void_p
        return f(v(a["q"]), v(a["K"]), _i64(8 * 4096 * 128), _i64(4096 * 128), _i64(128), v(a["V"]),
                 _i64(8 * 4096 * 128), _i64(4096 * 128), _i64(128), a["B"], a["Hq"], a["Hkv"], a["N"], a["D"],
                 ctypes.c_float(a["sm"]), v(a["out"]), v(a["ws"]), ctypes.c_size_t(a["wsb"]), None)

    for kw, code in ((dict(q=None), EINVAL), (dict(Hq=12), EINVAL), (dict(Hq=24), EUNSUP), (dict(D=64), EUNSUP),
                     (dict(sm=0.0), EINVAL), (dict(K=FAKE + 2), EALIGN), (dict(wsb=16), EWS)):
        assert call(**kw) == code, kw


def test_per_head_workspace_and_rejects(lib):
    ws = lib.bpc_decode_per_head_workspace_bytes
    ws.restype = ctypes.c_size_t
    assert ws(16, 32, 8, 131072, 128, 64, 2622) >= lib.bpc_decode_workspace_bytes(16, 32, 8, 131072, 128, 64, 2622)
    assert ws(1, 8, 8, 4096, 64, 32, 82) == 0  # D != 128
    assert ws(1, 12, 8, 4096, 128, 32, 82) == 0  # Hq % Hkv
    f = lib.bpc_decode_attention_per_head
    f.restype = ctypes.c_int

    def call(**kw):
        a = dict(q=FAKE, K=FAKE, sKb=8 * 4096 * 128, sKh=4096 * 128, sKn=128, V=FAKE, sVb=8 * 4096 * 128,
                 sVh=4096 * 128, sVn=128, codes=FAKE, sCb=8 * 4096, sCh=4096, P=FAKE, sPb=8 * 32 * 128,
                 sPh=32 * 128, B=1, Hq=32, Hkv=8, N=4096, D=128, L=32, k=82, sm=0.088, ws=FAKE, ws_bytes=0)
        a.update(kw)
        return f(ctypes.c_void_p(a["q"]), ctypes.c_void_p(a["K"]), _i64(a["sKb"]), _i64(a["sKh"]), _i64(a["sKn"]),
                 ctypes.c_void_p(a["V"]), _i64(a["sVb"]), _i64(a["sVh"]), _i64(a["sVn"]),
                 ctypes.c_void_p(a["codes"]), _i64(a["sCb"]), _i64(a["sCh"]), ctypes.c_void_p(a["P"]),
                 _i64(a["sPb"]), _i64(a["sPh"]), a["B"], a["Hq"], a["Hkv"], a["N"], a["D"], a["L"], a["k"],
                 ctypes.c_float(a["sm"]), ctypes.c_void_p(FAKE), None, None, None, ctypes.c_void_p(a["ws"]),
                 ctypes.c_size_t(a["ws_bytes"]), None)

    assert call(Hq=12) == EINVAL
    assert call(K=None) == EINVAL
    assert call(L=48) == EUNSUP
    assert call(ws=None) == EWS
    assert call(ws_bytes=1024) == EWS
    assert call(k=0, ws_bytes=1 << 40) == EINVAL
    assert call(D=64, ws_bytes=1 << 40) == EUNSUP
    # one call per sequence (batch stride != Hkv x head stride): a later
    # sequence's codes pointer that is not 16-byte aligned is found before
    # the first sequence launches (no HIP call is reached, so no EHIP here)
    assert call(B=2, sCb=8 * 4096 + 1, ws_bytes=1 << 40) == EALIGN
    assert b"sequence 1 of 2" in lib.bpc_last_error()


def test_decode_eas_rejects_misaligned_serr(lib):
    assert _decode_eas(lib, serr=FAKE + 2) == EALIGN
    assert b"serr" in lib.bpc_last_error()
