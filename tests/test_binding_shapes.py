"""The Python binding checks every tensor extent before it calls the library.

The kernels do no bounds checks of their own, so a tensor smaller than the
sizes passed to the library would be read or written out of bounds.  Each
case below builds CPU tensors of the right shapes, changes one extent, and
checks that the binding raises naming that tensor; with every shape right
it raises only because the tensors are not on a GPU.  Nothing reaches the
library (which could not launch on CPU tensors anyway), so this runs
without a GPU.
"""

import os

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2608_04405_amd", "libbpc.so")
pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libbpc.so not built")

B, Hq, Hkv, N, D, L, k = 2, 8, 2, 64, 128, 64, 5
W = L // 32
bf, f32, i32 = torch.bfloat16, torch.float32, torch.int32


@pytest.fixture(scope="module")
def bpc():
    import paper_2608_04405_amd as m
    return m


def base():
    return dict(q=torch.zeros(B, Hq, D, dtype=bf), K=torch.zeros(B, Hkv, N, D, dtype=bf),
                V=torch.zeros(B, Hkv, N, D, dtype=bf), codes=torch.zeros(B, Hkv, N, W, dtype=i32),
                P=torch.zeros(B, Hkv, L, D, dtype=f32))


def decode(bpc, over=None, **kw):
    a = base()
    a.update(over or {})
    return bpc.decode_attention(a["q"], a["K"], a["V"], a["codes"], a["P"], kw.pop("k", k), **kw)


def expect(fn, word):
    with pytest.raises((ValueError, TypeError)) as e:
        fn()
    assert word in str(e.value), str(e.value)


def test_decode_good_shapes_reach_the_device_check(bpc):
    expect(lambda: decode(bpc), "GPU")
    expect(lambda: decode(bpc, idx_out=torch.zeros(B, Hkv, k, dtype=i32), score_out=torch.zeros(B, Hkv, N, dtype=i32),
                          qcode_out=torch.zeros(B, Hkv, 8, W, dtype=i32), out=torch.zeros(B, Hq, D, dtype=f32)), "GPU")
    # a cache with room for more rows than N, and a shared projection
    big = dict(K=torch.zeros(B, Hkv, 2 * N, D, dtype=bf), V=torch.zeros(B, Hkv, 2 * N, D, dtype=bf),
               codes=torch.zeros(B, Hkv, 2 * N, W, dtype=i32), P=torch.zeros(Hkv, L, D, dtype=f32))
    expect(lambda: decode(bpc, big, N=N), "GPU")


@pytest.mark.parametrize("name,bad,word", [
    ("V", torch.zeros(B, Hkv, N - 1, D, dtype=bf), "V"),
    ("V", torch.zeros(B, Hkv + 1, N, D, dtype=bf), "V"),
    ("K", torch.zeros(B + 1, Hkv, N, D, dtype=bf), "K"),
    ("codes", torch.zeros(B, Hkv, N - 1, W, dtype=i32), "codes"),
    ("codes", torch.zeros(B, Hkv, N, W + 1, dtype=i32), "codes"),
    ("codes", torch.zeros(B, 1, N, W, dtype=i32), "codes"),
    ("P", torch.zeros(B, Hkv + 1, L, D, dtype=f32), "P"),
    ("P", torch.zeros(Hkv + 1, L, D, dtype=f32), "P"),
    ("P", torch.zeros(B, Hkv, 48, D, dtype=f32), "code length"),
    ("q", torch.zeros(B, Hq + 1, D, dtype=bf), "multiple"),
])
def test_decode_rejects_bad_inputs(bpc, name, bad, word):
    expect(lambda: decode(bpc, {name: bad}), word)


@pytest.mark.parametrize("kw,word", [
    (dict(out=torch.zeros(B, Hq, D - 1, dtype=f32)), "out"),
    (dict(idx_out=torch.zeros(B, Hkv, k + 1, dtype=i32)), "idx_out"),
    (dict(score_out=torch.zeros(B, Hkv, N - 1, dtype=i32)), "score_out"),
    (dict(qcode_out=torch.zeros(B, Hkv, 8, W + 1, dtype=i32)), "qcode_out"),
    (dict(k=N + 1), "k="),
    (dict(k=0), "k="),
    (dict(N=N + 1), "N="),
    (dict(serr=torch.zeros(B, Hkv + 1, 3, dtype=i32)), "serr"),
    (dict(serr=torch.zeros(B, Hkv, 3, dtype=i32), added_out=torch.zeros(B, Hkv, 4, dtype=i32)), "added_out"),
    (dict(added_out=torch.zeros(B, Hkv, 4, dtype=i32)), "serr"),
])
def test_decode_rejects_bad_outputs(bpc, kw, word):
    expect(lambda: decode(bpc, **kw), word)


def test_per_head_shapes(bpc):
    a = base()
    f = lambda **kw: bpc.decode_attention_per_head(a["q"], a["K"], a["V"], a["codes"], a["P"], k, **kw)  # noqa: E731
    expect(lambda: f(), "GPU")
    expect(lambda: f(idx_out=torch.zeros(B, Hkv, k, dtype=i32)), "idx_out")
    expect(lambda: f(score_out=torch.zeros(B, Hq, N + 1, dtype=i32)), "score_out")
    expect(lambda: bpc.decode_attention_per_head(a["q"], a["K"], a["V"][:, :, :N - 2], a["codes"], a["P"], k), "V")


def test_hash_and_build_shapes(bpc):
    K = torch.zeros(B, Hkv, N, D, dtype=bf)
    P = torch.zeros(B, Hkv, L, D, dtype=f32)
    G = torch.zeros(L, D, dtype=f32)
    expect(lambda: bpc.hash_keys(K, P), "GPU")
    expect(lambda: bpc.hash_keys(K, P, codes_out=torch.zeros(B, Hkv, N - 1, W, dtype=i32)), "codes_out")
    expect(lambda: bpc.hash_keys(K, P, err_out=torch.zeros(B, Hkv, N + 1, dtype=f32)), "err_out")
    expect(lambda: bpc.hash_keys(K, torch.zeros(B + 1, Hkv, L, D, dtype=f32)), "P")
    expect(lambda: bpc.hash_keys(K, P, N=N + 1), "N=")
    expect(lambda: bpc.build_hash(K, G), "GPU")
    expect(lambda: bpc.build_hash(K, torch.zeros(L, D + 1, dtype=f32)), "G")
    expect(lambda: bpc.build_hash(K, torch.zeros(40, D, dtype=f32)), "code length")
    expect(lambda: bpc.build_hash(K, G, P_out=torch.zeros(B, Hkv, L - 1, D, dtype=f32)), "P_out")
    expect(lambda: bpc.build_hash(K, G, codes_out=torch.zeros(B, Hkv, N, 1, dtype=i32)), "codes_out")
    expect(lambda: bpc.build_hash(K, G, err_out=torch.zeros(B, Hkv, N - 1, dtype=f32)), "err_out")
    expect(lambda: bpc.build_hash(K, G, fragile=torch.zeros(1, dtype=i32)), "fragile")


def test_append_select_dense_shapes(bpc):
    T = 3
    kn = torch.zeros(B, Hkv, T, D, dtype=bf)
    K = torch.zeros(B, Hkv, N, D, dtype=bf)
    codes = torch.zeros(B, Hkv, N, W, dtype=i32)
    P = torch.zeros(B, Hkv, L, D, dtype=f32)
    expect(lambda: bpc.append_kv(kn, kn, K, K, codes, P, N - T), "GPU")
    expect(lambda: bpc.append_kv(kn, kn, K, K, codes, P, N - T + 1), "pos=")
    expect(lambda: bpc.append_kv(kn, torch.zeros(B, Hkv, T + 1, D, dtype=bf), K, K, codes, P, 0), "v_new")
    expect(lambda: bpc.append_kv(kn, kn, K, K[:, :, :N - 1], codes, P, 0), "V")
    expect(lambda: bpc.append_kv(kn, kn, K, K, codes[:, :, :N - 1], P, N - T), "codes")
    expect(lambda: bpc.append_kv(kn, kn, K, K, codes, P, 0, err_out=torch.zeros(B, Hkv, T + 1, dtype=f32)), "err_out")
    err = torch.zeros(B, Hkv, N, dtype=f32)
    expect(lambda: bpc.select_hard(err, 4), "GPU")
    expect(lambda: bpc.select_hard(err, N + 1), "m=")
    expect(lambda: bpc.select_hard(err, 4, serr_out=torch.zeros(B, Hkv, 5, dtype=i32)), "serr_out")
    q = torch.zeros(B, Hq, D, dtype=bf)
    expect(lambda: bpc.dense_attention(q, K, K), "GPU")
    expect(lambda: bpc.dense_attention(q, K, K[:, :, :N - 1], N=N), "V")
    expect(lambda: bpc.dense_attention(q, K, K, out=torch.zeros(B, Hq + 1, D, dtype=f32)), "out")
