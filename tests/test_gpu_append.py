"""Decode-time append on the GPU (through the C ABI) against the oracle.

New tokens are written into the static cache and their keys hashed against
the fixed projection with Algorithm 2 ("Given projection, computing
hashcode"); the cache rows must equal the new rows bit for bit, the codes
must equal the oracle's Algorithm 2 codes, neighbouring rows must be left
alone, and a multi-step decode loop (append one token, then decode over the
grown cache) must match the oracle step by step.
"""

import math

import numpy as np
import pytest
import torch

import oracle
from _helpers import oracle_build_of
from workloads import CONFIGS, make_layer

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2608_04405_amd as bpc
else:  # pragma: no cover
    bpc = None

DEV = "cuda"

@pytest.fixture(autouse=True, params=["fused", "fused-16k", "three-launch"])
def decode_path(request):
    """Every test here runs on each decode path: the single fused launch
    (the default wherever the step's workgroups fit on the GPU at once, on
    4096-key slices where those fit), the fused launch on 16384-key slices
    only, and the three launches (the path for larger steps)."""
    bpc.set_decode_path({"fused": 0, "fused-16k": 2, "three-launch": 1}[request.param])
    yield request.param
    bpc.set_decode_path(0)

TOL = 2e-3


def bits(t):
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def u32(t):
    return t.detach().cpu().contiguous().numpy().view(np.uint32)


def rel_err(o, ref):
    o = np.asarray(o, np.float64)
    return np.max(np.abs(o - ref), axis=-1) / np.max(np.abs(ref), axis=-1)


def announce(msg):
    print(msg, flush=True)


def randn_bf16(rng, shape, scale=1.0):
    return torch.from_numpy((scale * rng.standard_normal(shape)).astype(np.float32)).to(torch.bfloat16).to(DEV)


@pytest.mark.parametrize("L,shared", [(32, False), (64, True), (128, False)])
def test_append_rows_and_codes(L, shared):
    announce(f"[append rows] L={L} shared={shared}")
    rng = np.random.default_rng(L)
    B, Hkv, Ncap, pos, T = 2, 3, 700, 512, 7
    K = randn_bf16(rng, (B, Hkv, Ncap, 128))
    V = randn_bf16(rng, (B, Hkv, Ncap, 128))
    codes = torch.from_numpy(rng.integers(-2**31, 2**31, size=(B, Hkv, Ncap, L // 32), dtype=np.int64)
                             .astype(np.int32)).to(DEV)
    kn = randn_bf16(rng, (B, Hkv, T, 128), 2.0)
    vn = randn_bf16(rng, (B, Hkv, T, 128))
    P_np = (0.3 * rng.standard_normal((L, 128) if shared else (B, Hkv, L, 128))).astype(np.float32)
    P = torch.from_numpy(P_np).to(DEV)
    K0, V0, C0 = K.clone(), V.clone(), codes.clone()
    err = torch.empty(B, Hkv, T, device=DEV)
    bpc.append_kv(kn, vn, K, V, codes, P, pos, err_out=err)
    torch.cuda.synchronize()
    rows = slice(pos, pos + T)
    assert torch.equal(K[:, :, rows], kn) and torch.equal(V[:, :, rows], vn)
    for t0, t1 in ((K, K0), (V, V0), (codes, C0)):  # rows outside [pos, pos + T) untouched
        assert torch.equal(t0[:, :, :pos], t1[:, :, :pos]) and torch.equal(t0[:, :, pos + T:], t1[:, :, pos + T:])
    knb = bits(kn)
    cn = u32(codes)
    for b in range(B):
        for h in range(Hkv):
            Ph = P_np if shared else P_np[b, h]
            ref_codes, ref_err, _ = oracle.hash_keys(knb[b, h], Ph)
            assert np.array_equal(cn[b, h, rows], ref_codes), f"codes differ at {(b, h)}"
            np.testing.assert_allclose(err[b, h].cpu().numpy(), ref_err, rtol=1e-6, atol=1e-6)


def test_decode_loop_with_append():
    """Prefill (Algorithm 1 on the first N0 keys), then eight decode steps,
    each appending one token and decoding over the grown cache with a 2 %
    budget; a needle aligned with the next queries is appended at step 3
    and must be selected from then on (steps 3..7 use the one query the
    needle is aligned with)."""
    cfg = CONFIGS[1].replace(B=1, N=3000, needles=0)
    announce(f"[append loop] {cfg}")
    d = make_layer(cfg, device=DEV)
    steps = 8
    Ncap = cfg.N + steps
    rng = np.random.default_rng(5)
    K = torch.zeros(cfg.B, cfg.Hkv, Ncap, 128, dtype=torch.bfloat16, device=DEV)
    V = torch.zeros_like(K)
    K[:, :, :cfg.N] = d["K"]
    V[:, :, :cfg.N] = d["V"]
    codes = torch.zeros(cfg.B, cfg.Hkv, Ncap, cfg.W, dtype=torch.int32, device=DEV)
    P, _, _ = bpc.build_hash(K, d["G"].to(DEV), N=cfg.N, codes_out=codes)
    torch.cuda.synchronize()
    # the oracle side keeps its own cache: its build of the prefill keys,
    # then the appended rows and the codes its Algorithm 2 gives them
    Pn, cref, _ = oracle_build_of(P, codes, K, d["G"], [(0, h) for h in range(cfg.Hkv)], N=cfg.N)
    cref[:, :, cfg.N:] = 0
    Kref = np.zeros((cfg.B, cfg.Hkv, Ncap, 128), np.uint16)
    Vref = np.zeros_like(Kref)
    Kref[:, :, :cfg.N], Vref[:, :, :cfg.N] = bits(d["K"]), bits(d["V"])
    sm = 1.0 / math.sqrt(128)
    q_next = randn_bf16(rng, (cfg.B, cfg.Hq, 128))
    for t in range(steps):
        N = cfg.N + t + 1
        kn = randn_bf16(rng, (cfg.B, cfg.Hkv, 1, 128), 8.0)
        vn = randn_bf16(rng, (cfg.B, cfg.Hkv, 1, 128))
        if t == 3:  # a needle: the next queries' group sum, scaled far above the background
            qs = q_next.float().view(cfg.B, cfg.Hkv, cfg.G, 128).sum(2, keepdim=True)
            kn = (qs / qs.norm(dim=-1, keepdim=True) * 400.0).to(torch.bfloat16)
        bpc.append_kv(kn, vn, K, V, codes, P, N - 1)
        q = q_next
        q_next = randn_bf16(rng, (cfg.B, cfg.Hq, 128)) if t < 2 else q  # from step 3 on: one query
        k = math.ceil(0.02 * N)
        idx = torch.empty(cfg.B, cfg.Hkv, k, dtype=torch.int32, device=DEV)
        out = bpc.decode_attention(q, K, V, codes, P, k, sm, N=N, idx_out=idx)
        torch.cuda.synchronize()
        cn = u32(codes)
        Kref[:, :, N - 1], Vref[:, :, N - 1] = bits(kn)[:, :, 0], bits(vn)[:, :, 0]
        for h in range(cfg.Hkv):
            new_codes, _, _ = oracle.hash_keys(bits(kn)[0, h], Pn[0, h])
            assert np.array_equal(cn[0, h, N - 1:N], new_codes), f"step {t}: appended code differs at head {h}"
            cref[0, h, N - 1:N] = new_codes
            ref = oracle.decode_head(bits(q)[0, h * cfg.G:(h + 1) * cfg.G], Kref[0, h, :N], Vref[0, h, :N],
                                     cref[0, h, :N], Pn[0, h], k, sm)
            assert np.array_equal(idx[0, h].cpu().numpy(), ref["idx"]), f"step {t}: indices differ at head {h}"
            e = rel_err(out[0, h * cfg.G:(h + 1) * cfg.G].cpu().numpy(), ref["out"])
            assert np.all(e <= TOL), f"step {t}: output error {e.max():.3g} at head {h}"
            if t >= 3:
                assert cfg.N + 3 in idx[0, h].cpu().numpy(), f"step {t}: the appended needle is not selected"
    announce("append loop: 8 steps match the oracle")
