"""Per-query-head selection on the GPU (through the C ABI) against the oracle.

Each query head quantises its own projection, scores the codes of its KV
head, takes its own top-k and attends over it (oracle.decode_per_query_head).
Query planes, scores and indices are compared bit for bit and the output
within 2e-3 per row.  Cases: a group of one (where it is the ordinary decode
step), the 8B-shaped group of four on a ragged cache, strides that are not
linear in (sequence, KV head) and a projection shared across the batch (both
take the one-call-per-sequence path), and a group of eight.
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


def compare(q, K, V, codes, P, k, N, label, P_np=None, heads=None, codes_np=None):
    B, Hq, D = q.shape
    Hkv = K.shape[1]
    G = Hq // Hkv
    L = P.shape[-2]
    sm = 1.0 / math.sqrt(D)
    idx = torch.full((B, Hq, k), -1, dtype=torch.int32, device=DEV)
    sc = torch.empty(B, Hq, N, dtype=torch.int32, device=DEV)
    qc = torch.empty(B, Hq, 8, L // 32, dtype=torch.int32, device=DEV)
    out = bpc.decode_attention_per_head(q, K, V, codes, P, k, sm, N=N, idx_out=idx, score_out=sc, qcode_out=qc)
    torch.cuda.synchronize()
    P_np = P.cpu().numpy() if P_np is None else P_np
    qb, Kb, Vb = bits(q), bits(K), bits(V)
    cn = u32(codes) if codes_np is None else codes_np
    worst = 0.0
    for b, h in (heads or [(b, h) for b in range(B) for h in range(Hkv)]):
        Ph = P_np[b, h] if P_np.ndim == 4 else P_np[h]
        ref = oracle.decode_per_query_head(qb[b, h * G:(h + 1) * G], Kb[b, h, :N], Vb[b, h, :N], cn[b, h, :N], Ph,
                                           k, sm)
        rows = slice(h * G, (h + 1) * G)
        assert np.array_equal(u32(qc[b, rows]), ref["qcode"]), f"{label}: query planes differ at {(b, h)}"
        assert np.array_equal(sc[b, rows].cpu().numpy(), ref["scores"]), f"{label}: scores differ at {(b, h)}"
        assert np.array_equal(idx[b, rows].cpu().numpy(), ref["idx"]), f"{label}: indices differ at {(b, h)}"
        e = rel_err(out[b, rows].cpu().numpy(), ref["out"])
        worst = max(worst, float(e.max()))
        assert np.all(e <= TOL), f"{label}: output error {e.max():.3g} at {(b, h)}"
    announce(f"{label}: max relative output error {worst:.3g}")
    return out, idx


def test_per_head_group_of_one_is_the_decode_step():
    cfg = CONFIGS[0]  # 8 query heads on 8 KV heads
    announce(f"[per head] {cfg}")
    d = make_layer(cfg, device=DEV)
    P, codes, _ = bpc.build_hash(d["K"], d["G"].to(DEV))
    Pn, cn, _ = oracle_build_of(P, codes, d["K"], d["G"], [(0, h) for h in range(cfg.Hkv)])
    out, idx = compare(d["q"], d["K"], d["V"], codes, P, cfg.k, cfg.N, "per head G=1", P_np=Pn, codes_np=cn)
    idx_g = torch.empty(cfg.B, cfg.Hkv, cfg.k, dtype=torch.int32, device=DEV)
    out_g = bpc.decode_attention(d["q"], d["K"], d["V"], codes, P, cfg.k, idx_out=idx_g)
    torch.cuda.synchronize()
    assert torch.equal(idx, idx_g)
    if bpc.decode_path_taken(cfg.B, cfg.Hq, cfg.Hkv, cfg.N, cfg.L) == 1:
        assert torch.equal(out, out_g)
    else:
        # the fused step sums the weighted V rows on the matrix cores (other
        # rounding order), the per-head launches on the vector unit
        assert torch.allclose(out, out_g, rtol=1e-5, atol=1e-6), (out - out_g).abs().max().item()


def test_per_head_llama8b_ragged():
    cfg = CONFIGS[1].replace(B=2, N=20000)
    announce(f"[per head] {cfg}")
    d = make_layer(cfg, device=DEV)
    P, codes, _ = bpc.build_hash(d["K"], d["G"].to(DEV))
    heads = [(0, 0), (1, 5)]
    Pn, cn, _ = oracle_build_of(P, codes, d["K"], d["G"], heads)
    _, idx = compare(d["q"], d["K"], d["V"], codes, P, cfg.k, cfg.N, "per head 8B-shaped", P_np=Pn, heads=heads,
                     codes_np=cn)
    # the heads of a group do select differently (else the variant were moot)
    idn = idx.cpu().numpy()
    assert any(not np.array_equal(idn[0, 0], idn[0, g]) for g in range(1, cfg.G))


def test_per_head_nonlinear_strides_and_shared_projection():
    rng = np.random.default_rng(9)
    B, Hkv, G, N, Ncap, L, k = 3, 2, 4, 5000, 5008, 64, 97
    big = torch.from_numpy(rng.standard_normal((B, Hkv + 1, Ncap, 128)).astype(np.float32)).to(torch.bfloat16)
    K = big.to(DEV)[:, :Hkv]  # batch stride (Hkv + 1) x head stride: not linear in (b, h)
    V = torch.from_numpy(rng.standard_normal((B, Hkv, Ncap, 128)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    q = torch.from_numpy(rng.standard_normal((B, Hkv * G, 128)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    codes_np = rng.integers(0, 1 << 32, size=(B, Hkv, Ncap, L // 32), dtype=np.uint64).astype(np.uint32)
    codes = torch.from_numpy(codes_np.view(np.int32)).to(DEV)
    P_np = (0.3 * rng.standard_normal((Hkv, L, 128))).astype(np.float32)
    P = torch.from_numpy(P_np).to(DEV)  # shared across the batch (batch stride 0)
    compare(q, K, V, codes, P, k, N, "per head, non-linear strides, shared P", P_np=P_np)


def test_per_head_group_of_eight():
    rng = np.random.default_rng(10)
    B, Hkv, G, N, L, k = 1, 1, 8, 17000, 32, 340
    K = torch.from_numpy(rng.standard_normal((B, Hkv, N, 128)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    V = torch.from_numpy(rng.standard_normal((B, Hkv, N, 128)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    q = torch.from_numpy(rng.standard_normal((B, Hkv * G, 128)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    G_dirs = torch.from_numpy(rng.standard_normal((L, 128)).astype(np.float32)).to(DEV)
    P, codes, _ = bpc.build_hash(K, G_dirs)
    Pn, cn, _ = oracle_build_of(P, codes, K, G_dirs, [(0, 0)])
    compare(q, K, V, codes, P, k, N, "per head G=8", P_np=Pn, codes_np=cn)
