"""HIP path (through the C ABI) against the CPU oracle, on the same inputs.

Bar: packed codes, projections, query planes, scores and selected indices
bit-exact; attention output within a relative error of 2e-3 per (sequence,
query head) row: max_d |o - o_ref| / max_d |o_ref|.
"""

import os

import numpy as np
import pytest
import torch

import oracle
from _helpers import oracle_build_of
from workloads import CONFIGS, make_layer

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2608_04405_amd as bpc
else:  # pragma: no cover - collected on CPU-only machines, never run
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
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_example.json")


def bits(t):
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def u32(t):
    return t.detach().cpu().contiguous().numpy().view(np.uint32)


def rel_err(o, ref):
    o = np.asarray(o, np.float64)
    return np.max(np.abs(o - ref), axis=-1) / np.max(np.abs(ref), axis=-1)


def to_dev_bits(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(DEV)


def announce(msg):
    print(msg, flush=True)


# ------------------------------------------------------------------ fixtures

@pytest.fixture(scope="module")
def tiny():
    cfg = CONFIGS[0]
    announce(f"[tiny] {cfg}")
    d = make_layer(cfg, device="cpu")
    host = {k: bits(d[k]) for k in ("q", "K", "V")}
    host["G"] = d["G"].numpy()
    builds = [oracle.build_binary_pcs(host["K"][0, h], host["G"]) for h in range(cfg.Hkv)]
    dev = {k: d[k].to(DEV) for k in ("q", "K", "V", "G")}
    return cfg, host, dev, builds


# ------------------------------------------------------------------ Algorithm 1

def test_build_parity_tiny(tiny):
    cfg, host, dev, builds = tiny
    frag = torch.zeros(1, dtype=torch.int64, device=DEV)
    err = torch.empty(cfg.B, cfg.Hkv, cfg.N, dtype=torch.float32, device=DEV)
    P, codes, _ = bpc.build_hash(dev["K"], dev["G"], err_out=err, fragile=frag)
    torch.cuda.synchronize()
    nfrag = 0
    for h in range(cfg.Hkv):
        Po, co, eo, fo = builds[h]
        nfrag += fo
        assert np.array_equal(u32(codes[0, h]), co), f"codes differ, head {h}"
        assert np.array_equal(P[0, h].cpu().numpy(), Po), f"P differs, head {h}"
        np.testing.assert_allclose(err[0, h].cpu().numpy(), eo.astype(np.float32), rtol=1e-6, atol=1e-6)
    assert int(frag.item()) == nfrag


@pytest.mark.parametrize("checkpoint", [False, True], ids=["recompute", "checkpoint"])
# 33330 keys: 261 chunk sums of 128 keys, folded in blocks of 32 with a short
# last block of 5 before the per-(b, h) tree; 32769 keys: a last block of one
# chunk sum holding one key
@pytest.mark.parametrize("L,N,B,H", [(64, 1000, 2, 2), (128, 300, 1, 3), (32, 513, 1, 1), (64, 33330, 1, 1),
                                     (32, 32769, 1, 1)])
def test_build_parity_ragged_strided(L, N, B, H, checkpoint):
    announce(f"[build ragged] L={L} N={N} B={B} H={H} checkpoint={checkpoint}")
    rng = np.random.default_rng(L + N)
    Ncap = N + 24
    A = rng.standard_normal((8, 128))
    Kf = rng.standard_normal((B, H, Ncap, 8)) @ A + 0.1 * rng.standard_normal((B, H, Ncap, 128))
    K = torch.from_numpy(Kf.astype(np.float32)).to(torch.bfloat16).to(DEV)
    G = torch.from_numpy(rng.standard_normal((L, 128)).astype(np.float32)).to(DEV)
    codes = torch.zeros(B, H, Ncap, L // 32, dtype=torch.int32, device=DEV)
    P, codes, _ = bpc.build_hash(K, G, N=N, codes_out=codes, checkpoint=checkpoint)
    torch.cuda.synchronize()
    Kb = bits(K)
    for b in range(B):
        for h in range(H):
            Po, co, _, _ = oracle.build_binary_pcs(Kb[b, h, :N], G.cpu().numpy())
            assert np.array_equal(u32(codes[b, h, :N]), co)
            assert np.array_equal(P[b, h].cpu().numpy(), Po)
            assert np.all(u32(codes[b, h, N:]) == 0)  # rows beyond N untouched


def test_build_golden_worked_example():
    import json
    g = json.load(open(GOLDEN))
    K = np.zeros((4, 128), np.float32)
    K[:, :4] = np.asarray(g["K_small"])
    Kt = torch.from_numpy(K).to(torch.bfloat16).to(DEV)[None, None]
    L = g["L_padded"]
    Gm = np.random.default_rng(0).standard_normal((L, 128)).astype(np.float32)
    Gm[:2] = 0
    Gm[:2, :4] = np.asarray(g["G_small"])
    frag = torch.zeros(1, dtype=torch.int64, device=DEV)
    err = torch.empty(1, 1, 4, dtype=torch.float32, device=DEV)
    P, codes, _ = bpc.build_hash(Kt, torch.from_numpy(Gm).to(DEV), err_out=err, fragile=frag)
    torch.cuda.synchronize()
    assert u32(codes[0, 0])[:, 0].tolist() == g["codes_padded"]
    Pn = P[0, 0].cpu().numpy()
    assert np.array_equal(Pn[:2, :4], np.asarray(g["P_small"], np.float32)) and np.all(Pn[2:] == 0)
    assert int(frag.item()) == g["fragile_padded"] and np.all(err.cpu().numpy() == 0)
    # decode on the worked example: scores and the top-2 with its tie
    q = np.zeros((1, 1, 128), np.float32)
    q[0, 0, :4] = g["query"]
    qt = torch.from_numpy(q).to(torch.bfloat16).to(DEV)
    V = torch.from_numpy(np.eye(4, 128, dtype=np.float32)).to(torch.bfloat16).to(DEV)[None, None].contiguous()
    idx = torch.empty(1, 1, g["k"], dtype=torch.int32, device=DEV)
    sc = torch.empty(1, 1, 4, dtype=torch.int32, device=DEV)
    out = bpc.decode_attention(qt, Kt, V, codes, P, g["k"], idx_out=idx, score_out=sc)
    torch.cuda.synchronize()
    assert sc.cpu().numpy().ravel().tolist() == g["scores"]
    assert idx.cpu().numpy().ravel().tolist() == g["topk"]
    # softmax over keys 0 and 1 with logits 4/sqrt(128) and 0, values e0 and e1
    w0 = 1.0 / (1.0 + np.exp(-4.0 / np.sqrt(128)))
    # the fused step weighs V on the matrix cores with each probability split
    # into two bf16 parts (about 16 significant bits, relative error below
    # 4e-6); the three-launch step keeps fp32 throughout
    np.testing.assert_allclose(out.cpu().numpy()[0, 0, :2], [w0, 1 - w0], rtol=1e-5)


# ------------------------------------------------------------------ Algorithm 2

@pytest.mark.parametrize("L", [32, 64, 128])
@pytest.mark.parametrize("shared", [False, True])
def test_hash_parity(L, shared):
    announce(f"[hash] L={L} shared={shared}")
    rng = np.random.default_rng(L)
    B, H, N = 2, 2, 777
    K = torch.from_numpy(rng.standard_normal((B, H, N, 128)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    if shared:
        P = torch.from_numpy((0.3 * rng.standard_normal((L, 128))).astype(np.float32)).to(DEV)
    else:
        P = torch.from_numpy((0.3 * rng.standard_normal((B, H, L, 128))).astype(np.float32)).to(DEV)
    frag = torch.zeros(1, dtype=torch.int64, device=DEV)
    err = torch.empty(B, H, N, dtype=torch.float32, device=DEV)
    codes, _ = bpc.hash_keys(K, P, err_out=err, fragile=frag)
    torch.cuda.synchronize()
    Kb = bits(K)
    nf = 0
    for b in range(B):
        for h in range(H):
            Ph = P.cpu().numpy() if shared else P[b, h].cpu().numpy()
            co, eo, fo = oracle.hash_keys(Kb[b, h], Ph)
            nf += fo
            assert np.array_equal(u32(codes[b, h]), co)
            np.testing.assert_allclose(err[b, h].cpu().numpy(), eo.astype(np.float32), rtol=1e-6, atol=1e-6)
    assert int(frag.item()) == nf


def test_hash_reproduces_build_on_rank1():
    rng = np.random.default_rng(3)
    h0 = np.where(rng.random(700) < 0.5, 1.0, -1.0)
    p0 = torch.from_numpy(rng.standard_normal(128).astype(np.float32)).to(torch.bfloat16).double().numpy()
    K = torch.from_numpy(np.outer(h0, p0).astype(np.float32)).to(torch.bfloat16).to(DEV)[None, None].contiguous()
    G = torch.from_numpy(rng.standard_normal((64, 128)).astype(np.float32)).to(DEV)
    P, c1, _ = bpc.build_hash(K, G)
    c2, _ = bpc.hash_keys(K, P)
    torch.cuda.synchronize()
    assert torch.equal(c1, c2)


# ------------------------------------------------------------------ decode

def _decode_and_compare(q, K, V, codes_np, P_np, k, N=None, heads=None, sm=None, G=None, label=""):
    """Run the GPU decode with the oracle's codes/P and compare (host arrays in)."""
    B, Hq, D = q.shape
    Hkv = K.shape[1]
    Gq = Hq // Hkv
    N = K.shape[2] if N is None else N
    sm = 1.0 / np.sqrt(D) if sm is None else sm
    codes = torch.from_numpy(np.ascontiguousarray(codes_np).view(np.int32)).to(DEV)
    P = torch.from_numpy(np.ascontiguousarray(P_np)).to(DEV)
    L = P_np.shape[-2]
    idx = torch.full((B, Hkv, k), -1, dtype=torch.int32, device=DEV)
    sc = torch.empty(B, Hkv, N, dtype=torch.int32, device=DEV)
    qc = torch.empty(B, Hkv, 8, L // 32, dtype=torch.int32, device=DEV)
    out = bpc.decode_attention(q, K, V, codes, P, k, sm, N=N, idx_out=idx, score_out=sc, qcode_out=qc)
    torch.cuda.synchronize()
    qb, Kb, Vb = bits(q), bits(K), bits(V)
    heads = [(b, h) for b in range(B) for h in range(Hkv)] if heads is None else heads
    worst = 0.0
    for b, h in heads:
        Ph = P_np if P_np.ndim == 2 else P_np[b, h]
        ref = oracle.decode_head(qb[b, h * Gq:(h + 1) * Gq], Kb[b, h, :N], Vb[b, h, :N], codes_np[b, h, :N], Ph, k, sm)
        assert np.array_equal(u32(qc[b, h]), ref["qcode"]), f"{label} qcode differs at {(b, h)}"
        assert np.array_equal(sc[b, h].cpu().numpy(), ref["scores"]), f"{label} scores differ at {(b, h)}"
        assert np.array_equal(idx[b, h].cpu().numpy(), ref["idx"]), f"{label} indices differ at {(b, h)}"
        e = rel_err(out[b, h * Gq:(h + 1) * Gq].cpu().numpy(), ref["out"])
        worst = max(worst, float(e.max()))
        assert np.all(e <= TOL), f"{label} output error {e.max():.3g} at {(b, h)}"
    announce(f"{label}: max relative output error {worst:.3g}")
    return out, idx


def test_decode_parity_tiny(tiny):
    cfg, host, dev, builds = tiny
    codes = np.stack([b[1] for b in builds])[None]
    P = np.stack([b[0] for b in builds])[None]
    _decode_and_compare(dev["q"], dev["K"], dev["V"], codes, P, cfg.k, label="tiny decode")


def test_full_chain_tiny(tiny):
    """GPU build + GPU decode against oracle build + oracle decode."""
    cfg, host, dev, builds = tiny
    P, codes, _ = bpc.build_hash(dev["K"], dev["G"])
    idx = torch.empty(cfg.B, cfg.Hkv, cfg.k, dtype=torch.int32, device=DEV)
    out = bpc.decode_attention(dev["q"], dev["K"], dev["V"], codes, P, cfg.k, idx_out=idx)
    torch.cuda.synchronize()
    sm = 1.0 / np.sqrt(cfg.D)
    for h in range(cfg.Hkv):
        Po, co = builds[h][0], builds[h][1]
        ref = oracle.decode_head(host["q"][0, h * cfg.G:(h + 1) * cfg.G], host["K"][0, h], host["V"][0, h], co, Po,
                                 cfg.k, sm)
        assert np.array_equal(idx[0, h].cpu().numpy(), ref["idx"])
        assert np.all(rel_err(out[0, h * cfg.G:(h + 1) * cfg.G].cpu().numpy(), ref["out"]) <= TOL)
        # the planted needles are selected (the oracle recalls all of them)
    pos = make_layer(cfg, device="cpu")["needle_pos"].numpy()
    for h in range(cfg.Hkv):
        assert np.all(np.isin(pos[0, h], idx[0, h].cpu().numpy()))


def test_decode_parity_llama8b_shape():
    cfg = CONFIGS[1]
    announce(f"[llama8b decode] {cfg}")
    d = make_layer(cfg, device="cpu")
    K, V, q = (d[x].to(DEV) for x in ("K", "V", "q"))
    G = d["G"].to(DEV)
    P, codes, _ = bpc.build_hash(K, G)
    torch.cuda.synchronize()
    heads = [(0, 0), (0, 5)]
    Pn, cn, _ = oracle_build_of(P, codes, K, G, heads)  # the oracle's own build of the checked heads
    _decode_and_compare(q, K, V, cn, Pn, cfg.k, heads=heads, label="llama8b decode")


def _random_case(rng, B, Hq, Hkv, N, L, Ncap=None, code_pool=None, qscale=1.0):
    Ncap = N if Ncap is None else Ncap
    q = torch.from_numpy((qscale * rng.standard_normal((B, Hq, 128))).astype(np.float32)).to(torch.bfloat16).to(DEV)
    K = torch.from_numpy(rng.standard_normal((B, Hkv, Ncap, 128)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    V = torch.from_numpy(rng.standard_normal((B, Hkv, Ncap, 128)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    W = L // 32
    if code_pool is None:
        codes = rng.integers(0, 1 << 32, size=(B, Hkv, Ncap, W), dtype=np.uint64).astype(np.uint32)
    else:  # few distinct codes -> massive score ties
        pool = rng.integers(0, 1 << 32, size=(code_pool, W), dtype=np.uint64).astype(np.uint32)
        codes = pool[rng.integers(0, code_pool, size=(B, Hkv, Ncap))]
    P = (0.5 * rng.standard_normal((B, Hkv, L, 128))).astype(np.float32)
    return q, K, V, codes, P


@pytest.mark.parametrize("case", [
    dict(B=1, Hq=4, Hkv=4, N=1, L=32, k=1),                       # a single key
    dict(B=1, Hq=4, Hkv=1, N=300, L=64, k=300),                   # k = N: every key
    dict(B=2, Hq=8, Hkv=4, N=5000, L=64, k=1),                    # k = 1
    dict(B=1, Hq=16, Hkv=1, N=16385, L=128, k=400),               # two slices, last holds one key
    dict(B=1, Hq=8, Hkv=8, N=50000, L=32, k=999, pool=3),         # multi-slice, massive ties
    dict(B=2, Hq=2, Hkv=2, N=40000, L=64, k=20000, pool=50),      # k larger than a slice
    dict(B=1, Hq=32, Hkv=4, N=20000, L=128, k=300, Ncap=20100),   # G = 8, strided cache
    dict(B=1, Hq=16, Hkv=16, N=3000, L=32, k=61),                 # G = 1
    dict(B=1, Hq=2, Hkv=1, N=70000, L=64, k=1400),                # G = 2, five slices
    dict(B=1, Hq=4, Hkv=2, N=1001, L=32, k=30),                   # last 16-byte group holds one key
    dict(B=2, Hq=4, Hkv=2, N=333, L=64, k=7, pool=5),             # odd key count, ties
    dict(B=1, Hq=8, Hkv=2, N=65537, L=64, k=1311),                # ragged second run
    dict(B=1, Hq=2, Hkv=1, N=1100000, L=32, k=50000, pool=40),    # over a million keys (68 slices): two-round threshold path
])
def test_decode_edge_cases(case):
    announce(f"[decode edge] {case}")
    rng = np.random.default_rng(sum(case.values()))
    q, K, V, codes, P = _random_case(rng, case["B"], case["Hq"], case["Hkv"], case["N"], case["L"], case.get("Ncap"),
                                     case.get("pool"))
    _decode_and_compare(q, K, V, codes, P, case["k"], N=case["N"], label=f"edge {case}")


def test_decode_threshold_below_the_windows():
    """Two slices, each with 60 keys whose code equals the query's sign plane
    (distance 0) and all other keys far away, k = 100: every slice's k-th
    smallest distance is far above 0, so the threshold lies below the
    per-slice windows the one-round threshold reads and the exact two-round
    path must produce it (ties at distance 0 go to the lowest indices)."""
    rng = np.random.default_rng(11)
    N, L, k = 32768, 64, 100
    announce(f"[decode window miss] N={N} L={L} k={k}")
    q, K, V, codes, P = _random_case(rng, 1, 4, 1, N, L)
    planes = oracle.quantize_query(bits(q)[0], P[0, 0])["qcode"]
    near = np.r_[0:60, 16384:16444]
    codes[0, 0, near] = planes[0]
    _, idx = _decode_and_compare(q, K, V, codes, P, k, label="window miss")
    assert np.array_equal(idx[0, 0].cpu().numpy(), near[:k])


def test_decode_garbage_workspace():
    """Only the workspace's counter region (its first DECODE_ZEROED_BYTES) needs zeroing
    once: a first call on a workspace holding random bytes elsewhere, and
    later calls on the same workspace, all match the oracle, on the fused
    path and on the three-launch path."""
    rng = np.random.default_rng(21)
    q, K, V, codes, P = _random_case(rng, 2, 8, 2, 40000, 64, code_pool=30)
    B, Hq, Hkv, N, L, k = 2, 8, 2, 40000, 64, 800
    ws = torch.randint(0, 256, (bpc.decode_workspace_bytes(B, Hq, Hkv, N, L, k),), dtype=torch.uint8, device=DEV)
    ws[:bpc.DECODE_ZEROED_BYTES] = 0
    cd = torch.from_numpy(codes.view(np.int32)).to(DEV)
    Pd = torch.from_numpy(P).to(DEV)
    outs = []
    for _ in range(3):
        idx = torch.empty(B, Hkv, k, dtype=torch.int32, device=DEV)
        outs.append((bpc.decode_attention(q, K, V, cd, Pd, k, workspace=ws, idx_out=idx).clone(), idx))
    torch.cuda.synchronize()
    qb, Kb, Vb = bits(q), bits(K), bits(V)
    for b in range(B):
        for h in range(Hkv):
            ref = oracle.decode_head(qb[b, 4 * h:4 * h + 4], Kb[b, h], Vb[b, h], codes[b, h], P[b, h], k,
                                     1 / np.sqrt(128))
            for out, idx in outs:
                assert np.array_equal(idx[b, h].cpu().numpy(), ref["idx"])
                assert np.all(rel_err(out[b, 4 * h:4 * h + 4].cpu().numpy(), ref["out"]) <= TOL)
    assert all(torch.equal(outs[0][0], o) for o, _ in outs[1:])


def test_decode_graph_replay():
    """A decode step captured in a HIP graph gives the eager result on every
    replay, with eager work and synchronisations between the replays."""
    rng = np.random.default_rng(22)
    q, K, V, codes, P = _random_case(rng, 2, 8, 2, 30000, 64)
    k = 600
    cd = torch.from_numpy(codes.view(np.int32)).to(DEV)
    Pd = torch.from_numpy(P).to(DEV)
    ws = torch.zeros(bpc.decode_workspace_bytes(2, 8, 2, 30000, 64, k), dtype=torch.uint8, device=DEV)
    out = torch.empty(2, 8, 128, dtype=torch.float32, device=DEV)
    eager = bpc.decode_attention(q, K, V, cd, Pd, k, out=torch.empty_like(out), workspace=ws).clone()
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        bpc.decode_attention(q, K, V, cd, Pd, k, out=out, workspace=ws, stream=s)  # warm-up on the side stream
        s.synchronize()
        with torch.cuda.graph(g, stream=s):
            bpc.decode_attention(q, K, V, cd, Pd, k, out=out, workspace=ws, stream=s)
    torch.cuda.synchronize()
    for r in range(4):
        out.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {r} differs from the eager result"
        bpc.decode_attention(q, K, V, cd, Pd, k, out=torch.empty_like(out), workspace=ws)  # eager work between
        torch.cuda.synchronize()


def test_decode_full_budget_is_full_attention():
    rng = np.random.default_rng(11)
    q, K, V, codes, P = _random_case(rng, 1, 4, 2, 2000, 64)
    out = bpc.decode_attention(q, K, V, torch.from_numpy(codes.view(np.int32)).to(DEV), torch.from_numpy(P).to(DEV),
                               2000)
    torch.cuda.synchronize()
    qb, Kb, Vb = bits(q), bits(K), bits(V)
    for h in range(2):
        full = oracle.full_attention(qb[0, 2 * h:2 * h + 2], Kb[0, h], Vb[0, h], 1 / np.sqrt(128))
        assert np.all(rel_err(out[0, 2 * h:2 * h + 2].cpu().numpy(), full) <= TOL)


def test_decode_shared_projection():
    rng = np.random.default_rng(12)
    q, K, V, codes, P = _random_case(rng, 2, 8, 2, 3000, 64)
    Ps = P[0, 0]
    _decode_and_compare(q, K, V, codes, Ps, 60, label="shared P")


def test_decode_zero_query():
    rng = np.random.default_rng(13)
    q, K, V, codes, P = _random_case(rng, 1, 4, 2, 1000, 32, qscale=0.0)
    _, idx = _decode_and_compare(q, K, V, codes, P, 20, label="zero query")
    assert idx.cpu().numpy()[0, 0].tolist() == list(range(20))  # all scores 0 -> lowest indices


def test_decode_deterministic(tiny):
    cfg, host, dev, builds = tiny
    P, codes, _ = bpc.build_hash(dev["K"], dev["G"])
    outs = [bpc.decode_attention(dev["q"], dev["K"], dev["V"], codes, P, cfg.k).clone() for _ in range(3)]
    torch.cuda.synchronize()
    assert all(torch.equal(outs[0], o) for o in outs[1:])


def test_decode_profiled_events(tiny):
    cfg, host, dev, builds = tiny
    P, codes, _ = bpc.build_hash(dev["K"], dev["G"])
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(bpc.DECODE_STAGES + 1)]
    out = bpc.decode_attention(dev["q"], dev["K"], dev["V"], codes, P, cfg.k, events=evs)
    ref = bpc.decode_attention(dev["q"], dev["K"], dev["V"], codes, P, cfg.k)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)
    times = [evs[i].elapsed_time(evs[i + 1]) for i in range(bpc.DECODE_STAGES)]
    assert all(t >= 0 for t in times)


def test_errors_raise():
    q = torch.zeros(1, 4, 128, dtype=torch.bfloat16, device=DEV)
    K = torch.zeros(1, 1, 10, 128, dtype=torch.bfloat16, device=DEV)
    codes = torch.zeros(1, 1, 10, 1, dtype=torch.int32, device=DEV)
    P = torch.zeros(1, 1, 32, 128, dtype=torch.float32, device=DEV)
    with pytest.raises(ValueError):  # the binding's own checks: k > N
        bpc.decode_attention(q, K, K, codes, P, 11)
    with pytest.raises(bpc.BPCError):  # the library's: a group of 3 query heads
        bpc.decode_attention(q[:, :3].contiguous(), K, K, codes, P, 4)
