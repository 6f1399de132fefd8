"""The error-aware safeguard on the GPU (through the C ABI) against the oracle.

* select_hard: the hard-to-hash set (top-m reconstruction errors, equal
  errors to the lower index) from the same float32 errors on both sides,
  bit-exact; random errors with many ties, negative and zero values, ragged
  sizes, and the errors of a real GPU build.
* decode with the safeguard: S_hash (idx_out), the added flags and the
  output over S_hash u S_err against oracle.decode_head_eas: indices and
  flags bit-exact, output within 2e-3 per row.  Cases cover the tiny and
  8B-shaped workloads with the paper's 10 % split of the budget, hard sets
  disjoint from and inside S_hash, a hard set large enough that the row list
  leaves LDS, several slices, and the exact two-round threshold path.
"""

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


# ------------------------------------------------------------------ select_hard

@pytest.mark.parametrize("B,H,N,m,pool", [
    (1, 1, 1, 1, None),
    (2, 3, 1000, 37, 5),          # many ties
    (1, 2, 16385, 16385, None),   # m = N
    (1, 1, 20000, 1, 3),
    (2, 2, 131073, 263, None),
    (1, 1, 5000, 700, 7),
])
def test_select_hard_parity(B, H, N, m, pool):
    announce(f"[select_hard] B={B} H={H} N={N} m={m} pool={pool}")
    rng = np.random.default_rng(N + m)
    if pool is None:
        err = np.abs(rng.standard_normal((B, H, N))).astype(np.float32) * 10
    else:
        vals = np.array([0.0, -0.0, 1.5, 2.25, -3.0, 8.0, 8.0][:pool], np.float32)
        err = rng.choice(vals, size=(B, H, N))
    e = torch.from_numpy(err).to(DEV)
    serr = bpc.select_hard(e, m)
    torch.cuda.synchronize()
    got = serr.cpu().numpy()
    for b in range(B):
        for h in range(H):
            assert np.array_equal(got[b, h], oracle.select_hard(err[b, h], m)), f"differs at {(b, h)}"


def test_select_hard_strided_from_build():
    """The reconstruction errors of a real build (the oracle's Algorithm 1
    on the tiny workload, rounded to float32 as the prefill kernels store
    them) in a buffer with a row stride past N."""
    cfg = CONFIGS[0]
    d = make_layer(cfg, device="cpu")
    Kb, Gn = bits(d["K"]), d["G"].numpy()
    eo = np.stack([oracle.build_binary_pcs(Kb[0, h], Gn)[2] for h in range(cfg.Hkv)]).astype(np.float32)
    Ncap = cfg.N + 40
    err = torch.full((cfg.B, cfg.Hkv, Ncap), -7.0, device=DEV)  # the tail past N must be ignored
    err[0, :, :cfg.N] = torch.from_numpy(eo).to(DEV)
    _, m = oracle.eas_budget(cfg.k)
    serr = bpc.select_hard(err, m, N=cfg.N)
    torch.cuda.synchronize()
    for h in range(cfg.Hkv):
        assert np.array_equal(serr[0, h].cpu().numpy(), oracle.select_hard(eo[h], m))


# ------------------------------------------------------------------ decode with the safeguard

def _eas_compare(q, K, V, codes_np, P_np, k, serr_np, N=None, label="", heads=None):
    B, Hq, D = q.shape
    Hkv = K.shape[1]
    Gq = Hq // Hkv
    N = K.shape[2] if N is None else N
    m = serr_np.shape[-1]
    sm = 1.0 / np.sqrt(D)
    codes = torch.from_numpy(np.ascontiguousarray(codes_np).view(np.int32)).to(DEV)
    P = torch.from_numpy(np.ascontiguousarray(P_np)).to(DEV)
    serr = torch.from_numpy(np.ascontiguousarray(serr_np).astype(np.int32)).to(DEV)
    idx = torch.full((B, Hkv, k), -1, dtype=torch.int32, device=DEV)
    added = torch.full((B, Hkv, m), -1, dtype=torch.int32, device=DEV)
    out = bpc.decode_attention(q, K, V, codes, P, k, sm, N=N, idx_out=idx, serr=serr, added_out=added)
    torch.cuda.synchronize()
    qb, Kb, Vb = bits(q), bits(K), bits(V)
    worst = 0.0
    for b, h in (heads or [(b, h) for b in range(B) for h in range(Hkv)]):
        ref = oracle.decode_head_eas(qb[b, h * Gq:(h + 1) * Gq], Kb[b, h, :N], Vb[b, h, :N], codes_np[b, h, :N],
                                     P_np[b, h], k, serr_np[b, h], sm)
        assert np.array_equal(idx[b, h].cpu().numpy(), ref["idx"]), f"{label}: S_hash differs at {(b, h)}"
        assert np.array_equal(added[b, h].cpu().numpy(), ref["added"]), f"{label}: added flags differ at {(b, h)}"
        e = rel_err(out[b, h * Gq:(h + 1) * Gq].cpu().numpy(), ref["out"])
        worst = max(worst, float(e.max()))
        assert np.all(e <= TOL), f"{label}: output error {e.max():.3g} at {(b, h)}"
    announce(f"{label}: max relative output error {worst:.3g}")
    return out


def _gpu_pipeline_vs_oracle(cfg, heads, label):
    """GPU: Algorithm 1, select_hard on its float32 errors, decode over
    S_hash u S_err.  Oracle: its own build of the checked heads, its
    selection from its own errors (rounded to float32 as the kernels store
    them), its decode.  The GPU's P, codes and hard sets are checked equal
    to the oracle's first; the checked heads then hold the oracle's values."""
    d = make_layer(cfg, device=DEV)
    P, codes, err = bpc.build_hash(d["K"], d["G"].to(DEV), err_out=torch.empty(cfg.B, cfg.Hkv, cfg.N, device=DEV))
    k_hash, m = oracle.eas_budget(cfg.k)
    serr = bpc.select_hard(err, m)
    torch.cuda.synchronize()
    Pn, cn, errs = oracle_build_of(P, codes, d["K"], d["G"], heads)
    sn = serr.cpu().numpy().astype(np.int64)
    for (b, h), eo in errs.items():
        so = oracle.select_hard(eo.astype(np.float32), m)
        assert np.array_equal(sn[b, h], so), f"{label}: hard set differs at {(b, h)}"
        sn[b, h] = so
    _eas_compare(d["q"], d["K"], d["V"], cn, Pn, k_hash, sn, label=label, heads=heads)


def test_decode_eas_tiny_budget_split():
    """The tiny workload with the paper's split: 10 % of the budget for the
    hard set, chosen on the GPU from the GPU build's errors."""
    cfg = CONFIGS[0]
    announce(f"[eas tiny] {cfg}")
    _gpu_pipeline_vs_oracle(cfg, [(0, h) for h in range(cfg.Hkv)], "eas tiny")


def test_decode_eas_llama8b_shape():
    cfg = CONFIGS[1]
    announce(f"[eas llama8b] {cfg}")
    _gpu_pipeline_vs_oracle(cfg, [(0, 0), (0, 5)], "eas llama8b")


def _random_case(rng, B, Hq, Hkv, N, L):
    q = torch.from_numpy(rng.standard_normal((B, Hq, 128)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    K = torch.from_numpy(rng.standard_normal((B, Hkv, N, 128)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    V = torch.from_numpy(rng.standard_normal((B, Hkv, N, 128)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    codes = rng.integers(0, 1 << 32, size=(B, Hkv, N, L // 32), dtype=np.uint64).astype(np.uint32)
    P = (0.5 * rng.standard_normal((B, Hkv, L, 128))).astype(np.float32)
    return q, K, V, codes, P


@pytest.mark.parametrize("case", [
    dict(B=2, Hq=8, Hkv=2, N=5000, L=64, k=90, m=10, kind="random"),
    dict(B=1, Hq=4, Hkv=1, N=70000, L=64, k=1260, m=140, kind="random"),    # five slices
    dict(B=1, Hq=4, Hkv=2, N=40000, L=32, k=300, m=2500, kind="random"),    # rows leave LDS
    dict(B=1, Hq=2, Hkv=1, N=3000, L=64, k=40, m=25, kind="disjoint"),
    dict(B=1, Hq=2, Hkv=1, N=3000, L=64, k=40, m=25, kind="inside"),
    dict(B=1, Hq=4, Hkv=1, N=1100000, L=32, k=9000, m=1000, kind="random"),  # 68 slices: two-round threshold
])
def test_decode_eas_cases(case):
    announce(f"[eas case] {case}")
    rng = np.random.default_rng(case["N"] + case["m"])
    B, Hkv, N, k, m = case["B"], case["Hkv"], case["N"], case["k"], case["m"]
    q, K, V, codes, P = _random_case(rng, B, case["Hq"], Hkv, N, case["L"])
    serr = np.empty((B, Hkv, m), np.int64)
    for b in range(B):
        for h in range(Hkv):
            if case["kind"] == "random":
                serr[b, h] = np.sort(rng.choice(N, m, replace=False))
            else:
                ref = oracle.decode_head(bits(q)[b, h * (case["Hq"] // Hkv):(h + 1) * (case["Hq"] // Hkv)],
                                         bits(K)[b, h], bits(V)[b, h], codes[b, h], P[b, h], k, 1.0)
                pool = ref["idx"] if case["kind"] == "inside" else np.setdiff1d(np.arange(N), ref["idx"])
                serr[b, h] = np.sort(rng.choice(pool, m, replace=False))
    _eas_compare(q, K, V, codes, P, k, serr, label=f"eas {case['kind']} N={N} m={m}")


def test_decode_eas_window_miss():
    """The planted distance-0 keys of the window-miss decode test, with a
    hard set: the exact two-round threshold and re-scored selection run."""
    rng = np.random.default_rng(11)
    N, L, k = 32768, 64, 100
    q, K, V, codes, P = _random_case(rng, 1, 4, 1, N, L)
    planes = oracle.quantize_query(bits(q)[0], P[0, 0])["qcode"]
    near = np.r_[0:60, 16384:16444]
    codes[0, 0, near] = planes[0]
    serr = np.sort(np.r_[near[:5], rng.choice(np.arange(20000, 30000), 20, replace=False)])[None, None]
    _eas_compare(q, K, V, codes, P, k, serr, label="eas window miss")


def test_decode_eas_out_of_range_entries_ignored():
    """Entries of S_err outside [0, N) lie in no slice: they are ignored and
    their added flags are 0 (the rest as the oracle on the in-range set)."""
    rng = np.random.default_rng(23)
    B, Hq, Hkv, N, L, k = 1, 4, 2, 20000, 64, 200
    q, K, V, codes, P = _random_case(rng, B, Hq, Hkv, N, L)
    inside = np.stack([np.sort(rng.choice(N, 12, replace=False)) for _ in range(Hkv)])[None]
    serr_np = np.concatenate([np.full((B, Hkv, 2), -1), inside, np.full((B, Hkv, 1), N),
                              np.full((B, Hkv, 1), N + 1000)], axis=-1)
    m = serr_np.shape[-1]
    codes_t = torch.from_numpy(np.ascontiguousarray(codes).view(np.int32)).to(DEV)
    serr = torch.from_numpy(serr_np.astype(np.int32)).to(DEV)
    idx = torch.full((B, Hkv, k), -1, dtype=torch.int32, device=DEV)
    added = torch.full((B, Hkv, m), 7, dtype=torch.int32, device=DEV)
    sm = 1.0 / np.sqrt(128)
    out = bpc.decode_attention(q, K, V, codes_t, torch.from_numpy(P).to(DEV), k, sm, idx_out=idx, serr=serr,
                               added_out=added)
    torch.cuda.synchronize()
    G = Hq // Hkv
    for h in range(Hkv):
        ref = oracle.decode_head_eas(bits(q)[0, h * G:(h + 1) * G], bits(K)[0, h], bits(V)[0, h], codes[0, h],
                                     P[0, h], k, inside[0, h], sm)
        got = added[0, h].cpu().numpy()
        assert np.array_equal(got[2:-2], ref["added"]) and np.all(got[:2] == 0) and np.all(got[-2:] == 0), got
        assert np.array_equal(idx[0, h].cpu().numpy(), ref["idx"])
        e = rel_err(out[0, h * G:(h + 1) * G].cpu().numpy(), ref["out"])
        assert np.all(e <= TOL), e
