"""Algorithm 2 on the matrix cores with certified signs (bpc_hash_keys_mm)
against the CPU oracle: codes and fragile counts bit-exact.

Besides random and workload keys, the inputs include keys built to put
decisions exactly at zero or close to it, zero and non-finite rows, and very
large and very small scales, so that the recomputation in fixed-order fp64
runs and its results are checked too.  The full-size heads of every workload
are checked in test_gpu_fullsize.py.
"""

import numpy as np
import pytest
import torch

import oracle
from workloads import config_by_name, make_layer

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2608_04405_amd as bpc
else:  # pragma: no cover - collected on CPU-only machines, never run
    bpc = None

DEV = "cuda"


def bits(t):
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def u32(t):
    return t.detach().cpu().contiguous().numpy().view(np.uint32)


def announce(msg):
    print(msg, flush=True)


def run_mm(K, P, N=None, codes_out=None):
    frag = torch.zeros(1, dtype=torch.int64, device=DEV)
    fall = torch.zeros(1, dtype=torch.int64, device=DEV)
    codes = bpc.hash_keys_mm(K, P, N=N, codes_out=codes_out, fragile=frag, fallbacks=fall)
    torch.cuda.synchronize()
    return codes, int(frag.item()), int(fall.item())


def check_against_oracle(K, P, shared, N, label):
    codes, frag, fall = run_mm(K, P, N=N)
    B, H = K.shape[:2]
    Kb = bits(K)
    nf = 0
    for b in range(B):
        for h in range(H):
            Ph = P.cpu().numpy() if shared else P[b, h].cpu().numpy()
            co, _, fo = oracle.hash_keys(Kb[b, h, :N], Ph)
            nf += fo
            got = u32(codes[b, h, :N])
            bad = np.nonzero(np.any(got != co, axis=1))[0]
            assert bad.size == 0, f"{label}: codes differ at keys {bad[:8].tolist()} of (b, h) = ({b}, {h})"
    assert frag == nf, f"{label}: fragile count {frag} against {nf}"
    announce(f"{label}: bit-exact, {frag} fragile, {fall} decisions recomputed of {B * H * N * P.shape[-2]}")
    return fall


@pytest.mark.parametrize("L", [32, 64, 128])
@pytest.mark.parametrize("shared", [False, True])
def test_mm_random(L, shared):
    rng = np.random.default_rng(100 + L)
    B, H, N = 2, 2, 1777  # several wavefronts and workgroups, a ragged tail
    K = torch.from_numpy(rng.standard_normal((B, H, N, 128)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    shape = (L, 128) if shared else (B, H, L, 128)
    P = torch.from_numpy((0.3 * rng.standard_normal(shape)).astype(np.float32)).to(DEV)
    check_against_oracle(K, P, shared, N, f"random L={L} shared={shared}")


@pytest.mark.parametrize("name,N", [("tiny_mha_4k", 4096), ("llama8b_32k", 6000), ("million_1m", 3000)])
def test_mm_workload_keys_with_built_projection(name, N):
    """Workload keys with the projection Algorithm 1 builds from them (the
    oracle's own build), the distribution the prefill sees."""
    cfg = config_by_name(name).replace(N=N, B=1)
    d = make_layer(cfg, device="cpu", heads=[(0, 0), (0, 1)])
    Kb = bits(d["K"][0, :2])
    Ps = np.stack([oracle.build_binary_pcs(Kb[h], d["G"].numpy())[0] for h in range(2)])
    K = d["K"][:, :2].contiguous().to(DEV)
    P = torch.from_numpy(Ps[None]).to(DEV)
    check_against_oracle(K, P, False, N, f"{name} N={N}")


def test_mm_strided_cache_and_codes():
    """K rows with padding and a cache longer than N; codes written into a
    larger buffer whose rows past N stay untouched."""
    rng = np.random.default_rng(7)
    B, H, Ncap, N, L = 2, 3, 1200, 1029, 64
    big = torch.from_numpy(rng.standard_normal((B, H, Ncap, 136)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    K = big[..., :128]
    P = torch.from_numpy((0.2 * rng.standard_normal((B, H, L, 128))).astype(np.float32)).to(DEV)
    codes = torch.full((B, H, Ncap, L // 32), -1, dtype=torch.int32, device=DEV)
    run_mm(K, P, N=N, codes_out=codes)
    Kb = bits(K)
    for b in range(B):
        for h in range(H):
            co, _, _ = oracle.hash_keys(Kb[b, h, :N], P[b, h].cpu().numpy())
            assert np.array_equal(u32(codes[b, h, :N]), co)
    assert bool((codes[:, :, N:] == -1).all())


def _exact_decisions_inputs(L, rng):
    """P with bf16-representable entries on disjoint supports plus a dense
    tail, and keys that are exact signed sums of its rows (so residuals reach
    exactly zero and later decisions are exactly zero), keys orthogonal to the
    first row, zero rows, and keys a hair away from such cases."""
    P = np.zeros((L, 128), np.float32)
    for i in range(L):
        d0 = (i * 3) % 128
        P[i, d0] = np.float32(2.0 ** -(i % 5))
        P[i, (d0 + 1) % 128] = np.float32(-0.5)
    P[L // 2:] += np.float32(1.0 / 64) * np.sign(rng.standard_normal((L - L // 2, 128))).astype(np.float32)
    rows = []
    for n in range(400):
        s = np.where(rng.random(L) < 0.5, 1.0, -1.0)
        m = 1 + n % L
        k = (s[:m, None] * P[:m].astype(np.float64)).sum(0)  # exact sum of m signed rows
        if np.array_equal(k.astype(np.float32).astype(np.float64), k) and \
                np.array_equal(torch.from_numpy(k.astype(np.float32)).to(torch.bfloat16).double().numpy(), k):
            rows.append(k)  # kept only where bf16 holds it exactly
        if len(rows) == 96:
            break
    n_exact = len(rows)
    for n in range(64):
        k = rng.standard_normal(128)
        k[0] = 0.0  # orthogonal to P[0] (support {0, 1}) only if k[1] = 0 too
        k[1] = 0.0
        rows.append(k)
    rows += [np.zeros(128)] * 8
    for n in range(64):
        k = rows[n % n_exact].copy()
        k[(5 * n) % 128] += 2.0 ** -12  # a small step off an exact case
        rows.append(k)
    Kf = np.asarray(rows, np.float64)
    return Kf, P, n_exact


@pytest.mark.parametrize("L", [32, 64, 128])
def test_mm_exact_zero_and_near_zero_decisions(L):
    rng = np.random.default_rng(11 + L)
    Kf, P, n_exact = _exact_decisions_inputs(L, rng)
    assert n_exact >= 16
    K = torch.from_numpy(Kf.astype(np.float32)).to(torch.bfloat16)
    assert np.array_equal(K[:n_exact].double().numpy(), Kf[:n_exact])
    K = K[None, None].contiguous().to(DEV)
    fall = check_against_oracle(K, torch.from_numpy(P).to(DEV), True, K.shape[2], f"exact cases L={L}")
    assert fall > 0  # the recomputation ran and its decisions were checked


def test_mm_extreme_scales_and_non_finite_rows():
    rng = np.random.default_rng(5)
    L = 64
    base = rng.standard_normal((200, 128))
    Kf = np.concatenate([base * 1e30, base * 1e-30, base * 1e-38, base[:4] * np.inf, base[:4]])
    Kf[-4:, 3] = np.nan
    K = torch.from_numpy(Kf.astype(np.float32)).to(torch.bfloat16)[None, None].contiguous().to(DEV)
    P = torch.from_numpy((0.3 * rng.standard_normal((L, 128))).astype(np.float32)).to(DEV)
    with np.errstate(all="ignore"):
        check_against_oracle(K, P, True, K.shape[2], "extreme scales and non-finite rows")


def test_mm_large_and_tiny_projection():
    rng = np.random.default_rng(9)
    K = torch.from_numpy(rng.standard_normal((1, 2, 500, 128)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    P = np.stack([1e18 * rng.standard_normal((64, 128)), 1e-18 * rng.standard_normal((64, 128))])
    P = torch.from_numpy(P.astype(np.float32)[None]).to(DEV)
    check_against_oracle(K, P, False, 500, "projection scaled by 1e18 and 1e-18")


def test_mm_matches_canonical_kernel_on_a_large_batch():
    """Consistency over many keys: the matrix-core codes equal those of the
    fixed-order fp64 kernel (itself checked against the oracle) on one
    workload layer of 8 x 8 heads x 65536 keys; the fragile counts agree."""
    cfg = config_by_name("stack32_b8_64k")
    d = make_layer(cfg, device=DEV)
    P, _, _ = bpc.build_hash(d["K"], d["G"].to(DEV))
    f1 = torch.zeros(1, dtype=torch.int64, device=DEV)
    c1, _ = bpc.hash_keys(d["K"], P, fragile=f1)
    c2, f2, fall = run_mm(d["K"], P)
    assert torch.equal(c1, c2)
    assert int(f1.item()) == f2
    announce(f"stack layer 0: {cfg.B * cfg.Hkv * cfg.N} keys equal, {f2} fragile, {fall} recomputed")
