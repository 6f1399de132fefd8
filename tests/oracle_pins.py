"""Pins of the CPU oracle against facts that do not come from the oracle.

Each pin is a function of the oracle module `o`, so the same checks run on
the real oracle (test_oracle_pins.py) and on deliberately broken copies of
it (test_oracle_mutants.py), which shows that a plausible slip in the oracle
(a dropped term, a wrong sign, index or operand) fails at least one pin.

The facts used: the hand-worked example in golden/worked_example.json,
closed forms (rank-1 keys, disjoint-support projections, uniform
magnitudes), exact rational re-evaluation with `fractions`, algebraic
identities of the greedy decomposition (the optimal v for a fixed u, see the
Appendix "Procedure Overview"), symmetries, brute-force sorting, and
library routines (torch's bf16 conversion and scaled-dot-product attention).
"""

from __future__ import annotations

import json
import os
from fractions import Fraction

import numpy as np
import torch

from _helpers import bf16_values, fp32_ulp, popcount32, random_bf16, to_bf16_bits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_example.json")


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def _pad(rows, D):
    a = np.zeros((len(rows), D), dtype=np.float64)
    r = np.asarray(rows, dtype=np.float64)
    a[:, : r.shape[1]] = r
    return a


# ---------------------------------------------------------------- formats

def pin_bf16_widening(o):
    rng = np.random.default_rng(1)
    bits = rng.integers(0, 1 << 16, size=4096, dtype=np.uint64).astype(np.uint16)
    bits = bits[(bits & 0x7F80) != 0x7F80]  # drop inf / nan
    assert np.array_equal(o.bf16_bits_to_f64(bits), bf16_values(bits))


def pin_canonical_dot_order(o):
    # integer data: no rounding, so the result is the exact dot product
    rng = np.random.default_rng(2)
    X = rng.integers(-50, 50, size=(7, 128)).astype(np.float64)
    w = rng.integers(-50, 50, size=128).astype(np.float64)
    assert np.array_equal(o.canonical_dot(X, w), (X.astype(np.int64) @ w.astype(np.int64)).astype(np.float64))
    # the order: 4 blocks summed ascending, combined as (b0+b1)+(b2+b3)
    big = 1e16
    X = np.array([[big, 1.0, -big, 1.0]])
    # blocks of one element: (1e16 + 1) + (-1e16 + 1) = 1e16 + (-1e16) = 0
    assert o.canonical_dot(X, np.ones(4))[0] == 0.0
    X = np.zeros((1, 8))
    X[0, :2] = [big, 1.0]  # block 0 = (0 + 1e16) + 1 = 1e16
    X[0, 2:4] = [1.0, 1.0]  # block 1 = 2
    assert o.canonical_dot(X, np.ones(8))[0] == big + 2.0


def pin_pairwise_tree(o):
    big = 1e16
    # ((1e16 + 1) + (1 + 1)) = 1e16 + 2 ; a sequential sum would give 1e16
    assert o.pairwise_tree_sum(np.array([[big], [1.0], [1.0], [1.0]]))[0] == big + 2.0
    # odd count: ((a + b) + c) with the last element carried
    x = np.array([[1.0], [big], [-big]])
    assert o.pairwise_tree_sum(x)[0] == (1.0 + big) + (-big)
    # five elements: ((x0+x1)+(x2+x3)) + x4
    x = np.array([[big], [1.0], [1.0], [1.0], [1.0]])
    assert o.pairwise_tree_sum(x)[0] == ((big + 1.0) + (1.0 + 1.0)) + 1.0
    rng = np.random.default_rng(3)
    ints = rng.integers(-1000, 1000, size=(37, 5)).astype(np.float64)
    assert np.array_equal(o.pairwise_tree_sum(ints), ints.sum(axis=0))


def pin_pack_bits(o):
    H = -np.ones((3, 64), dtype=np.int8)
    H[0, 0] = 1
    H[1, 33] = 1
    H[2, :] = 1
    c = o.pack_codes(H)
    assert c.dtype == np.uint32 and c.shape == (3, 2)
    assert c.tolist() == [[1, 0], [0, 2], [0xFFFFFFFF, 0xFFFFFFFF]]
    rng = np.random.default_rng(4)
    H = np.where(rng.random((9, 128)) < 0.5, 1, -1).astype(np.int8)
    assert np.array_equal(o.unpack_codes(o.pack_codes(H), 128), H)


def pin_budget(o):
    # the budgets of the workloads: 2 % of 4096, 32768, 65536, 131072; 1 % of 2^20
    assert [o.budget_keys(n, 2, 100) for n in (4096, 32768, 65536, 131072)] == [82, 656, 1311, 2622]
    assert o.budget_keys(1 << 20, 1, 100) == 10486
    assert o.budget_keys(100, 2, 100) == 2


# ---------------------------------------------------------------- Algorithm 1

def pin_alg1_worked_example(o):
    g = _golden()
    K = to_bf16_bits(g["K_small"])
    P, codes, err, fr, tr = o.build_binary_pcs(K, np.asarray(g["G_small"], np.float32), trace=True)
    assert np.array_equal(P, np.asarray(g["P_small"], np.float32))
    assert np.array_equal(tr["H"], np.asarray(g["H_small"]))
    assert np.all(err == 0.0) and fr == 0
    # padded to D = 128, L = 32
    L = g["L_padded"]
    Kp = to_bf16_bits(_pad(g["K_small"], 128))
    rng = np.random.default_rng(5)
    Gp = rng.standard_normal((L, 128)).astype(np.float32)
    Gp[:2] = _pad(g["G_small"], 128).astype(np.float32)
    P, codes, err, fr = o.build_binary_pcs(Kp, Gp)
    assert codes[:, 0].tolist() == g["codes_padded"]
    assert np.array_equal(P[:2, :4], np.asarray(g["P_small"], np.float32)) and np.all(P[2:] == 0) and np.all(P[:, 4:] == 0)
    assert fr == g["fragile_padded"]


def pin_decode_worked_example(o):
    # the decode step of the hand-worked example: query planes, scores
    # [254, 0, 0, -254], the top-2 with its tie at 0 going to key 1, and the
    # two-key softmax output (closed form in the fixture)
    g = _golden()
    L = g["L_padded"]
    K = to_bf16_bits(_pad(g["K_small"], 128))
    V = to_bf16_bits(_pad(g["V_small"], 128))
    q = to_bf16_bits(_pad([g["query"]], 128))
    P = np.zeros((L, 128), np.float32)
    P[:2, :4] = np.asarray(g["P_small"], np.float32)
    codes = np.asarray(g["codes_padded"], np.uint32)[:, None]
    r = o.decode_head(q, K, V, codes, P, g["k"], g["sm_scale"])
    assert r["p"][:2].tolist() == g["p_padded_first2"] and np.all(r["p"][2:] == 0) and r["T"] == g["T"]
    assert r["scores"].tolist() == g["scores"]
    assert r["idx"].tolist() == g["topk"]
    np.testing.assert_allclose(r["out"][0, :4], g["out_first4"], rtol=1e-14, atol=1e-15)
    assert np.all(r["out"][0, 4:] == 0)


def pin_alg1_rank1(o):
    rng = np.random.default_rng(6)
    N, D, L = 300, 128, 32
    h0 = np.where(rng.random(N) < 0.5, 1.0, -1.0)
    p0 = bf16_values(random_bf16(rng, D))
    K = to_bf16_bits(np.outer(h0, p0))
    G = rng.standard_normal((L, D)).astype(np.float32)
    P, codes, err, fr, tr = o.build_binary_pcs(K, G, trace=True)
    s = 1.0 if float(np.dot(p0, G[0].astype(np.float64))) >= 0 else -1.0
    assert np.array_equal(P[0].astype(np.float64), s * p0)
    assert np.array_equal(tr["H"][:, 0], (s * h0).astype(np.int8))
    assert np.all(tr["H"][:, 1:] == 1) and np.all(P[1:] == 0)
    assert np.all(tr["R"] == 0) and np.all(err == 0)


def pin_alg1_zero_keys(o):
    N, D, L = 50, 128, 32
    K = np.zeros((N, D), dtype=np.uint16)
    G = np.random.default_rng(7).standard_normal((L, D)).astype(np.float32)
    P, codes, err, fr = o.build_binary_pcs(K, G)
    assert np.all(P == 0) and np.all(codes == 0xFFFFFFFF) and fr == N * L and np.all(err == 0)


def _lowrank_keys(rng, N, D, rank=4):
    A = rng.standard_normal((rank, D))
    Z = rng.standard_normal((N, rank))
    return to_bf16_bits(Z @ A + 0.1 * rng.standard_normal((N, D)))


def pin_alg1_energy_identity(o):
    # For the closed-form v = u^T R / N and the rounded P = v + delta:
    # ||R - u P^T||^2 = ||R||^2 - N ||v||^2 + N ||P - v||^2  (exact algebra),
    # and u^T R_next = N (v - P).
    rng = np.random.default_rng(8)
    N, D, L = 257, 16, 12
    K = _lowrank_keys(rng, N, D)
    G = rng.standard_normal((L, D)).astype(np.float32)
    P, codes, err, fr, tr = o.build_binary_pcs(K, G, trace=True)
    f2 = tr["R_fro2"]
    for i in range(L):
        v = tr["v"][i]
        Pi = P[i].astype(np.float64)
        pred = f2[i] - N * np.dot(v, v) + N * np.dot(Pi - v, Pi - v)
        assert abs(f2[i + 1] - pred) <= 1e-11 * f2[0], (i, f2[i + 1], pred)
        assert f2[i + 1] <= f2[i] * (1 + 1e-12)  # Fig. 3 (left): the norm never grows
    # u_L^T R_L = N (v_L - P_L) for the last iteration
    u = tr["u"][-1]
    lhs = u @ tr["R"]
    assert np.allclose(lhs, N * (tr["v"][-1] - P[-1].astype(np.float64)), atol=1e-9 * np.sqrt(f2[0]))


def pin_alg1_reconstruction(o):
    rng = np.random.default_rng(9)
    N, D, L = 200, 32, 20
    K = _lowrank_keys(rng, N, D)
    G = rng.standard_normal((L, D)).astype(np.float32)
    P, codes, err, fr, tr = o.build_binary_pcs(K, G, trace=True)
    Kd = bf16_values(K)
    recon = Kd - tr["H"].astype(np.float64) @ P.astype(np.float64)
    assert np.allclose(recon, tr["R"], rtol=0, atol=1e-12 * np.abs(Kd).max())
    assert np.allclose(err, np.linalg.norm(recon, axis=1), rtol=1e-12, atol=1e-12)


def _exact_alg1(Kv, G):
    N, D = Kv.shape
    R = [[Fraction(float(x)) for x in row] for row in Kv]
    P = np.zeros(G.shape, np.float32)
    H = np.zeros((N, G.shape[0]), np.int8)
    margin = np.inf
    for i in range(G.shape[0]):
        g = [Fraction(float(x)) for x in G[i]]
        a = [sum(r * gg for r, gg in zip(row, g)) for row in R]
        u = [1 if ai >= 0 else -1 for ai in a]
        scale = max(1e-300, max(abs(float(x)) for row in R for x in row))
        margin = min(margin, min(abs(float(ai)) for ai in a) / scale)
        v = [sum(u[j] * R[j][d] for j in range(N)) / N for d in range(D)]
        P[i] = np.array([float(x) for x in v], dtype=np.float64).astype(np.float32)
        R = [[R[j][d] - u[j] * Fraction(float(P[i, d])) for d in range(D)] for j in range(N)]
        H[:, i] = u
    return P, H, margin


def pin_alg1_exact_rational(o):
    rng = np.random.default_rng(10)
    for trial in range(3):
        N, D, L = 12, 8, 6
        K = _lowrank_keys(rng, N, D, rank=3)
        G = rng.standard_normal((L, D)).astype(np.float32)
        Pe, He, margin = _exact_alg1(bf16_values(K), G)
        assert margin > 1e-9, "test input too close to a sign boundary"
        P, codes, err, fr, tr = o.build_binary_pcs(K, G, trace=True)
        assert np.array_equal(tr["H"], He)
        assert np.all(np.abs(P.astype(np.float64) - Pe.astype(np.float64)) <= 2 * fp32_ulp(Pe) + 1e-30)


def pin_alg1_symmetries(o):
    rng = np.random.default_rng(11)
    N, D, L = 150, 128, 32
    K = _lowrank_keys(rng, N, D)
    G = rng.standard_normal((L, D)).astype(np.float32)
    P, codes, err, fr, tr = o.build_binary_pcs(K, G, trace=True)
    assert fr == 0
    # negating every key flips every code bit and leaves P unchanged
    Kneg = K ^ np.uint16(0x8000)
    P2, codes2, err2, fr2 = o.build_binary_pcs(Kneg, G)
    assert np.array_equal(P2, P) and np.array_equal(codes2, ~codes) and np.array_equal(err2, err)
    # doubling every key (exact in bf16) doubles P and keeps the codes
    K2 = to_bf16_bits(2.0 * bf16_values(K))
    P3, codes3, err3, fr3 = o.build_binary_pcs(K2, G)
    assert np.array_equal(P3, 2 * P) and np.array_equal(codes3, codes)


def pin_alg1_first_bit(o):
    # bit 0 is sign(K g0) and P[0] is the mean of u_j k_j (exact rationals)
    rng = np.random.default_rng(12)
    N, D = 40, 128
    K = _lowrank_keys(rng, N, D)
    G = rng.standard_normal((32, D)).astype(np.float32)
    P, codes, err, fr, tr = o.build_binary_pcs(K, G, trace=True)
    Kv = bf16_values(K)
    g = [Fraction(float(x)) for x in G[0]]
    u = []
    for row in Kv:
        a = sum(Fraction(float(x)) * gg for x, gg in zip(row, g))
        u.append(1 if a >= 0 else -1)
    assert tr["H"][:, 0].tolist() == u
    mean = [float(sum(u[j] * Fraction(float(Kv[j, d])) for j in range(N)) / N) for d in range(D)]
    mean = np.asarray(mean).astype(np.float32)
    assert np.all(np.abs(P[0].astype(np.float64) - mean) <= fp32_ulp(mean) + 1e-30)


# ---------------------------------------------------------------- Algorithm 2

def pin_alg2_worked_example(o):
    g = _golden()
    Kp = to_bf16_bits(_pad(g["K_small"], 128))
    P = np.zeros((32, 128), np.float32)
    P[:2, :4] = np.asarray(g["P_small"], np.float32)
    codes, err, fr = o.hash_keys(Kp, P)
    assert codes[:, 0].tolist() == g["codes_padded"] and np.all(err == 0)
    assert fr == g["fragile_padded"]


def pin_alg2_disjoint_support(o):
    # rows of P with disjoint supports: the iterative residual never changes
    # the coordinates other rows look at, so h = sign(k P^T) exactly
    rng = np.random.default_rng(13)
    N, D, L = 500, 128, 64
    K = random_bf16(rng, (N, D))
    P = np.zeros((L, D), np.float32)
    perm = rng.permutation(D)
    for i in range(L):
        P[i, perm[2 * i: 2 * i + 2]] = rng.standard_normal(2).astype(np.float32)
    codes, err, fr, H = o.hash_keys(K, P, return_H=True)
    Kv = bf16_values(K)
    expect = np.where(Kv @ P.astype(np.float64).T >= 0, 1, -1)
    assert np.array_equal(H, expect)


def pin_alg2_reproduces_rank1(o):
    rng = np.random.default_rng(14)
    N, D, L = 200, 128, 32
    h0 = np.where(rng.random(N) < 0.5, 1.0, -1.0)
    p0 = bf16_values(random_bf16(rng, D))
    K = to_bf16_bits(np.outer(h0, p0))
    G = rng.standard_normal((L, D)).astype(np.float32)
    P, codes1, err1, fr1 = o.build_binary_pcs(K, G)
    codes2, err2, fr2 = o.hash_keys(K, P)
    assert np.array_equal(codes1, codes2) and np.all(err2 == 0)


def pin_alg2_reconstruction(o):
    rng = np.random.default_rng(15)
    N, D, L = 100, 128, 64
    K = random_bf16(rng, (N, D))
    P = (rng.standard_normal((L, D)) * 0.3).astype(np.float32)
    codes, err, fr, H = o.hash_keys(K, P, return_H=True)
    r = bf16_values(K) - H.astype(np.float64) @ P.astype(np.float64)
    assert np.allclose(err, np.linalg.norm(r, axis=1), rtol=1e-10, atol=1e-10)


def pin_alg2_exact_rational(o):
    rng = np.random.default_rng(16)
    N, D, L = 30, 8, 8
    K = random_bf16(rng, (N, D))
    P = (rng.standard_normal((L, D)) * 0.4).astype(np.float32)
    codes, err, fr, H = o.hash_keys(K, P, return_H=True)
    Pf = [[Fraction(float(x)) for x in row] for row in P]
    for j in range(N):
        r = [Fraction(float(x)) for x in bf16_values(K[j])]
        for i in range(L):
            a = sum(x * y for x, y in zip(r, Pf[i]))
            assert abs(float(a)) > 1e-12
            u = 1 if a >= 0 else -1
            assert H[j, i] == u, (j, i)
            r = [x - u * y for x, y in zip(r, Pf[i])]


def pin_alg2_sign_flip(o):
    rng = np.random.default_rng(17)
    K = random_bf16(rng, (300, 128))
    P = (rng.standard_normal((64, 128)) * 0.2).astype(np.float32)
    c1, e1, f1 = o.hash_keys(K, P)
    c2, e2, f2 = o.hash_keys(K ^ np.uint16(0x8000), P)
    assert f1 == 0 and np.array_equal(c2, ~c1) and np.array_equal(e1, e2)


# ---------------------------------------------------------------- query

def pin_quantize_properties(o):
    rng = np.random.default_rng(18)
    for Gq, L in ((1, 32), (4, 64), (8, 128)):
        q = random_bf16(rng, (Gq, 128))
        P = (rng.standard_normal((L, 128)) * 0.5).astype(np.float32)
        r = o.quantize_query(q, P)
        p, x = r["p"], r["x"]
        m = np.abs(x).max()
        y = x * 127.0 / m
        assert np.all(np.abs(y - p) <= 0.5 + 1e-12)
        assert np.abs(p).max() == 127 and np.all(np.abs(p) <= 127)
        nz = p != 0
        assert np.all(np.sign(p[nz]) == np.sign(x[nz]))
        assert r["T"] == int(np.abs(p).sum())
        # bit planes: plane 0 signs (1 <=> p >= 0), plane 1+j = bit j of |p|
        words = r["qcode"]
        assert words.shape == (8, L // 32)
        bits = ((words[:, :, None] >> np.arange(32, dtype=np.uint32)) & 1).reshape(8, L)
        mag = sum(bits[1 + j].astype(np.int64) << j for j in range(7))
        assert np.array_equal(np.where(bits[0] == 1, mag, -mag), p)
        assert np.all(bits[0][p > 0] == 1) and np.all(bits[0][p < 0] == 0)
        assert np.array_equal(o.unpack_query_planes(words, L), p)


def pin_quantize_exact(o):
    # exact rational projection, scaling and half-away rounding
    rng = np.random.default_rng(19)
    q = random_bf16(rng, (3, 128))
    P = (rng.standard_normal((32, 128)) * 0.5).astype(np.float32)
    r = o.quantize_query(q, P)
    qv = bf16_values(q)
    x = [sum(Fraction(float(qv[g, d])) * Fraction(float(P[i, d])) for g in range(3) for d in range(128))
         for i in range(32)]
    m = max(abs(v) for v in x)
    expect = []
    for v in x:
        y = v * 127 / m
        t = int(abs(y))
        frac = abs(y) - t
        assert abs(frac - Fraction(1, 2)) > Fraction(1, 10 ** 9)
        mag = t + (1 if frac >= Fraction(1, 2) else 0)
        expect.append(mag if y >= 0 else -mag)
    assert r["p"].tolist() == expect


def pin_quantize_invariances(o):
    rng = np.random.default_rng(20)
    q = random_bf16(rng, (1, 128))
    P = (rng.standard_normal((64, 128)) * 0.5).astype(np.float32)
    p1 = o.quantize_query(q, P)["p"]
    q2 = to_bf16_bits(4.0 * bf16_values(q))  # exact power-of-two scaling
    assert np.array_equal(o.quantize_query(q2, P)["p"], p1)
    assert np.array_equal(o.quantize_query(np.concatenate([q, q]), P)["p"], p1)  # G = 2 equal heads
    # projection rows that pick single coordinates: x = q restricted
    Pi = np.zeros((32, 128), np.float32)
    Pi[np.arange(32), np.arange(32) * 4] = 1.0
    r = o.quantize_query(q, Pi)
    qv = bf16_values(q)[0, ::4][:32]
    assert np.array_equal(r["x"], qv)
    zero = o.quantize_query(np.zeros((2, 128), np.uint16), P)
    assert np.all(zero["p"] == 0) and zero["T"] == 0


# ---------------------------------------------------------------- score

def pin_score_bitplane_identity(o):
    # Appendix "CUDA Optimizations": sum_i h_i p_i = sum_j 2^j (popc(m_j & w+) - popc(m_j & w-)),
    # evaluated here with the magnitude planes weighted 1, 2, ..., 64
    rng = np.random.default_rng(21)
    for L in (32, 64, 128):
        W = L // 32
        p = rng.integers(-127, 128, size=L)
        codes = rng.integers(0, 1 << 32, size=(400, W), dtype=np.uint64).astype(np.uint32)
        sign_bits = np.zeros(W, np.uint32)
        planes = np.zeros((7, W), np.uint32)
        for i in range(L):
            if p[i] >= 0:
                sign_bits[i // 32] |= np.uint32(1 << (i % 32))
            for j in range(7):
                if (abs(p[i]) >> j) & 1:
                    planes[j, i // 32] |= np.uint32(1 << (i % 32))
        agree = ~(codes ^ sign_bits[None, :])  # bit set where h_i and s_i agree
        c = np.zeros(400, np.int64)
        for j in range(7):
            pos = popcount32(planes[j][None, :] & agree).sum(axis=1)
            neg = popcount32(planes[j][None, :] & ~agree).sum(axis=1)
            c += (pos - neg) << j
        assert np.array_equal(o.hash_scores(codes, p, L), c)


def pin_score_hamming(o):
    rng = np.random.default_rng(22)
    L = 64
    codes = rng.integers(0, 1 << 32, size=(50, 2), dtype=np.uint64).astype(np.uint32)
    H = np.where(((codes[:, :, None] >> np.arange(32, dtype=np.uint32)) & 1).reshape(50, L) == 1, 1, -1)

    def ham(a, b):
        return int(popcount32(codes[a] ^ codes[b]).sum())

    for mu in (1, 5, 127):
        for a in range(5):
            p = mu * H[a]
            c = o.hash_scores(codes, p, L)
            for b in range(50):
                assert c[b] == mu * (L - 2 * ham(a, b))
            assert c[a] == mu * L == int(np.abs(p).sum())  # equality iff h = sign(p)
            assert np.all(c[np.arange(50) != a] < mu * L) or len(set(map(tuple, codes))) < 50
    # symmetry and triangle inequality of the Hamming distance recovered from scores
    D = np.array([[(L - o.hash_scores(codes[[b]], H[a], L)[0]) // 2 for b in range(12)] for a in range(12)])
    assert np.array_equal(D, D.T) and np.all(np.diag(D) == 0) and np.all((0 <= D) & (D <= L))
    for a in range(12):
        for b in range(12):
            assert np.all(D[a, b] <= D[a, :] + D[:, b])
    full = o.hash_scores(~codes[:1], H[0], L)[0]
    assert full == -L


# ---------------------------------------------------------------- select

def pin_select(o):
    rng = np.random.default_rng(23)
    for N, k in ((50, 7), (200, 200), (333, 1), (1000, 20)):
        c = rng.integers(-5, 6, size=N)  # many ties
        expect = sorted(sorted(range(N), key=lambda j: (-int(c[j]), j))[:k])
        assert o.select_topk(c, k).tolist() == expect
    assert o.select_topk(np.zeros(10, np.int64), 4).tolist() == [0, 1, 2, 3]
    c = np.array([3, 9, 9, 1, 9, 9])
    assert o.select_topk(c, 3).tolist() == [1, 2, 4]


# ---------------------------------------------------------------- attention

def pin_attend_full(o):
    rng = np.random.default_rng(24)
    N, D, Gq = 300, 128, 4
    q = random_bf16(rng, (Gq, D))
    K = random_bf16(rng, (N, D), 2.0)
    V = random_bf16(rng, (N, D))
    sm = 1.0 / np.sqrt(D)
    out = o.full_attention(q, K, V, sm)
    tq = torch.from_numpy(bf16_values(q))[None]
    tk = torch.from_numpy(bf16_values(K))[None, None].expand(1, Gq, N, D)
    tv = torch.from_numpy(bf16_values(V))[None, None].expand(1, Gq, N, D)
    ref = torch.nn.functional.scaled_dot_product_attention(tq[:, :, None, :], tk, tv, scale=sm)[0, :, 0].numpy()
    assert np.allclose(out, ref, rtol=1e-12, atol=1e-13)
    idx = np.array([17])
    assert np.array_equal(o.attend(q, K, V, idx, sm), np.repeat(bf16_values(V[17])[None], Gq, axis=0))
    z = o.attend(np.zeros((1, D), np.uint16), K, V, np.array([1, 5, 9]), sm)
    assert np.allclose(z[0], bf16_values(V[[1, 5, 9]]).mean(axis=0), rtol=1e-14, atol=1e-15)


def pin_topk_baseline(o):
    # exact-score selection followed by sparse attention is the TOPK baseline
    rng = np.random.default_rng(25)
    N, D, Gq, k = 400, 128, 4, 9
    q = random_bf16(rng, (Gq, D))
    K = random_bf16(rng, (N, D))
    V = random_bf16(rng, (N, D))
    idx = o.exact_topk(q, K, k)
    s = bf16_values(K) @ bf16_values(q).sum(axis=0)
    expect = np.sort(np.argsort(-s, kind="stable")[:k])
    assert np.array_equal(idx, expect)
    sm = 1.0 / np.sqrt(D)
    out = o.attend(q, K, V, idx, sm)
    logits = bf16_values(q) @ bf16_values(K[expect]).T * sm
    w = torch.softmax(torch.from_numpy(logits), dim=1).numpy()
    assert np.allclose(out, w @ bf16_values(V[expect]), rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------------- error-aware safeguard

def pin_eas_budget(o):
    # 10 % of the budget is reserved for the safeguard (Sec. 4.1), rounded up
    # like the budget itself; k_hash keeps at least one key
    assert o.eas_budget(2622) == (2359, 263)   # 2 % of 131072 keys
    assert o.eas_budget(10) == (9, 1)
    assert o.eas_budget(11) == (9, 2)
    assert o.eas_budget(2) == (1, 1)
    assert o.eas_budget(1) == (1, 0)
    assert o.eas_budget(100, 15, 100) == (85, 15)


def pin_select_hard(o):
    rng = np.random.default_rng(26)
    for N, m in ((40, 5), (300, 300), (257, 1), (1000, 37)):
        e = rng.choice(np.array([0.0, 0.5, 1.25, 3.0, 7.5], np.float32), size=N)  # many ties
        expect = sorted(sorted(range(N), key=lambda j: (-float(e[j]), j))[:m])
        assert o.select_hard(e, m).tolist() == expect
    assert o.select_hard(np.ones(5, np.float32), 0).tolist() == []
    # IEEE total order: -0 below +0, negatives below both
    assert o.select_hard(np.array([0.0, -0.0], np.float32), 1).tolist() == [0]
    assert o.select_hard(np.array([-0.0, 0.0], np.float32), 1).tolist() == [1]
    assert o.select_hard(np.array([-1.0, -0.0, -2.0], np.float32), 2).tolist() == [0, 1]
    # a key far outside the subspace of the others is the hardest to hash
    # (the "passkey" situation the safeguard is for, Sec. 4.3)
    N, D, L = 200, 128, 32
    Kv = bf16_values(_lowrank_keys(rng, N, D))
    out = np.zeros(D)
    out[7] = 3.0 * np.linalg.norm(Kv, axis=1).max()  # off the keys' 4-dimensional subspace
    Kv[113] = out
    Kb = to_bf16_bits(Kv)
    G = rng.standard_normal((L, D)).astype(np.float32)
    _, _, err, _ = o.build_binary_pcs(Kb, G)
    assert o.select_hard(err.astype(np.float32), 1).tolist() == [113]


def pin_eas_union(o):
    rng = np.random.default_rng(27)
    N, D, Gq, L, k = 500, 128, 2, 64, 20
    q = random_bf16(rng, (Gq, D))
    K = random_bf16(rng, (N, D))
    V = random_bf16(rng, (N, D))
    codes = rng.integers(0, 1 << 32, size=(N, L // 32), dtype=np.uint64).astype(np.uint32)
    P = (0.5 * rng.standard_normal((L, D))).astype(np.float32)
    sm = 1.0 / np.sqrt(D)
    plain = o.decode_head(q, K, V, codes, P, k, sm)
    # no hard keys: the plain decode step
    r = o.decode_head_eas(q, K, V, codes, P, k, np.zeros(0, np.int64), sm)
    assert np.array_equal(r["idx"], plain["idx"]) and np.array_equal(r["union"], plain["idx"])
    assert np.array_equal(r["out"], plain["out"])
    # hard keys already selected by hash: nothing added, same output
    inside = plain["idx"][::3]
    r = o.decode_head_eas(q, K, V, codes, P, k, inside, sm)
    assert np.all(r["added"] == 0) and np.array_equal(r["out"], plain["out"])
    # disjoint hard keys: the union has k + m keys and attention runs over all of them
    outside = np.setdiff1d(np.arange(N), plain["idx"])[[0, 5, 77, 200]]
    r = o.decode_head_eas(q, K, V, codes, P, k, outside, sm)
    assert np.all(r["added"] == 1) and r["union"].size == k + 4
    expect = np.sort(np.concatenate([plain["idx"], outside]))
    assert np.array_equal(r["union"], expect)
    logits = bf16_values(q) @ bf16_values(K[expect]).T * sm
    w = torch.softmax(torch.from_numpy(logits), dim=1).numpy()
    assert np.allclose(r["out"], w @ bf16_values(V[expect]), rtol=1e-12, atol=1e-13)
    # every key by hash: full attention whatever the hard set is
    r = o.decode_head_eas(q, K, V, codes, P, N, outside, sm)
    assert np.allclose(r["out"], o.full_attention(q, K, V, sm), rtol=1e-12, atol=1e-13)


def pin_per_query_head(o):
    """Per-query-head selection against facts that fix it without retyping it:
    opposite queries give exactly negated scores (while the group rule sees a
    zero sum and ties everything), identical queries reproduce the group rule
    (the quantisation is scale invariant for a power-of-two group), a head's
    result does not depend on the other heads' queries, and G = 1 is the
    ordinary decode step."""
    rng = np.random.default_rng(31)
    N, D, L, k = 600, 128, 64, 25
    K = random_bf16(rng, (N, D))
    V = random_bf16(rng, (N, D))
    codes = rng.integers(0, 1 << 32, size=(N, L // 32), dtype=np.uint64).astype(np.uint32)
    P = (0.5 * rng.standard_normal((L, D))).astype(np.float32)
    sm = 1.0 / np.sqrt(D)
    q0 = random_bf16(rng, (1, D))
    # opposite heads: q1 = -q0 exactly (bf16 negation flips the sign bit)
    q = np.concatenate([q0, q0 ^ np.uint16(0x8000)])
    r = o.decode_per_query_head(q, K, V, codes, P, k, sm)
    assert np.array_equal(r["scores"][1], -r["scores"][0])
    assert np.array_equal(r["p"][1], -r["p"][0])
    grp = o.decode_head(q, K, V, codes, P, k, sm)
    assert np.all(grp["scores"] == 0) and np.array_equal(grp["idx"], np.arange(k))
    H = o.unpack_codes(codes, L).astype(np.int64)
    best0 = np.lexsort((np.arange(N), -(H @ r["p"][0])))[:k]
    assert np.array_equal(r["idx"][0], np.sort(best0))
    for g in range(2):
        logits = bf16_values(q[g]) @ bf16_values(K[r["idx"][g]]).T * sm
        w = torch.softmax(torch.from_numpy(logits), dim=0).numpy()
        assert np.allclose(r["out"][g], w @ bf16_values(V[r["idx"][g]]), rtol=1e-12, atol=1e-13)
    # identical heads (G = 4): every head selects what the group selects
    q4 = np.repeat(q0, 4, axis=0)
    r4 = o.decode_per_query_head(q4, K, V, codes, P, k, sm)
    g4 = o.decode_head(q4, K, V, codes, P, k, sm)
    for g in range(4):
        assert np.array_equal(r4["idx"][g], g4["idx"]) and np.array_equal(r4["p"][g], g4["p"])
    assert np.allclose(r4["out"], g4["out"], rtol=1e-12, atol=1e-13)
    # a head ignores the other heads' queries; permuting heads permutes results
    qa = random_bf16(rng, (3, D))
    qb = qa.copy()
    qb[1:] = random_bf16(rng, (2, D))
    ra, rb = o.decode_per_query_head(qa, K, V, codes, P, k, sm), o.decode_per_query_head(qb, K, V, codes, P, k, sm)
    assert np.array_equal(ra["idx"][0], rb["idx"][0]) and np.array_equal(ra["out"][0], rb["out"][0])
    rp = o.decode_per_query_head(qa[::-1], K, V, codes, P, k, sm)
    assert np.array_equal(rp["idx"], ra["idx"][::-1]) and np.array_equal(rp["qcode"], ra["qcode"][::-1])


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
