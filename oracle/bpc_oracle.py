"""Plain, slow, fp64 CPU reference of the BinaryPC decode hot path.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the
benchmark's CPU-baseline leg are the only callers.  Nothing here is used by,
or uses, the HIP library.

Paper: "Training-Free Hashing-Based Attention via Binary Principal
Components" (BinaryPC).  Every function names the passage it follows.
Notation follows the paper: K [N, D] keys, H in {-1,+1}^{N x L} hash codes,
P [L, D] projection (binary principal components), q a query, p the
quantised projected query, c = p . h the hash score.

Arithmetic that decides a bit or an index is fixed here so that it is
reproducible (the paper does not fix it):

* All floating point is IEEE binary64 unless stated; bf16 and fp32 inputs
  are widened exactly.
* "canonical dot" of two D-vectors (D a multiple of 4): the coordinates are
  split into 4 consecutive blocks of D/4; each block is summed in ascending
  order starting from +0 with a separately rounded multiply and add (no fused
  multiply-add); the block sums are combined as ((b0 + b1) + (b2 + b3)).
* "pairwise tree" over N rows: adjacent pairs (0,1), (2,3), ... are added
  level by level; an odd last element is carried up unchanged.
* sign(a) = +1 when a >= 0 (so both zeros give +1), else -1.
* A sign bit is "fragile" when |float32(a)| < 1e-6; fragile bits are counted.
* Code bit i of a key lives in bit (i mod 32) of 32-bit word floor(i / 32);
  bit value 1 means h_i = +1.

Parity status: every function below is pinned by the CPU tests (closed
forms, exact rational re-evaluation, invariants, library routines, brute
force); none is "parity unpinned".  The method-quality diagnostics (needle recall, cosine
similarity with full attention) are reported, not part of parity.
"""

from __future__ import annotations

import numpy as np

__all__ = [
    "bf16_bits_to_f64",
    "canonical_dot",
    "canonical_sumsq",
    "pairwise_tree_sum",
    "pack_codes",
    "unpack_codes",
    "build_binary_pcs",
    "hash_keys",
    "quantize_query",
    "unpack_query_planes",
    "hash_scores",
    "select_topk",
    "attend",
    "full_attention",
    "exact_topk",
    "decode_head",
    "select_hard",
    "eas_budget",
    "decode_head_eas",
    "decode_per_query_head",
    "budget_keys",
    "FRAGILE_THRESHOLD",
]

FRAGILE_THRESHOLD = np.float32(1e-6)


# --------------------------------------------------------------------------
# number formats and fixed-order reductions
# --------------------------------------------------------------------------

def bf16_bits_to_f64(bits) -> np.ndarray:
    """bfloat16 bit patterns (uint16) widened exactly to float64."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def canonical_dot(X: np.ndarray, w: np.ndarray) -> np.ndarray:
    """sum_d X[..., d] * w[d] in the fixed order described in the module doc."""
    X = np.asarray(X, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    D = X.shape[-1]
    if D % 4 != 0 or w.shape != (D,):
        raise ValueError("canonical_dot needs D % 4 == 0 and w of shape [D]")
    blk = D // 4
    parts = []
    for b in range(4):
        acc = np.zeros(X.shape[:-1], dtype=np.float64)
        for d in range(b * blk, (b + 1) * blk):
            prod = X[..., d] * w[d]
            acc = acc + prod
        parts.append(acc)
    return (parts[0] + parts[1]) + (parts[2] + parts[3])


def canonical_sumsq(X: np.ndarray) -> np.ndarray:
    """sum_d X[..., d]^2 in the canonical-dot order."""
    X = np.asarray(X, dtype=np.float64)
    D = X.shape[-1]
    blk = D // 4
    parts = []
    for b in range(4):
        acc = np.zeros(X.shape[:-1], dtype=np.float64)
        for d in range(b * blk, (b + 1) * blk):
            acc = acc + X[..., d] * X[..., d]
        parts.append(acc)
    return (parts[0] + parts[1]) + (parts[2] + parts[3])


def pairwise_tree_sum(T: np.ndarray) -> np.ndarray:
    """Sum over axis 0 with the pairwise tree (odd last element carried)."""
    T = np.asarray(T, dtype=np.float64)
    if T.shape[0] == 0:
        return np.zeros(T.shape[1:], dtype=np.float64)
    while T.shape[0] > 1:
        n = T.shape[0]
        even = n - (n % 2)
        s = T[0:even:2] + T[1:even:2]
        if n % 2:
            s = np.concatenate([s, T[n - 1:n]], axis=0)
        T = s
    return T[0].copy()


def budget_keys(N: int, num: int, den: int) -> int:
    """Budget k = ceil(N * num / den) keys (Sec. 4.1 'Baselines': a fixed
    percentage of the context), in exact integer arithmetic."""
    return -((-N * num) // den)


# --------------------------------------------------------------------------
# code packing
# --------------------------------------------------------------------------

def pack_codes(H: np.ndarray) -> np.ndarray:
    """±1 codes [N, L] -> uint32 words [N, L/32]; bit set <=> +1."""
    H = np.asarray(H)
    N, L = H.shape
    if L % 32:
        raise ValueError("L must be a multiple of 32")
    bits = (H > 0).astype(np.uint64).reshape(N, L // 32, 32)
    weights = (np.uint64(1) << np.arange(32, dtype=np.uint64))
    return (bits * weights).sum(axis=2).astype(np.uint32)


def unpack_codes(codes: np.ndarray, L: int) -> np.ndarray:
    """uint32 words [N, L/32] -> ±1 int8 codes [N, L]."""
    c = np.asarray(codes, dtype=np.uint32)
    N = c.shape[0]
    shifts = np.arange(32, dtype=np.uint32)
    bits = (c[:, :, None] >> shifts[None, None, :]) & np.uint32(1)
    bits = bits.reshape(N, -1)[:, :L]
    return np.where(bits == 1, 1, -1).astype(np.int8)


def _fragile_count(a: np.ndarray) -> int:
    return int(np.count_nonzero(np.abs(a.astype(np.float32)) < FRAGILE_THRESHOLD))


# --------------------------------------------------------------------------
# Algorithm 1: binary principal components (Sec. 3.2, "Binary Principal
# Components Finding"; Algorithm "Constructing hash codes and corresponding
# hashing projection"; Appendix "Procedure Overview" for the closed-form v)
# --------------------------------------------------------------------------

def build_binary_pcs(K_bits, G, trace: bool = False):
    """Greedy rank-1 binary decomposition K ~ H P.

    For i = 0..L-1, with residual R (initially K) and the i-th Gaussian
    direction g = G[i] (the random v* of the algorithm, supplied by the
    caller):
        a  = R g           (canonical dot per row)
        u  = sign(a)
        v  = u^T R / N     (pairwise tree over rows, then one rounded divide)
        P[i] = float32(v);  H[:, i] = u
        R  = R - u P[i]    (the stored float32 P is what is subtracted)
    Returns (P [L, D] float32, codes [N, L/32] uint32, err [N] float64 =
    ||k - h P|| per row, fragile count[, trace dict]).
    """
    K = bf16_bits_to_f64(K_bits)
    G = np.asarray(G, dtype=np.float32)
    N, D = K.shape
    L = G.shape[0]
    if G.shape[1] != D:
        raise ValueError("G must be [L, D]")
    R = K.copy()
    P = np.zeros((L, D), dtype=np.float32)
    H = np.empty((N, L), dtype=np.int8)
    fragile = 0
    tr = {"R_fro2": [float(np.sum(R * R))], "v": [], "u": []}
    for i in range(L):
        g = G[i].astype(np.float64)
        a = canonical_dot(R, g)
        u = np.where(a >= 0.0, 1.0, -1.0)
        fragile += _fragile_count(a)
        s = pairwise_tree_sum(R * u[:, None])
        v = s / np.float64(N) if N > 0 else s
        P[i] = v.astype(np.float32)
        R = R - u[:, None] * P[i].astype(np.float64)[None, :]
        H[:, i] = u.astype(np.int8)
        if trace:
            tr["R_fro2"].append(float(np.sum(R * R)))
            tr["v"].append(v.copy())
            tr["u"].append(u.copy())
    err = np.sqrt(canonical_sumsq(R))
    codes = pack_codes(H) if L % 32 == 0 else None
    if trace:
        tr["R"] = R
        tr["H"] = H
        return P, codes, err, fragile, tr
    return P, codes, err, fragile


# --------------------------------------------------------------------------
# Algorithm 2: hash a key given P (Sec. 3.2, "Given projection, computing
# hashcode"; the iterative residual form is required because rows of P are
# not orthogonal)
# --------------------------------------------------------------------------

def hash_keys(K_bits, P, return_H: bool = False):
    """Per key: r = k; for i: u = sign(r . P[i]); r = r - u P[i]; h[i] = u.

    Returns (codes [N, L/32] uint32, err [N] float64 = ||r_final||,
    fragile count[, H])."""
    r = bf16_bits_to_f64(K_bits)
    P = np.asarray(P, dtype=np.float32)
    Pd = P.astype(np.float64)
    N = r.shape[0]
    L = P.shape[0]
    H = np.empty((N, L), dtype=np.int8)
    fragile = 0
    for i in range(L):
        a = canonical_dot(r, Pd[i])
        u = np.where(a >= 0.0, 1.0, -1.0)
        fragile += _fragile_count(a)
        r = r - u[:, None] * Pd[i][None, :]
        H[:, i] = u.astype(np.int8)
    err = np.sqrt(canonical_sumsq(r))
    codes = pack_codes(H) if L % 32 == 0 else None
    if return_H:
        return codes, err, fragile, H
    return codes, err, fragile


# --------------------------------------------------------------------------
# Query projection and quantisation (Sec. 3.2 "Retrieval Phase"; Appendix
# "CUDA Optimizations on Bitwise Operations", packing kernel)
# --------------------------------------------------------------------------

def _round_half_away(y: np.ndarray) -> np.ndarray:
    """Exact round-half-away-from-zero of float64 values, as int64."""
    t = np.trunc(y)
    frac = y - t  # exact for |y| < 2**52
    bump = (np.abs(frac) >= 0.5).astype(np.int64)
    return t.astype(np.int64) + np.sign(y).astype(np.int64) * bump


def quantize_query(q_bits, P):
    """Project the query group onto P and quantise to 7-bit magnitudes.

    q_bits [Gq, D] are the bf16 query heads sharing one KV head.  Each head
    is projected, x_g = q_g P^T (canonical dot per component), and the
    projections are summed in ascending head order, x = sum_g x_g.  With
    m = max_i |x_i|, y_i = (x_i * 127) / m and p_i = round-half-away(y_i) in
    [-127, 127] (p = 0 when m = 0).  Packing: plane 0 holds sign bits
    (1 <=> p_i >= 0), plane 1 + j holds bit j of |p_i| (j = 0..6).

    Returns dict(p [L] int64, x [L] float64, qcode [8, L/32] uint32,
    T = sum |p_i|, round_fragile = #{| |y| - floor(|y|) - 0.5 | < 1e-9}).
    """
    q = bf16_bits_to_f64(np.atleast_2d(q_bits))
    P = np.asarray(P, dtype=np.float32).astype(np.float64)
    L = P.shape[0]
    xs = [canonical_dot(P, q[g]) for g in range(q.shape[0])]
    x = xs[0]
    for g in range(1, len(xs)):
        x = x + xs[g]
    m = float(np.max(np.abs(x))) if L else 0.0
    if m == 0.0:
        p = np.zeros(L, dtype=np.int64)
        y = np.zeros(L, dtype=np.float64)
    else:
        y = (x * 127.0) / m
        p = _round_half_away(y)
    ay = np.abs(y)
    round_fragile = int(np.count_nonzero(np.abs(ay - np.floor(ay) - 0.5) < 1e-9))
    planes = np.empty((8, L), dtype=np.int8)
    planes[0] = np.where(p >= 0, 1, -1)
    mag = np.abs(p)
    for j in range(7):
        planes[1 + j] = np.where(((mag >> j) & 1) == 1, 1, -1)
    qcode = pack_codes(planes) if L % 32 == 0 else None
    return {"p": p, "x": x, "qcode": qcode, "T": int(mag.sum()), "round_fragile": round_fragile}


def unpack_query_planes(qcode, L: int) -> np.ndarray:
    """Packed query planes [8, L/32] -> integers p [L] (inverse of packing)."""
    planes = unpack_codes(np.asarray(qcode, dtype=np.uint32), L)  # [8, L] of ±1
    sign = np.where(planes[0] > 0, 1, -1).astype(np.int64)
    mag = np.zeros(L, dtype=np.int64)
    for j in range(7):
        mag += (planes[1 + j] > 0).astype(np.int64) << j
    return sign * mag


# --------------------------------------------------------------------------
# Hash score (Sec. 3.2 "Retrieval Phase": c = (q P^T) h^T; Algorithm
# "Computing hashing score" evaluates the same integer with bit planes)
# --------------------------------------------------------------------------

def hash_scores(codes, p, L: int | None = None) -> np.ndarray:
    """c_j = sum_i h_{j,i} p_i as an exact integer dot of unpacked codes."""
    p = np.asarray(p, dtype=np.int64)
    L = p.shape[0] if L is None else L
    H = unpack_codes(codes, L).astype(np.int64)
    return H @ p


# --------------------------------------------------------------------------
# Top-k selection (Sec. 3.2: "the top-k candidates with highest hash scores")
# --------------------------------------------------------------------------

def select_topk(c, k: int) -> np.ndarray:
    """Indices of the k largest scores; equal scores go to the lower index.
    Returned in ascending index order (int64)."""
    c = np.asarray(c, dtype=np.int64)
    N = c.shape[0]
    if not 1 <= k <= N:
        raise ValueError("need 1 <= k <= N")
    order = np.lexsort((np.arange(N), -c))
    return np.sort(order[:k])


# --------------------------------------------------------------------------
# Sparse attention over the selected rows (Sec. 4.2 "Kernel Evaluation":
# gather the selected K/V rows, then ordinary softmax attention over them)
# --------------------------------------------------------------------------

def attend(q_bits, K_bits, V_bits, idx, sm_scale: float) -> np.ndarray:
    """softmax((q . K_j) * sm_scale over j in idx) weighted sum of V_j, fp64.

    q_bits [Gq, D]; K_bits, V_bits [N, D]; returns [Gq, D] float64."""
    q = bf16_bits_to_f64(np.atleast_2d(q_bits))
    idx = np.asarray(idx, dtype=np.int64)
    Ks = bf16_bits_to_f64(np.asarray(K_bits)[idx])
    Vs = bf16_bits_to_f64(np.asarray(V_bits)[idx])
    logits = (q @ Ks.T) * np.float64(sm_scale)
    mx = logits.max(axis=1, keepdims=True)
    w = np.exp(logits - mx)
    w = w / w.sum(axis=1, keepdims=True)
    return w @ Vs


def full_attention(q_bits, K_bits, V_bits, sm_scale: float) -> np.ndarray:
    """Dense softmax attention over all N rows (the k = N special case)."""
    N = np.asarray(K_bits).shape[0]
    return attend(q_bits, K_bits, V_bits, np.arange(N), sm_scale)


def exact_topk(q_bits, K_bits, k: int) -> np.ndarray:
    """The TOPK baseline (Appendix A.1): top-k keys by exact full-precision
    scores.  For a query group the score of key j is sum_g q_g . k_j, the
    exact counterpart of the summed projected query used for hashing."""
    q = bf16_bits_to_f64(np.atleast_2d(q_bits))
    K = bf16_bits_to_f64(K_bits)
    s = K @ q.sum(axis=0)
    N = K.shape[0]
    order = np.lexsort((np.arange(N), -s))
    return np.sort(order[:k])


# --------------------------------------------------------------------------
# one decode step for one (sequence, KV head)
# --------------------------------------------------------------------------

def decode_head(q_bits, K_bits, V_bits, codes, P, k: int, sm_scale: float):
    """Quantise the query group, score every cached code, select top-k and
    attend over the selected rows.  q_bits [Gq, D]; K_bits, V_bits [N, D];
    codes [N, L/32]; P [L, D]."""
    P = np.asarray(P, dtype=np.float32)
    L = P.shape[0]
    qq = quantize_query(q_bits, P)
    c = hash_scores(codes, qq["p"], L)
    idx = select_topk(c, k)
    out = attend(q_bits, K_bits, V_bits, idx, sm_scale)
    return {"p": qq["p"], "qcode": qq["qcode"], "T": qq["T"], "scores": c, "idx": idx, "out": out}


def decode_per_query_head(q_bits, K_bits, V_bits, codes, P, k: int, sm_scale: float):
    """Per-query-head selection, the alternative to one selection per KV
    head: every query head g of the group projects and quantises its own
    query q_g P^T (Sec. 3.2 "Retrieval Phase"), scores every cached code of
    the shared KV head against it (Alg. 3), takes its own top-k and attends
    over its own selection.  q_bits [Gq, D]; returns per-head stacks:
    p [Gq, L], qcode [Gq, 8, L/32], scores [Gq, N], idx [Gq, k], out [Gq, D]."""
    q_bits = np.asarray(q_bits)
    heads = [decode_head(q_bits[g:g + 1], K_bits, V_bits, codes, P, k, sm_scale) for g in range(q_bits.shape[0])]
    return {"p": np.stack([r["p"] for r in heads]), "qcode": np.stack([r["qcode"] for r in heads]),
            "scores": np.stack([r["scores"] for r in heads]), "idx": np.stack([r["idx"] for r in heads]),
            "out": np.concatenate([r["out"] for r in heads], axis=0)}


# --------------------------------------------------------------------------
# Error-Aware Safeguard (Sec. 3.2 "Error-Aware Safeguard (EAS)", Eq.
# reconstruction_error and Eq. safeguard_union; Sec. 4.1 "Baselines": 10 %
# of the token budget is reserved for EAS)
# --------------------------------------------------------------------------

def eas_budget(budget: int, num: int = 1, den: int = 10) -> tuple[int, int]:
    """Split a token budget into (k_hash, m): m = ceil(budget * num / den)
    keys are reserved for the hard-to-hash set and k_hash = budget - m are
    taken by hash score; m is capped at budget - 1 so that k_hash >= 1."""
    if budget < 1:
        raise ValueError("budget must be >= 1")
    m = min(-(-budget * num // den), budget - 1)
    return budget - m, m


def select_hard(err, m: int) -> np.ndarray:
    """The hard-to-hash set S_err: indices of the m largest reconstruction
    errors ||k - h P|| (given as float32, the precision the library stores
    them in), ordered by value with equal values going to the lower index.
    Values are compared in the IEEE total order of float32.  Returned in
    ascending index order (int64)."""
    e = np.asarray(err, dtype=np.float32)
    N = e.shape[0]
    if not 0 <= m <= N:
        raise ValueError("need 0 <= m <= N")
    u = e.view(np.uint32).astype(np.int64)
    key = np.where(u >= (1 << 31), (~u) & 0xFFFFFFFF, u | (1 << 31))  # total order, larger = larger
    order = np.lexsort((np.arange(N), -key))
    return np.sort(order[:m])


def decode_head_eas(q_bits, K_bits, V_bits, codes, P, k_hash: int, serr, sm_scale: float):
    """decode_head with the safeguard: attention over S_attn = S_hash u S_err,
    S_hash the k_hash keys with the highest hash scores and S_err a given
    index set (from select_hard at prefill).  Also returns, per entry of
    S_err, whether it was added to S_hash (1) or already in it (0)."""
    P = np.asarray(P, dtype=np.float32)
    L = P.shape[0]
    qq = quantize_query(q_bits, P)
    c = hash_scores(codes, qq["p"], L)
    idx = select_topk(c, k_hash)
    serr = np.asarray(serr, dtype=np.int64)
    added = (~np.isin(serr, idx)).astype(np.int32)
    union = np.union1d(idx, serr)
    out = attend(q_bits, K_bits, V_bits, union, sm_scale)
    return {"p": qq["p"], "qcode": qq["qcode"], "scores": c, "idx": idx, "union": union, "added": added,
            "out": out}
