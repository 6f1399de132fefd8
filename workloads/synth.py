"""Seeded synthetic KV caches, queries and Gaussian directions.

The paper evaluates on Llama-family KV caches drawn from long-context
benchmarks (Sec. 4.1, Appendix A.2); none of those are available here, so
these generators stand in for them with the shapes the paper measures
(head_dim 128, 8 KV heads, GQA group 4, bf16 keys/values, 32K-1M cached
tokens) and with keys that have the two properties the method relies on:
a low-rank principal subspace and a few outlier channels.

Recipe (per layer, per KV head; the basis is shared by the batch):
  A  [rank, D] ~ N(0, 1),  outlier channels = `n_outliers` distinct indices
  Z  [N, rank] ~ N(0, 1),  E [N, D] ~ N(0, 1)           (per sequence)
  K  = Z A + noise * E, outlier channels x outlier_scale, rounded to bf16
  V  [N, D] ~ N(0, 1) -> bf16,  q [B, Hq, D] ~ N(0, 1) -> bf16
Needles: `needles` positions per (sequence, KV head), uniform without
replacement; needle j is aligned with query head g = h*G + (j mod G) of that
group and set to scale * q_g / |q_g| (bf16), where scale is 3*rho (rho = the
head's RMS key norm; default), 3 (literal), or 3*|q_g| ("3q").
Gaussian directions for the binary-PC build: G [L, D] ~ N(0, 1) drawn in
float64 and rounded to float32, one matrix per configuration.

Random numbers come from torch generators seeded per (config, layer, batch,
head, tensor) so that any single head can be regenerated on its own.  The
values depend on the device the generator runs on (CPU and GPU streams
differ), so a caller that needs the same head on both sides generates it once
and copies it.  On the CPU they do not depend on the host: the normals are
drawn in float64 (torch's float32 normals take a vectorised path whose values
change with the CPU's instruction set) and Z A is accumulated elementwise in
a fixed order (a BLAS product's summation order changes with the CPU), so
values stored from one machine are reproduced on another.
"""

from __future__ import annotations

import dataclasses
from typing import Optional, Sequence

import torch

__all__ = [
    "DecodeConfig",
    "CONFIGS",
    "config_by_name",
    "make_gaussian_directions",
    "make_layer",
    "make_head",
    "seed_for",
]


@dataclasses.dataclass(frozen=True)
class DecodeConfig:
    """Shape of one decode workload."""

    name: str
    B: int
    layers: int
    Hq: int
    Hkv: int
    D: int
    N: int
    L: int
    budget_num: int  # budget fraction = budget_num / budget_den of the N keys
    budget_den: int
    needles: int  # planted needle keys per (sequence, KV head)
    rank: int = 16
    n_outliers: int = 4
    outlier_scale: float = 10.0
    noise: float = 0.1
    seed: int = 1000

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def k(self) -> int:
        """Selection budget: ceil(fraction * N), computed exactly."""
        return budget_keys(self.N, self.budget_num, self.budget_den)

    @property
    def W(self) -> int:
        return self.L // 32

    def replace(self, **kw) -> "DecodeConfig":
        return dataclasses.replace(self, **kw)


def budget_keys(N: int, num: int, den: int) -> int:
    return -((-N * num) // den)


CONFIGS = (
    # tiny decode step: 1 x 8/8 heads, 4096 keys, 32-bit codes, 2 % budget
    DecodeConfig("tiny_mha_4k", B=1, layers=1, Hq=8, Hkv=8, D=128, N=4096, L=32,
                 budget_num=2, budget_den=100, needles=16, seed=1000),
    # Llama-3-8B-shaped single layer: 32/8 heads, 32768 keys, 64-bit codes
    DecodeConfig("llama8b_32k", B=1, layers=1, Hq=32, Hkv=8, D=128, N=32768, L=64,
                 budget_num=2, budget_den=100, needles=16, seed=1001),
    # batched long context: batch 16, 32/8 heads, 131072 keys, 64-bit codes
    DecodeConfig("batch16_128k", B=16, layers=1, Hq=32, Hkv=8, D=128, N=131072, L=64,
                 budget_num=2, budget_den=100, needles=0, seed=1002),
    # 8B-shaped stack: 32 layers, batch 8, 65536 keys, 64-bit codes
    DecodeConfig("stack32_b8_64k", B=8, layers=32, Hq=32, Hkv=8, D=128, N=65536, L=64,
                 budget_num=2, budget_den=100, needles=0, seed=1003),
    # million-token stress: 1M keys, 128-bit codes, 1 % budget, 64 needles
    DecodeConfig("million_1m", B=1, layers=1, Hq=32, Hkv=8, D=128, N=1048576, L=128,
                 budget_num=1, budget_den=100, needles=64, seed=1004),
)


def config_by_name(name: str) -> DecodeConfig:
    for c in CONFIGS:
        if c.name == name:
            return c
    raise KeyError(name)


_MASK64 = (1 << 64) - 1


def _splitmix64(x: int) -> int:
    x = (x + 0x9E3779B97F4A7C15) & _MASK64
    z = x
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
    return z ^ (z >> 31)


def seed_for(*parts: int) -> int:
    """Derive a 63-bit generator seed from a tuple of small integers."""
    h = 0x243F6A8885A308D3
    for p in parts:
        h = _splitmix64(h ^ (int(p) & _MASK64))
    return h & ((1 << 63) - 1)


_TAG_BASIS, _TAG_KEYS, _TAG_VALUES, _TAG_QUERY, _TAG_NEEDLE, _TAG_G = range(6)


def _generator(device, *parts) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed_for(*parts))
    return g


def make_gaussian_directions(cfg: DecodeConfig, L: Optional[int] = None) -> torch.Tensor:
    """G [L, D] float32 on the CPU: float64 normals rounded to float32."""
    L = cfg.L if L is None else L
    g = _generator("cpu", cfg.seed, _TAG_G)
    return torch.randn(L, cfg.D, generator=g, dtype=torch.float64).to(torch.float32)


def _normals(shape, g, device) -> torch.Tensor:
    """float64 standard normals (host-independent on the CPU, see above)."""
    return torch.randn(shape, generator=g, device=device, dtype=torch.float64)


def _to_bf16(x: torch.Tensor) -> torch.Tensor:
    """float64 -> float32 (round to nearest even) -> bf16 (round to nearest even)."""
    return x.to(torch.float32).to(torch.bfloat16)


def _key_basis(cfg: DecodeConfig, layer: int, h: int, device):
    g = _generator(device, cfg.seed, _TAG_BASIS, layer, h)
    A = _normals((cfg.rank, cfg.D), g, device)
    perm = torch.randperm(cfg.D, generator=g, device=device)
    return A, perm[: cfg.n_outliers]


def make_query(cfg: DecodeConfig, layer: int = 0, device="cpu") -> torch.Tensor:
    g = _generator(device, cfg.seed, _TAG_QUERY, layer)
    return _to_bf16(_normals((cfg.B, cfg.Hq, cfg.D), g, device))


_CHUNK = 65536  # rows per independently seeded block of normals


def _rows_of_head(cfg: DecodeConfig, A: torch.Tensor, outl: torch.Tensor, layer: int, b: int, h: int,
                  c: int, device):
    """K and V rows [c * _CHUNK, ...) of one head, bf16.  Each block of rows
    has generators of its own, so blocks can be drawn in parallel."""
    rows = min(_CHUNK, cfg.N - c * _CHUNK)
    gk = _generator(device, cfg.seed, _TAG_KEYS, layer, b, h, c)
    Z = _normals((rows, cfg.rank), gk, device)
    K = _normals((rows, cfg.D), gk, device).mul_(cfg.noise)
    # K = noise E + Z A, the rank terms added in ascending order, each product
    # and sum rounded separately (no fused multiply-add, no BLAS)
    for r in range(cfg.rank):
        K.add_(Z[:, r:r + 1] * A[r])
    K[:, outl] *= cfg.outlier_scale
    gv = _generator(device, cfg.seed, _TAG_VALUES, layer, b, h, c)
    return _to_bf16(K), _to_bf16(_normals((rows, cfg.D), gv, device))


def make_head(cfg: DecodeConfig, q: torch.Tensor, layer: int, b: int, h: int,
              device="cpu", needle_mode: str = "rho", basis=None):
    """K, V [N, D] bf16 and needle positions for one (layer, sequence, KV head)."""
    A, outl = basis if basis is not None else _key_basis(cfg, layer, h, device)
    K = torch.empty(cfg.N, cfg.D, dtype=torch.bfloat16, device=device)
    V = torch.empty_like(K)
    nblk = (cfg.N + _CHUNK - 1) // _CHUNK

    def fill(c):
        Kc, Vc = _rows_of_head(cfg, A, outl, layer, b, h, c, device)
        K[c * _CHUNK:c * _CHUNK + Kc.shape[0]] = Kc
        V[c * _CHUNK:c * _CHUNK + Vc.shape[0]] = Vc

    if torch.device(device).type == "cpu" and nblk > 1:
        import concurrent.futures as cf
        with cf.ThreadPoolExecutor(max_workers=min(nblk, max(1, min(16, torch.get_num_threads())))) as ex:
            list(ex.map(fill, range(nblk)))
    else:
        for c in range(nblk):
            fill(c)
    pos = torch.empty(0, dtype=torch.int64, device=device)
    if cfg.needles > 0:
        gn = _generator(device, cfg.seed, _TAG_NEEDLE, layer, b, h)
        pos = torch.randperm(cfg.N, generator=gn, device=device)[: cfg.needles]
        Kf = K.double()
        rho = torch.sqrt((Kf * Kf).sum(dim=1).mean())
        Gq = cfg.G
        for j in range(cfg.needles):
            qg = q[b, h * Gq + (j % Gq)].double()
            unit = qg / torch.linalg.vector_norm(qg)
            if needle_mode == "rho":
                vec = 3.0 * rho * unit
            elif needle_mode == "literal":
                vec = 3.0 * unit
            elif needle_mode == "q3":
                vec = 3.0 * qg
            else:
                raise ValueError(needle_mode)
            K[pos[j]] = _to_bf16(vec)
    return K, V, pos


def make_layer(cfg: DecodeConfig, layer: int = 0, device="cpu",
               needle_mode: str = "rho", heads: Optional[Sequence[tuple]] = None,
               Ncap: Optional[int] = None):
    """One layer of the workload.

    Returns a dict with q [B, Hq, D], K and V [B, Hkv, Ncap, D] (bf16; rows
    at and beyond N are zero), G [L, D] float32 (CPU) and needle positions
    [B, Hkv, needles] int64.  `heads` restricts generation to a list of
    (b, h) pairs (the other heads stay zero), which lets a test regenerate a
    sample of a large configuration cheaply.
    """
    Ncap = cfg.N if Ncap is None else Ncap
    assert Ncap >= cfg.N
    q = make_query(cfg, layer, device)
    K = torch.zeros(cfg.B, cfg.Hkv, Ncap, cfg.D, dtype=torch.bfloat16, device=device)
    V = torch.zeros_like(K)
    pos = torch.zeros(cfg.B, cfg.Hkv, cfg.needles, dtype=torch.int64, device=device)
    todo = heads if heads is not None else [(b, h) for b in range(cfg.B) for h in range(cfg.Hkv)]
    bases = {}
    for b, h in todo:
        if h not in bases:
            bases[h] = _key_basis(cfg, layer, h, device)
        Kh, Vh, ph = make_head(cfg, q, layer, b, h, device, needle_mode, bases[h])
        K[b, h, : cfg.N] = Kh
        V[b, h, : cfg.N] = Vh
        if cfg.needles:
            pos[b, h] = ph
        del Kh, Vh
    return {"q": q, "K": K, "V": V, "G": make_gaussian_directions(cfg), "needle_pos": pos}


def make_calibration_keys(cfg: DecodeConfig, layer: int = 0, n_seq: int = 4, device="cpu") -> torch.Tensor:
    """Keys of n_seq held-out sequences of the same layer (sequence indices
    B .. B + n_seq - 1, so they share the layer's key basis but none of the
    batch's keys, and carry no needles), concatenated per KV head:
    [1, Hkv, n_seq * N, D] bf16.  They stand in for the calibration corpus
    of offline projection calibration."""
    c = cfg.replace(needles=0)
    K = torch.zeros(1, c.Hkv, n_seq * c.N, c.D, dtype=torch.bfloat16, device=device)
    q = torch.zeros(c.B + n_seq, c.Hq, c.D, dtype=torch.bfloat16, device=device)  # unused without needles
    for h in range(c.Hkv):
        basis = _key_basis(c, layer, h, device)
        for i in range(n_seq):
            Kh, _, _ = make_head(c, q, layer, c.B + i, h, device, basis=basis)
            K[0, h, i * c.N:(i + 1) * c.N] = Kh
    return K
