"""Small helpers for the tests (no method arithmetic lives here)."""

import numpy as np
import torch


def to_bf16_bits(x) -> np.ndarray:
    """Round float values to bf16 with torch and return the uint16 patterns."""
    t = torch.as_tensor(np.asarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def bits_of(t: torch.Tensor) -> np.ndarray:
    """bf16 torch tensor -> uint16 numpy bit patterns (copied to host)."""
    return t.detach().to("cpu").contiguous().view(torch.int16).numpy().view(np.uint16).copy()


def bf16_values(bits) -> np.ndarray:
    """uint16 bf16 patterns -> float64 values via torch's own conversion."""
    b = np.ascontiguousarray(np.asarray(bits, dtype=np.uint16))
    return torch.from_numpy(b.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()


def random_bf16(rng, shape, scale=1.0) -> np.ndarray:
    return to_bf16_bits(rng.standard_normal(shape) * scale)


def popcount32(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.uint32)
    return np.bitwise_count(x).astype(np.int64)


def fp32_ulp(x: np.ndarray) -> np.ndarray:
    x = np.abs(np.asarray(x, dtype=np.float32))
    return np.spacing(x).astype(np.float64)


def oracle_build_of(P_dev, codes_dev, K_dev, G_dev, heads, N=None):
    """The oracle side of a GPU Algorithm 1 build.

    Runs the oracle's own build on the keys of every (b, h) in `heads`,
    checks that the GPU build (P_dev [B, Hkv, L, 128], codes_dev
    [B, Hkv, >= N, W]) equals it bit for bit, and returns host copies
    (P, codes) in which those heads hold the oracle's values, with the
    oracle's reconstruction errors {(b, h): float64 [N]}.  A parity test
    whose oracle side reads only these heads feeds the oracle nothing that
    the GPU computed."""
    import oracle  # only the GPU tests call this

    Pn = P_dev.detach().to("cpu").contiguous().numpy().copy()
    cn = codes_dev.detach().to("cpu").contiguous().numpy().view(np.uint32).copy()
    Kb = bits_of(K_dev)
    Gn = G_dev.detach().to("cpu").numpy()
    N = Kb.shape[2] if N is None else N
    errs = {}
    for b, h in heads:
        print(f"  oracle build of head {(b, h)} over {N} keys", flush=True)
        Po, co, eo, _ = oracle.build_binary_pcs(Kb[b, h, :N], Gn)
        assert np.array_equal(Pn[b, h], Po), f"projection differs at {(b, h)}"
        assert np.array_equal(cn[b, h, :N], co), f"codes differ at {(b, h)}"
        Pn[b, h], cn[b, h, :N] = Po, co
        errs[(b, h)] = eo
    return Pn, cn, errs
