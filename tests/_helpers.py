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
