"""BinaryPC decode hot path on AMD Instinct MI355X (gfx950).

A thin ctypes binding over libbpc.so (see include/bpc.h): it only checks
tensor metadata and marshals pointers, strides and the current HIP stream.
Every step of the computation runs in the library's HIP kernels; there is
no Python or CPU fallback.  Importing the package fails loudly when the
library has not been built (``python -m paper_2608_04405_amd.build_lib``).
"""

from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence

import torch

__all__ = [
    "BPCError",
    "append_kv",
    "LIB_PATH",
    "build_hash",
    "build_workspace_bytes",
    "build_checkpoint_workspace_bytes",
    "hash_keys",
    "hash_keys_mm",
    "decode_attention",
    "decode_workspace_bytes",
    "decode_attention_per_head",
    "decode_attention_noalloc",
    "decode_noalloc_max_bytes",
    "decode_per_head_workspace_bytes",
    "dense_attention",
    "select_hard",
    "DECODE_STAGES",
    "DECODE_STAGE_NAMES",
    "version",
    "set_decode_path",
    "decode_path_taken",
    "decode_slice_keys",
    "DECODE_ZEROED_BYTES",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libbpc.so")
if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2608_04405_amd.build_lib`")

_lib = ctypes.CDLL(LIB_PATH)

_p = ctypes.c_void_p
_i64 = ctypes.c_int64
_i = ctypes.c_int
_sz = ctypes.c_size_t

_lib.bpc_status_string.restype = ctypes.c_char_p
_lib.bpc_status_string.argtypes = [_i]
_lib.bpc_last_error.restype = ctypes.c_char_p
_lib.bpc_last_error.argtypes = []
_lib.bpc_version.restype = _i
_lib.bpc_build_workspace_bytes.restype = _sz
_lib.bpc_build_workspace_bytes.argtypes = [_i, _i, _i, _i, _i]
_lib.bpc_build_checkpoint_workspace_bytes.restype = _sz
_lib.bpc_build_checkpoint_workspace_bytes.argtypes = [_i, _i, _i, _i, _i]
_lib.bpc_build_hash.restype = _i
_lib.bpc_build_hash.argtypes = [_p, _i64, _i64, _i64, _i, _i, _i, _i, _i, _p, _p, _p, _i64, _i64, _p, _p, _p, _sz, _p]
_lib.bpc_hash_keys.restype = _i
_lib.bpc_hash_keys.argtypes = [_p, _i64, _i64, _i64, _i, _i, _i, _i, _i, _p, _i64, _i64, _p, _i64, _i64, _p, _p, _p]
_lib.bpc_hash_keys_mm.restype = _i
_lib.bpc_hash_keys_mm.argtypes = [_p, _i64, _i64, _i64, _i, _i, _i, _i, _i, _p, _i64, _i64, _p, _i64, _i64, _p, _p, _p]
_lib.bpc_decode_workspace_bytes.restype = _sz
_lib.bpc_decode_workspace_bytes.argtypes = [_i, _i, _i, _i, _i, _i, _i]
_DECODE_ARGS = [_p, _p, _i64, _i64, _i64, _p, _i64, _i64, _i64, _p, _i64, _i64, _p, _i64, _i64,
                _i, _i, _i, _i, _i, _i, _i, ctypes.c_float, _p, _p, _p, _p, _p, _sz, _p]
_lib.bpc_decode_attention.restype = _i
_lib.bpc_decode_attention.argtypes = _DECODE_ARGS
_lib.bpc_decode_per_head_workspace_bytes.restype = _sz
_lib.bpc_decode_per_head_workspace_bytes.argtypes = [_i, _i, _i, _i, _i, _i, _i]
_lib.bpc_decode_attention_per_head.restype = _i
_lib.bpc_decode_attention_per_head.argtypes = _DECODE_ARGS
_lib.bpc_decode_attention_eas.restype = _i
_lib.bpc_decode_attention_eas.argtypes = [_p, _p, _i64, _i64, _i64, _p, _i64, _i64, _i64, _p, _i64, _i64, _p, _i64, _i64,
                                          _i, _i, _i, _i, _i, _i, _i, ctypes.c_float, _p, _i64, _i64, _i, _p, _p, _p,
                                          _p, _sz, _p]
_lib.bpc_append_kv.restype = _i
_lib.bpc_append_kv.argtypes = [_p, _i64, _i64, _i64, _p, _i64, _i64, _i64, _p, _i64, _i64, _i64, _p, _i64, _i64, _i64,
                               _p, _i64, _i64, _p, _i64, _i64, _i, _i, _i, _i, _i, _i, _i, _p, _p, _p]
_lib.bpc_dense_workspace_bytes.restype = _sz
_lib.bpc_dense_workspace_bytes.argtypes = [_i, _i, _i, _i, _i]
_lib.bpc_dense_attention.restype = _i
_lib.bpc_dense_attention.argtypes = [_p, _p, _i64, _i64, _i64, _p, _i64, _i64, _i64, _i, _i, _i, _i, _i,
                                     ctypes.c_float, _p, _p, _sz, _p]
_lib.bpc_select_hard.restype = _i
_lib.bpc_select_hard.argtypes = [_p, _i64, _i64, _i, _i, _i, _i, _p, _p]
_lib.bpc_set_decode_path.restype = _i
_lib.bpc_set_decode_path.argtypes = [_i]
_lib.bpc_decode_slice_keys.restype = _i
_lib.bpc_decode_slice_keys.argtypes = [_i, _i, _i, _i, _i]
_lib.bpc_decode_path_taken.restype = _i
_lib.bpc_decode_path_taken.argtypes = [_i, _i, _i, _i, _i]
_lib.bpc_decode_noalloc_max_bytes.restype = _sz
_lib.bpc_decode_noalloc_max_bytes.argtypes = []
_lib.bpc_decode_attention_noalloc.restype = _i
_lib.bpc_decode_attention_noalloc.argtypes = _DECODE_ARGS[:-3] + [_p]
_lib.bpc_decode_attention_profiled.restype = _i
_lib.bpc_decode_attention_profiled.argtypes = _DECODE_ARGS + [ctypes.POINTER(_p), _i]

DECODE_STAGES = 3
DECODE_STAGE_NAMES = ("score", "attend", "merge")
# a decode workspace's leading bytes that must be zero before its first use
# (the fused path's arrival counters; every call leaves them zero)
DECODE_ZEROED_BYTES = 1088 * 1024


class BPCError(RuntimeError):
    def __init__(self, status: int, where: str):
        msg = _lib.bpc_status_string(status).decode()
        detail = _lib.bpc_last_error().decode()
        super().__init__(f"{where}: {msg} ({status}): {detail}")
        self.status = status


def _check(status: int, where: str) -> None:
    if status != 0:
        raise BPCError(status, where)


def version() -> int:
    return _lib.bpc_version()


def set_decode_path(path: int) -> None:
    """0: a decode step runs as one fused launch whenever its workgroups fit
    on the GPU at once (the default; 4096- or 8192-key slices where
    16384-key ones would leave the GPU mostly idle); 1: always the three
    launches; 2: the fused launch on 16384-key slices only."""
    _check(_lib.bpc_set_decode_path(int(path)), "bpc_set_decode_path")


def decode_path_taken(B: int, Hq: int, Hkv: int, N: int, L: int) -> int:
    """0 if a decode step of this shape runs as one fused launch on the
    current device, 1 if as three launches (needs a GPU)."""
    return int(_lib.bpc_decode_path_taken(B, Hq, Hkv, N, L))


def decode_slice_keys(B: int, Hq: int, Hkv: int, N: int, L: int) -> int:
    """Keys per slice (16384, 8192 or 4096) of a decode step of this shape on the
    current device (needs a GPU)."""
    return int(_lib.bpc_decode_slice_keys(B, Hq, Hkv, N, L))


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream or None


def _need(t: torch.Tensor, name: str, dtype, dim: int) -> None:
    """dtype, number of dims and a contiguous innermost dimension; the device
    is checked separately (`_on_gpu`), after every shape check, so that a
    shape mistake is reported as such wherever the tensors live."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.dim() != dim:
        raise ValueError(f"{name} must have {dim} dims, got shape {tuple(t.shape)}")
    if t.numel() and t.stride(-1) != 1:
        raise ValueError(f"{name}: innermost dimension must be contiguous")


def _extent(t: torch.Tensor, name: str, spec) -> None:
    """Check every extent of t against spec: an int is an exact size, ("ge",
    n) a lower bound (a cache with room for more rows), None anything."""
    shape = tuple(t.shape)
    if len(shape) != len(spec):
        raise ValueError(f"{name} must have {len(spec)} dims, got shape {shape}")
    for i, (got, want) in enumerate(zip(shape, spec)):
        if want is None:
            continue
        if isinstance(want, tuple):
            if got < want[1]:
                raise ValueError(f"{name}: dim {i} is {got}, needs at least {want[1]} (shape {shape})")
        elif got != want:
            raise ValueError(f"{name}: dim {i} is {got}, expected {want} (shape {shape})")


def _exact_out(t: Optional[torch.Tensor], name: str, dtype, shape) -> None:
    """An optional output the kernels address as a dense array of `shape`."""
    if t is None:
        return
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous tensor of shape {tuple(shape)}, got {tuple(t.shape)}")


def _on_gpu(*tensors) -> None:
    """Every given tensor (None entries skipped) on one GPU."""
    dev = None
    for t in tensors:
        if t is None:
            continue
        if t.device.type != "cuda":
            raise ValueError("every tensor must be on a GPU")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError(f"tensors on different devices: {dev} and {t.device}")


def _budget(k: int, N: int, Ncap: int) -> None:
    if not 1 <= N <= Ncap:
        raise ValueError(f"N={N} must satisfy 1 <= N <= {Ncap} (the rows the cache holds)")
    if not 1 <= k <= N:
        raise ValueError(f"k={k} must satisfy 1 <= k <= N={N}")


def _kv_strides(t: torch.Tensor):
    return t.stride(0), t.stride(1), t.stride(2)


def _proj(P: torch.Tensor, D: int = 128, B: Optional[int] = None, Hkv: Optional[int] = None):
    """(L, sP_b, sP_h) of a projection given as [B, Hkv, L, D] (one per
    (sequence, KV head)), [Hkv, L, D] (one per KV head, shared by the batch:
    offline calibration) or [L, D] (one for everything).  When B and Hkv are
    given, the leading dims must match them."""
    if not isinstance(P, torch.Tensor) or P.dtype != torch.float32:
        raise TypeError("P must be a float32 tensor")
    if P.dim() not in (2, 3, 4):
        raise ValueError("P must be [B, Hkv, L, 128], [Hkv, L, 128] or [L, 128]")
    if P.stride(-1) != 1 or P.shape[-1] != D or (P.shape[-2] > 1 and P.stride(-2) != D):
        raise ValueError("P rows must be contiguous [.., L, 128]")
    L = P.shape[-2]
    if L not in (32, 64, 128):
        raise ValueError(f"P has {L} rows: the code length must be 32, 64 or 128")
    if P.dim() == 3 and Hkv is not None and P.shape[0] != Hkv:
        raise ValueError(f"P is [Hkv, L, 128] with {P.shape[0]} heads, expected Hkv={Hkv}")
    if P.dim() == 4 and B is not None and (P.shape[0], P.shape[1]) != (B, Hkv):
        raise ValueError(f"P is {tuple(P.shape)}, expected [{B}, {Hkv}, L, 128]")
    if P.dim() == 2:
        return L, 0, 0
    if P.dim() == 3:
        return L, 0, P.stride(0)
    return L, P.stride(0), P.stride(1)


def build_workspace_bytes(B: int, Hkv: int, N: int, L: int, D: int = 128) -> int:
    return int(_lib.bpc_build_workspace_bytes(B, Hkv, N, D, L))


def build_checkpoint_workspace_bytes(B: int, Hkv: int, N: int, L: int, D: int = 128) -> int:
    return int(_lib.bpc_build_checkpoint_workspace_bytes(B, Hkv, N, D, L))


def decode_workspace_bytes(B: int, Hq: int, Hkv: int, N: int, L: int, k: int, D: int = 128) -> int:
    return int(_lib.bpc_decode_workspace_bytes(B, Hq, Hkv, N, D, L, k))


def decode_per_head_workspace_bytes(B: int, Hq: int, Hkv: int, N: int, L: int, k: int, D: int = 128) -> int:
    return int(_lib.bpc_decode_per_head_workspace_bytes(B, Hq, Hkv, N, D, L, k))


def _u32_codes(codes: torch.Tensor, name: str = "codes") -> torch.Tensor:
    # torch has no uint32 arithmetic on every build; int32 storage is used and
    # reinterpreted by the library.
    if not isinstance(codes, torch.Tensor) or codes.dtype not in (torch.int32, torch.uint32):
        raise TypeError(f"{name} must be int32/uint32 storage")
    if codes.dim() != 4 or (codes.numel() and codes.stride(-1) != 1) or (codes.shape[2] > 1 and codes.stride(2) != codes.shape[3]):
        raise ValueError(f"{name} must be [B, Hkv, Ncap, L/32] with the words of a key and the keys of a head contiguous")
    return codes


def _fragile(fragile: Optional[torch.Tensor]) -> None:
    if fragile is not None and (fragile.dtype != torch.int64 or fragile.numel() < 1):
        raise ValueError("fragile must be an int64 tensor with at least one element")


def build_hash(K: torch.Tensor, G: torch.Tensor, N: Optional[int] = None, *,
               P_out: Optional[torch.Tensor] = None, codes_out: Optional[torch.Tensor] = None,
               err_out: Optional[torch.Tensor] = None, fragile: Optional[torch.Tensor] = None,
               workspace: Optional[torch.Tensor] = None, checkpoint: bool = False, stream=None):
    """Binary principal components of every (b, h): returns (P, codes, err).

    K [B, Hkv, >=N, 128] bf16; G [L, 128] fp32 Gaussian directions.  codes
    are int32 storage [B, Hkv, Ncap, L/32] holding the packed bits; err_out,
    when given, is a contiguous [B, Hkv, N] fp32 tensor.  When `fragile` (a
    1-element int64 GPU tensor) is given, the number of fragile sign
    decisions is added to it.  With `checkpoint` the workspace allocated
    here also holds the fp64 residual checkpoint (1 KiB per key); a given
    workspace enables it by its size alone.  Results are the same."""
    _need(K, "K", torch.bfloat16, 4)
    B, Hkv, Ncap, D = K.shape
    N = Ncap if N is None else N
    if not 1 <= N <= Ncap:
        raise ValueError(f"N={N} must satisfy 1 <= N <= {Ncap}")
    _need(G, "G", torch.float32, 2)
    L = G.shape[0]
    _extent(G, "G", (L, D))
    if L not in (32, 64, 128):
        raise ValueError(f"G has {L} rows: the code length must be 32, 64 or 128")
    G = G.contiguous()
    W = L // 32
    if P_out is not None:
        _exact_out(P_out, "P_out", torch.float32, (B, Hkv, L, D))
    if codes_out is not None:
        _u32_codes(codes_out, "codes_out")
        _extent(codes_out, "codes_out", (B, Hkv, ("ge", N), W))
    _exact_out(err_out, "err_out", torch.float32, (B, Hkv, N))
    _fragile(fragile)
    _on_gpu(K, G, P_out, codes_out, err_out, fragile, workspace)
    dev = K.device
    if P_out is None:
        P_out = torch.empty(B, Hkv, L, D, dtype=torch.float32, device=dev)
    if codes_out is None:
        codes_out = torch.zeros(B, Hkv, Ncap, W, dtype=torch.int32, device=dev)
    ws_bytes = (build_checkpoint_workspace_bytes if checkpoint else build_workspace_bytes)(B, Hkv, N, L, D)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    _check(_lib.bpc_build_hash(_ptr(K), *_kv_strides(K), B, Hkv, N, D, L, _ptr(G), _ptr(P_out),
                               _ptr(codes_out), codes_out.stride(0), codes_out.stride(1), _ptr(err_out),
                               _ptr(fragile), _ptr(workspace), workspace.numel(), _stream(stream)),
           "bpc_build_hash")
    return P_out, codes_out, err_out


def hash_keys(K: torch.Tensor, P: torch.Tensor, N: Optional[int] = None, *,
              codes_out: Optional[torch.Tensor] = None, err_out: Optional[torch.Tensor] = None,
              fragile: Optional[torch.Tensor] = None, stream=None):
    """Hash keys against P (Algorithm 2).  P is [B, Hkv, L, 128], or
    [Hkv, L, 128] / [L, 128] shared across the batch (offline calibration).
    err_out, when given, is a contiguous [B, Hkv, N] fp32 tensor.  Returns
    (codes, err)."""
    _need(K, "K", torch.bfloat16, 4)
    B, Hkv, Ncap, D = K.shape
    N = Ncap if N is None else N
    if not 1 <= N <= Ncap:
        raise ValueError(f"N={N} must satisfy 1 <= N <= {Ncap}")
    L, sPb, sPh = _proj(P, D, B, Hkv)
    if codes_out is not None:
        _u32_codes(codes_out, "codes_out")
        _extent(codes_out, "codes_out", (B, Hkv, ("ge", N), L // 32))
    _exact_out(err_out, "err_out", torch.float32, (B, Hkv, N))
    _fragile(fragile)
    _on_gpu(K, P, codes_out, err_out, fragile)
    if codes_out is None:
        codes_out = torch.zeros(B, Hkv, Ncap, L // 32, dtype=torch.int32, device=K.device)
    _check(_lib.bpc_hash_keys(_ptr(K), *_kv_strides(K), B, Hkv, N, D, L, _ptr(P), sPb, sPh, _ptr(codes_out),
                              codes_out.stride(0), codes_out.stride(1), _ptr(err_out), _ptr(fragile),
                              _stream(stream)),
           "bpc_hash_keys")
    return codes_out, err_out


def hash_keys_mm(K: torch.Tensor, P: torch.Tensor, N: Optional[int] = None, *,
                 codes_out: Optional[torch.Tensor] = None, fragile: Optional[torch.Tensor] = None,
                 fallbacks: Optional[torch.Tensor] = None, stream=None):
    """The codes of hash_keys (Algorithm 2), bit for bit, with the
    projections on the matrix cores and certified signs.  fragile and
    fallbacks are device uint64 accumulators ([1] int64 tensors).  Returns
    codes."""
    _need(K, "K", torch.bfloat16, 4)
    B, Hkv, Ncap, D = K.shape
    N = Ncap if N is None else N
    if not 1 <= N <= Ncap:
        raise ValueError(f"N={N} must satisfy 1 <= N <= {Ncap}")
    L, sPb, sPh = _proj(P, D, B, Hkv)
    if codes_out is not None:
        _u32_codes(codes_out, "codes_out")
        _extent(codes_out, "codes_out", (B, Hkv, ("ge", N), L // 32))
    _fragile(fragile)
    _fragile(fallbacks)
    _on_gpu(K, P, codes_out, fragile, fallbacks)
    if codes_out is None:
        codes_out = torch.zeros(B, Hkv, Ncap, L // 32, dtype=torch.int32, device=K.device)
    _check(_lib.bpc_hash_keys_mm(_ptr(K), *_kv_strides(K), B, Hkv, N, D, L, _ptr(P), sPb, sPh, _ptr(codes_out),
                                 codes_out.stride(0), codes_out.stride(1), _ptr(fragile), _ptr(fallbacks),
                                 _stream(stream)),
           "bpc_hash_keys_mm")
    return codes_out


def _decode_inputs(q, K, V, codes, P, k, N):
    """Shape checks shared by the decode entry points; returns the sizes."""
    _need(q, "q", torch.bfloat16, 3)
    _need(K, "K", torch.bfloat16, 4)
    _need(V, "V", torch.bfloat16, 4)
    if not q.is_contiguous():
        raise ValueError("q must be contiguous")
    B, Hq, D = q.shape
    _, Hkv, Ncap, _ = K.shape
    N = Ncap if N is None else N
    _extent(K, "K", (B, Hkv, ("ge", 1), D))
    _budget(k, N, Ncap)
    _extent(V, "V", (B, Hkv, ("ge", N), D))
    if Hq % Hkv:
        raise ValueError(f"Hq={Hq} must be a multiple of Hkv={Hkv}")
    L, sPb, sPh = _proj(P, D, B, Hkv)
    _u32_codes(codes)
    _extent(codes, "codes", (B, Hkv, ("ge", N), L // 32))
    return B, Hq, Hkv, D, N, L, sPb, sPh


def decode_attention(q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, codes: torch.Tensor,
                     P: torch.Tensor, k: int, sm_scale: Optional[float] = None, N: Optional[int] = None, *,
                     out: Optional[torch.Tensor] = None, idx_out: Optional[torch.Tensor] = None,
                     score_out: Optional[torch.Tensor] = None, qcode_out: Optional[torch.Tensor] = None,
                     serr: Optional[torch.Tensor] = None, added_out: Optional[torch.Tensor] = None,
                     workspace: Optional[torch.Tensor] = None, stream=None,
                     events: Optional[Sequence] = None) -> torch.Tensor:
    """One BinaryPC decode step; returns out [B, Hq, 128] fp32.

    q [B, Hq, 128] bf16 contiguous; K, V [B, Hkv, >=N, 128] bf16; codes
    int32 storage [B, Hkv, >=N, L/32]; P [B, Hkv, L, 128] fp32, or shared
    across the batch as [Hkv, L, 128] (offline calibration) or [L, 128].
    Optional debug outputs (contiguous): idx_out [B, Hkv, k] int32,
    score_out [B, Hkv, N] int32, qcode_out [B, Hkv, 8, L/32] int32.
    `events`: BPC_DECODE_STAGES + 1 torch.cuda.Event objects recorded at the
    stage boundaries (for measurement).

    With `serr` [B, Hkv, m] int32 (the hard-to-hash set from select_hard),
    attention runs over the union of the k hash-selected keys and serr (the
    error-aware safeguard); added_out [B, Hkv, m] int32 then marks the
    entries of serr that the hash selection had not taken."""
    B, Hq, Hkv, D, N, L, sPb, sPh = _decode_inputs(q, K, V, codes, P, k, N)
    _exact_out(out, "out", torch.float32, (B, Hq, D))
    _exact_out(idx_out, "idx_out", torch.int32, (B, Hkv, k))
    _exact_out(score_out, "score_out", torch.int32, (B, Hkv, N))
    _exact_out(qcode_out, "qcode_out", torch.int32, (B, Hkv, 8, L // 32))
    m = 0
    if serr is not None:
        if events is not None or score_out is not None or qcode_out is not None:
            raise ValueError("serr cannot be combined with events, score_out or qcode_out")
        if not isinstance(serr, torch.Tensor) or serr.dtype != torch.int32 or serr.dim() != 3 or \
                (serr.numel() and serr.stride(-1) != 1):
            raise ValueError("serr must be a [B, Hkv, m] int32 tensor, innermost dimension contiguous")
        _extent(serr, "serr", (B, Hkv, None))
        m = serr.shape[-1]
        if m > N:
            raise ValueError(f"serr holds m={m} keys per head, more than N={N}")
        _exact_out(added_out, "added_out", torch.int32, (B, Hkv, m))
    elif added_out is not None:
        raise ValueError("added_out needs serr")
    if workspace is not None and (workspace.dtype != torch.uint8 or not workspace.is_contiguous()):
        raise ValueError("workspace must be a contiguous uint8 tensor")
    _on_gpu(q, K, V, codes, P, out, idx_out, score_out, qcode_out, serr, added_out, workspace)
    if sm_scale is None:
        sm_scale = 1.0 / math.sqrt(D)
    if out is None:
        out = torch.empty(B, Hq, D, dtype=torch.float32, device=q.device)
    ws_bytes = decode_workspace_bytes(B, Hq, Hkv, N, L, k, D)
    if workspace is None:
        workspace = torch.zeros(max(ws_bytes, 1), dtype=torch.uint8, device=q.device)
    args = [_ptr(q), _ptr(K), *_kv_strides(K), _ptr(V), *_kv_strides(V), _ptr(codes), codes.stride(0),
            codes.stride(1), _ptr(P), sPb, sPh, B, Hq, Hkv, N, D, L, k, float(sm_scale), _ptr(out),
            _ptr(idx_out), _ptr(score_out), _ptr(qcode_out), _ptr(workspace), workspace.numel(),
            _stream(stream)]
    if serr is not None:
        _check(_lib.bpc_decode_attention_eas(*args[:23], _ptr(serr), serr.stride(0), serr.stride(1), m, _ptr(out),
                                             _ptr(idx_out), _ptr(added_out), _ptr(workspace), workspace.numel(),
                                             _stream(stream)),
               "bpc_decode_attention_eas")
    elif events is None:
        _check(_lib.bpc_decode_attention(*args), "bpc_decode_attention")
    else:
        handles = (_p * len(events))()
        st = torch.cuda.current_stream() if stream is None else stream
        for i, ev in enumerate(events):
            if ev.cuda_event == 0:  # torch creates the event lazily on first record
                ev.record(st)
            handles[i] = ev.cuda_event
        _check(_lib.bpc_decode_attention_profiled(*args, handles, len(events)), "bpc_decode_attention_profiled")
    return out


def decode_noalloc_max_bytes() -> int:
    """Size of the library's static decode scratch (the limit of
    decode_attention_noalloc)."""
    return int(_lib.bpc_decode_noalloc_max_bytes())


def decode_attention_noalloc(q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, codes: torch.Tensor,
                             P: torch.Tensor, k: int, out: torch.Tensor, sm_scale: Optional[float] = None,
                             N: Optional[int] = None, *, idx_out: Optional[torch.Tensor] = None,
                             score_out: Optional[torch.Tensor] = None, qcode_out: Optional[torch.Tensor] = None,
                             stream=None) -> torch.Tensor:
    """decode_attention with the library's static scratch as the workspace:
    the call allocates no device memory (the caller passes `out`).  Calls on
    one GPU share the scratch, so calls that overlap in time race."""
    B, Hq, Hkv, D, N, L, sPb, sPh = _decode_inputs(q, K, V, codes, P, k, N)
    if out is None:
        raise ValueError("out is required (the call allocates nothing)")
    _exact_out(out, "out", torch.float32, (B, Hq, D))
    _exact_out(idx_out, "idx_out", torch.int32, (B, Hkv, k))
    _exact_out(score_out, "score_out", torch.int32, (B, Hkv, N))
    _exact_out(qcode_out, "qcode_out", torch.int32, (B, Hkv, 8, L // 32))
    _on_gpu(q, K, V, codes, P, out, idx_out, score_out, qcode_out)
    if sm_scale is None:
        sm_scale = 1.0 / math.sqrt(D)
    _check(_lib.bpc_decode_attention_noalloc(
        _ptr(q), _ptr(K), *_kv_strides(K), _ptr(V), *_kv_strides(V), _ptr(codes), codes.stride(0), codes.stride(1),
        _ptr(P), sPb, sPh, B, Hq, Hkv, N, D, L, k, float(sm_scale), _ptr(out), _ptr(idx_out), _ptr(score_out),
        _ptr(qcode_out), _stream(stream)), "bpc_decode_attention_noalloc")
    return out


def decode_attention_per_head(q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, codes: torch.Tensor,
                              P: torch.Tensor, k: int, sm_scale: Optional[float] = None, N: Optional[int] = None, *,
                              out: Optional[torch.Tensor] = None, idx_out: Optional[torch.Tensor] = None,
                              score_out: Optional[torch.Tensor] = None, qcode_out: Optional[torch.Tensor] = None,
                              workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """The decode step with one selection per query head: query head j
    quantises its own projection, scores the codes of KV head j // G, takes
    its own top-k and attends over it.  Shapes as decode_attention, except
    idx_out [B, Hq, k], score_out [B, Hq, N], qcode_out [B, Hq, 8, L/32]."""
    B, Hq, Hkv, D, N, L, sPb, sPh = _decode_inputs(q, K, V, codes, P, k, N)
    _exact_out(out, "out", torch.float32, (B, Hq, D))
    _exact_out(idx_out, "idx_out", torch.int32, (B, Hq, k))
    _exact_out(score_out, "score_out", torch.int32, (B, Hq, N))
    _exact_out(qcode_out, "qcode_out", torch.int32, (B, Hq, 8, L // 32))
    if workspace is not None and (workspace.dtype != torch.uint8 or not workspace.is_contiguous()):
        raise ValueError("workspace must be a contiguous uint8 tensor")
    _on_gpu(q, K, V, codes, P, out, idx_out, score_out, qcode_out, workspace)
    if sm_scale is None:
        sm_scale = 1.0 / math.sqrt(D)
    if out is None:
        out = torch.empty(B, Hq, D, dtype=torch.float32, device=q.device)
    ws_bytes = decode_per_head_workspace_bytes(B, Hq, Hkv, N, L, k, D)
    if workspace is None:
        workspace = torch.zeros(max(ws_bytes, 1), dtype=torch.uint8, device=q.device)
    _check(_lib.bpc_decode_attention_per_head(
        _ptr(q), _ptr(K), *_kv_strides(K), _ptr(V), *_kv_strides(V), _ptr(codes), codes.stride(0), codes.stride(1),
        _ptr(P), sPb, sPh, B, Hq, Hkv, N, D, L, k, float(sm_scale), _ptr(out), _ptr(idx_out), _ptr(score_out),
        _ptr(qcode_out), _ptr(workspace), workspace.numel(), _stream(stream)), "bpc_decode_attention_per_head")
    return out


def select_hard(err: torch.Tensor, m: int, N: Optional[int] = None, *, serr_out: Optional[torch.Tensor] = None,
                stream=None) -> torch.Tensor:
    """The error-aware safeguard's hard-to-hash set: per (b, KV head), the m
    keys with the largest reconstruction errors (err [B, Hkv, >=N] fp32, as
    written by build_hash / hash_keys), ascending; returns [B, Hkv, m] int32."""
    _need(err, "err", torch.float32, 3)
    B, Hkv, Ncap = err.shape
    N = Ncap if N is None else N
    if not 1 <= N <= Ncap:
        raise ValueError(f"N={N} must satisfy 1 <= N <= {Ncap}")
    if not 0 <= m <= N:
        raise ValueError(f"m={m} must satisfy 0 <= m <= N={N}")
    _exact_out(serr_out, "serr_out", torch.int32, (B, Hkv, m))
    _on_gpu(err, serr_out)
    if serr_out is None:
        serr_out = torch.empty(B, Hkv, m, dtype=torch.int32, device=err.device)
    _check(_lib.bpc_select_hard(_ptr(err), err.stride(0), err.stride(1), B, Hkv, N, m, _ptr(serr_out),
                                _stream(stream)),
           "bpc_select_hard")
    return serr_out


def append_kv(k_new: torch.Tensor, v_new: torch.Tensor, K: torch.Tensor, V: torch.Tensor, codes: torch.Tensor,
              P: torch.Tensor, pos: int, *, err_out: Optional[torch.Tensor] = None,
              fragile: Optional[torch.Tensor] = None, stream=None) -> None:
    """Decode-time append: store k_new, v_new [B, Hkv, T, 128] bf16 at rows
    [pos, pos + T) of the caches K, V [B, Hkv, Ncap, 128] and their codes
    (Algorithm 2 against P, [B, Hkv, L, 128] or a shared [L, 128]) at the same
    rows of codes [B, Hkv, Ncap, L/32].  err_out, when given, is a
    contiguous [B, Hkv, T] fp32 tensor."""
    for t, nm in ((k_new, "k_new"), (v_new, "v_new"), (K, "K"), (V, "V")):
        _need(t, nm, torch.bfloat16, 4)
    B, Hkv, T, D = k_new.shape
    _extent(v_new, "v_new", (B, Hkv, T, D))
    Ncap = K.shape[2]
    _extent(K, "K", (B, Hkv, Ncap, D))
    _extent(V, "V", (B, Hkv, ("ge", Ncap), D))
    if T < 1 or pos < 0 or pos + T > Ncap:
        raise ValueError(f"pos={pos}, T={T}: the new rows must lie within the {Ncap} cache rows")
    L, sPb, sPh = _proj(P, D, B, Hkv)
    _u32_codes(codes)
    _extent(codes, "codes", (B, Hkv, ("ge", pos + T), L // 32))
    _exact_out(err_out, "err_out", torch.float32, (B, Hkv, T))
    _fragile(fragile)
    _on_gpu(k_new, v_new, K, V, codes, P, err_out, fragile)
    _check(_lib.bpc_append_kv(_ptr(k_new), *_kv_strides(k_new), _ptr(v_new), *_kv_strides(v_new), _ptr(K),
                              *_kv_strides(K), _ptr(V), *_kv_strides(V), _ptr(codes), codes.stride(0),
                              codes.stride(1), _ptr(P), sPb, sPh, B, Hkv, Ncap, pos, T, D, L, _ptr(err_out),
                              _ptr(fragile), _stream(stream)),
           "bpc_append_kv")


def dense_attention(q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, sm_scale: Optional[float] = None,
                    N: Optional[int] = None, *, out: Optional[torch.Tensor] = None,
                    workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Dense decode attention over all N cached keys (the comparison point
    for the sparse step); returns out [B, Hq, 128] fp32."""
    _need(q, "q", torch.bfloat16, 3)
    _need(K, "K", torch.bfloat16, 4)
    _need(V, "V", torch.bfloat16, 4)
    if not q.is_contiguous():
        raise ValueError("q must be contiguous")
    B, Hq, D = q.shape
    _, Hkv, Ncap, _ = K.shape
    N = Ncap if N is None else N
    _extent(K, "K", (B, Hkv, ("ge", N), D))
    _extent(V, "V", (B, Hkv, ("ge", N), D))
    if not 1 <= N or Hq % Hkv:
        raise ValueError(f"N={N} must be >= 1 and Hq={Hq} a multiple of Hkv={Hkv}")
    _exact_out(out, "out", torch.float32, (B, Hq, D))
    _on_gpu(q, K, V, out, workspace)
    if sm_scale is None:
        sm_scale = 1.0 / math.sqrt(D)
    if out is None:
        out = torch.empty(B, Hq, D, dtype=torch.float32, device=q.device)
    need = int(_lib.bpc_dense_workspace_bytes(B, Hq, Hkv, N, D))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    _check(_lib.bpc_dense_attention(_ptr(q), _ptr(K), *_kv_strides(K), _ptr(V), *_kv_strides(V), B, Hq, Hkv, N, D,
                                    float(sm_scale), _ptr(out), _ptr(workspace), workspace.numel(), _stream(stream)),
           "bpc_dense_attention")
    return out
