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
    "hash_keys",
    "decode_attention",
    "decode_workspace_bytes",
    "decode_attention_per_head",
    "decode_per_head_workspace_bytes",
    "dense_attention",
    "select_hard",
    "DECODE_STAGES",
    "DECODE_STAGE_NAMES",
    "version",
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
_lib.bpc_build_hash.restype = _i
_lib.bpc_build_hash.argtypes = [_p, _i64, _i64, _i64, _i, _i, _i, _i, _i, _p, _p, _p, _i64, _i64, _p, _p, _p, _sz, _p]
_lib.bpc_hash_keys.restype = _i
_lib.bpc_hash_keys.argtypes = [_p, _i64, _i64, _i64, _i, _i, _i, _i, _i, _p, _i64, _i64, _p, _i64, _i64, _p, _p, _p]
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
_lib.bpc_decode_attention_profiled.restype = _i
_lib.bpc_decode_attention_profiled.argtypes = _DECODE_ARGS + [ctypes.POINTER(_p), _i]

DECODE_STAGES = 3
DECODE_STAGE_NAMES = ("score", "attend", "merge")


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


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream or None


def _need(t: torch.Tensor, name: str, dtype, dim: int) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a GPU")
    if t.dim() != dim:
        raise ValueError(f"{name} must have {dim} dims, got shape {tuple(t.shape)}")
    if t.stride(-1) != 1:
        raise ValueError(f"{name}: innermost dimension must be contiguous")


def _kv_strides(t: torch.Tensor):
    return t.stride(0), t.stride(1), t.stride(2)


def _proj(P: torch.Tensor, D: int = 128):
    """(L, sP_b, sP_h) of a projection given as [B, Hkv, L, D] (one per
    (sequence, KV head)), [Hkv, L, D] (one per KV head, shared by the batch:
    offline calibration) or [L, D] (one for everything)."""
    if P.dtype != torch.float32 or P.device.type != "cuda":
        raise TypeError("P must be a float32 GPU tensor")
    if P.stride(-1) != 1 or P.shape[-1] != D or (P.dim() >= 2 and P.shape[-2] > 1 and P.stride(-2) != D):
        raise ValueError("P rows must be contiguous [.., L, 128]")
    if P.dim() == 2:
        return P.shape[0], 0, 0
    if P.dim() == 3:
        return P.shape[1], 0, P.stride(0)
    if P.dim() == 4:
        return P.shape[2], P.stride(0), P.stride(1)
    raise ValueError("P must be [B, Hkv, L, 128], [Hkv, L, 128] or [L, 128]")


def build_workspace_bytes(B: int, Hkv: int, N: int, L: int, D: int = 128) -> int:
    return int(_lib.bpc_build_workspace_bytes(B, Hkv, N, D, L))


def decode_workspace_bytes(B: int, Hq: int, Hkv: int, N: int, L: int, k: int, D: int = 128) -> int:
    return int(_lib.bpc_decode_workspace_bytes(B, Hq, Hkv, N, D, L, k))


def decode_per_head_workspace_bytes(B: int, Hq: int, Hkv: int, N: int, L: int, k: int, D: int = 128) -> int:
    return int(_lib.bpc_decode_per_head_workspace_bytes(B, Hq, Hkv, N, D, L, k))


def _u32_codes(codes: torch.Tensor, name: str = "codes") -> torch.Tensor:
    # torch has no uint32 arithmetic on every build; int32 storage is used and
    # reinterpreted by the library.
    if codes.dtype not in (torch.int32, torch.uint32):
        raise TypeError(f"{name} must be int32/uint32 storage")
    return codes


def build_hash(K: torch.Tensor, G: torch.Tensor, N: Optional[int] = None, *,
               P_out: Optional[torch.Tensor] = None, codes_out: Optional[torch.Tensor] = None,
               err_out: Optional[torch.Tensor] = None, fragile: Optional[torch.Tensor] = None,
               workspace: Optional[torch.Tensor] = None, stream=None):
    """Binary principal components of every (b, h): returns (P, codes, err).

    K [B, Hkv, >=N, 128] bf16; G [L, 128] fp32 Gaussian directions.  codes
    are int32 storage [B, Hkv, Ncap, L/32] holding the packed bits.  When
    `fragile` (a 1-element int64 GPU tensor) is given, the number of fragile
    sign decisions is added to it."""
    _need(K, "K", torch.bfloat16, 4)
    B, Hkv, Ncap, D = K.shape
    N = Ncap if N is None else N
    _need(G, "G", torch.float32, 2)
    G = G.contiguous()
    L = G.shape[0]
    dev = K.device
    if P_out is None:
        P_out = torch.empty(B, Hkv, L, D, dtype=torch.float32, device=dev)
    if codes_out is None:
        codes_out = torch.zeros(B, Hkv, Ncap, max(1, L // 32), dtype=torch.int32, device=dev)
    _u32_codes(codes_out, "codes_out")
    ws_bytes = build_workspace_bytes(B, Hkv, N, L, D)
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
    Returns (codes, err)."""
    _need(K, "K", torch.bfloat16, 4)
    B, Hkv, Ncap, D = K.shape
    N = Ncap if N is None else N
    L, sPb, sPh = _proj(P, D)
    if codes_out is None:
        codes_out = torch.zeros(B, Hkv, Ncap, max(1, L // 32), dtype=torch.int32, device=K.device)
    _u32_codes(codes_out, "codes_out")
    _check(_lib.bpc_hash_keys(_ptr(K), *_kv_strides(K), B, Hkv, N, D, L, _ptr(P), sPb, sPh, _ptr(codes_out),
                              codes_out.stride(0), codes_out.stride(1), _ptr(err_out), _ptr(fragile),
                              _stream(stream)),
           "bpc_hash_keys")
    return codes_out, err_out


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
    across the batch as [Hkv, L, 128] (offline calibration) or [L, 128].  Optional debug outputs: idx_out [B, Hkv, k] int32,
    score_out [B, Hkv, N] int32, qcode_out [B, Hkv, 8, L/32] int32.
    `events`: BPC_DECODE_STAGES + 1 torch.cuda.Event objects recorded at the
    stage boundaries (for measurement).

    With `serr` [B, Hkv, m] int32 (the hard-to-hash set from select_hard),
    attention runs over the union of the k hash-selected keys and serr (the
    error-aware safeguard); added_out [B, Hkv, m] int32 then marks the
    entries of serr that the hash selection had not taken."""
    _need(q, "q", torch.bfloat16, 3)
    _need(K, "K", torch.bfloat16, 4)
    _need(V, "V", torch.bfloat16, 4)
    if not q.is_contiguous():
        raise ValueError("q must be contiguous")
    B, Hq, D = q.shape
    _, Hkv, Ncap, _ = K.shape
    N = Ncap if N is None else N
    _u32_codes(codes)
    L, sPb, sPh = _proj(P, D)
    if sm_scale is None:
        sm_scale = 1.0 / math.sqrt(D)
    if out is None:
        out = torch.empty(B, Hq, D, dtype=torch.float32, device=q.device)
    ws_bytes = decode_workspace_bytes(B, Hq, Hkv, N, L, k, D)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=q.device)
    args = [_ptr(q), _ptr(K), *_kv_strides(K), _ptr(V), *_kv_strides(V), _ptr(codes), codes.stride(0),
            codes.stride(1), _ptr(P), sPb, sPh, B, Hq, Hkv, N, D, L, k, float(sm_scale), _ptr(out),
            _ptr(idx_out), _ptr(score_out), _ptr(qcode_out), _ptr(workspace), workspace.numel(),
            _stream(stream)]
    if serr is not None:
        if events is not None or score_out is not None or qcode_out is not None:
            raise ValueError("serr cannot be combined with events, score_out or qcode_out")
        if serr.dtype != torch.int32 or serr.dim() != 3 or serr.stride(-1) != 1 or serr.device != q.device:
            raise ValueError("serr must be a [B, Hkv, m] int32 tensor on the GPU, innermost dimension contiguous")
        m = serr.shape[-1]
        if added_out is not None and (added_out.dtype != torch.int32 or not added_out.is_contiguous()
                                      or tuple(added_out.shape) != (B, Hkv, m)):
            raise ValueError("added_out must be a contiguous [B, Hkv, m] int32 tensor")
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



def decode_attention_per_head(q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, codes: torch.Tensor,
                              P: torch.Tensor, k: int, sm_scale: Optional[float] = None, N: Optional[int] = None, *,
                              out: Optional[torch.Tensor] = None, idx_out: Optional[torch.Tensor] = None,
                              score_out: Optional[torch.Tensor] = None, qcode_out: Optional[torch.Tensor] = None,
                              workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """The decode step with one selection per query head: query head j
    quantises its own projection, scores the codes of KV head j // G, takes
    its own top-k and attends over it.  Shapes as decode_attention, except
    idx_out [B, Hq, k], score_out [B, Hq, N], qcode_out [B, Hq, 8, L/32]."""
    _need(q, "q", torch.bfloat16, 3)
    _need(K, "K", torch.bfloat16, 4)
    _need(V, "V", torch.bfloat16, 4)
    if not q.is_contiguous():
        raise ValueError("q must be contiguous")
    B, Hq, D = q.shape
    _, Hkv, Ncap, _ = K.shape
    N = Ncap if N is None else N
    _u32_codes(codes)
    L, sPb, sPh = _proj(P, D)
    if sm_scale is None:
        sm_scale = 1.0 / math.sqrt(D)
    if out is None:
        out = torch.empty(B, Hq, D, dtype=torch.float32, device=q.device)
    for t, name, shape in ((idx_out, "idx_out", (B, Hq, k)), (score_out, "score_out", (B, Hq, N)),
                           (qcode_out, "qcode_out", (B, Hq, 8, L // 32))):
        if t is not None and (t.dtype != torch.int32 or not t.is_contiguous() or tuple(t.shape) != shape):
            raise ValueError(f"{name} must be a contiguous int32 tensor of shape {shape}")
    ws_bytes = decode_per_head_workspace_bytes(B, Hq, Hkv, N, L, k, D)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=q.device)
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
    if serr_out is None:
        serr_out = torch.empty(B, Hkv, max(m, 0), dtype=torch.int32, device=err.device)
    elif serr_out.dtype != torch.int32 or not serr_out.is_contiguous() or tuple(serr_out.shape) != (B, Hkv, m):
        raise ValueError("serr_out must be a contiguous [B, Hkv, m] int32 tensor")
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
    rows of codes [B, Hkv, Ncap, L/32]."""
    for t, nm in ((k_new, "k_new"), (v_new, "v_new"), (K, "K"), (V, "V")):
        _need(t, nm, torch.bfloat16, 4)
    B, Hkv, T, D = k_new.shape
    if tuple(v_new.shape) != (B, Hkv, T, D):
        raise ValueError("v_new must have the shape of k_new")
    Ncap = K.shape[2]
    if tuple(K.shape[:2]) != (B, Hkv) or tuple(V.shape[:3]) != (B, Hkv, Ncap):
        raise ValueError("K and V must be [B, Hkv, Ncap, D] with the batch and heads of k_new")
    _u32_codes(codes)
    L, sPb, sPh = _proj(P, D)
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
