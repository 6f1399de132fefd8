"""The decode entry point that allocates nothing (bpc_decode_attention_noalloc,
through the C ABI) against the one with a caller workspace
(bpc_decode_attention): two calls in a row on the library's static scratch,
the second with a smaller input, each equal to the workspace call (same
kernels, so indices, scores, query planes and outputs are identical), and a
call too large for the scratch rejected before any launch.
"""

import numpy as np
import pytest
import torch

from workloads import config_by_name, make_layer

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2608_04405_amd as bpc
else:  # pragma: no cover
    bpc = None

DEV = "cuda"


def _inputs(cfg):
    d = make_layer(cfg, device=DEV)
    P, codes, _ = bpc.build_hash(d["K"], d["G"].to(DEV))
    return d, P, codes


def _both(cfg, d, P, codes, k):
    B, Hq, Hkv, N, L = cfg.B, cfg.Hq, cfg.Hkv, cfg.N, cfg.L
    res = []
    for noalloc in (False, True):
        out = torch.full((B, Hq, 128), float("nan"), device=DEV)
        idx = torch.full((B, Hkv, k), -1, dtype=torch.int32, device=DEV)
        sc = torch.full((B, Hkv, N), -1, dtype=torch.int32, device=DEV)
        qc = torch.full((B, Hkv, 8, L // 32), -1, dtype=torch.int32, device=DEV)
        if noalloc:
            bpc.decode_attention_noalloc(d["q"], d["K"], d["V"], codes, P, k, out, idx_out=idx, score_out=sc,
                                         qcode_out=qc)
        else:
            bpc.decode_attention(d["q"], d["K"], d["V"], codes, P, k, out=out, idx_out=idx, score_out=sc,
                                 qcode_out=qc)
        torch.cuda.synchronize()
        res.append((out, idx, sc, qc))
    return res


def test_noalloc_matches_workspace_call_twice():
    big = config_by_name("llama8b_32k").replace(B=2, N=40000)        # 3 slices per head, ragged
    small = config_by_name("tiny_mha_4k").replace(Hq=16, Hkv=4, N=3000)
    for cfg in (big, small):  # the second call smaller than the first, on the same scratch
        print(f"[no-alloc] {cfg.name} B={cfg.B} Hq={cfg.Hq} Hkv={cfg.Hkv} N={cfg.N} L={cfg.L} k={cfg.k}", flush=True)
        assert bpc.decode_workspace_bytes(cfg.B, cfg.Hq, cfg.Hkv, cfg.N, cfg.L, cfg.k) <= bpc.decode_noalloc_max_bytes()
        d, P, codes = _inputs(cfg)
        (o0, i0, s0, q0), (o1, i1, s1, q1) = _both(cfg, d, P, codes, cfg.k)
        assert torch.equal(i0, i1) and torch.equal(s0, s1) and torch.equal(q0, q1)
        assert torch.isfinite(o1).all()
        assert torch.equal(o0, o1)


def test_noalloc_rejects_a_call_beyond_the_scratch():
    # 2048 slices of 16384 keys: more workgroups than fit on the GPU at once,
    # so the three-launch path with its per-slice candidate areas (~200 MiB)
    cfg = config_by_name("batch16_128k").replace(N=262144)
    need = bpc.decode_workspace_bytes(cfg.B, cfg.Hq, cfg.Hkv, cfg.N, cfg.L, cfg.k)
    assert need > bpc.decode_noalloc_max_bytes()
    # the sizes alone decide: small stand-in tensors with the batch's extents
    q = torch.zeros(cfg.B, cfg.Hq, 128, dtype=torch.bfloat16, device=DEV)
    K = torch.zeros(1, 1, cfg.N, 128, dtype=torch.bfloat16, device=DEV).expand(cfg.B, cfg.Hkv, cfg.N, 128)
    codes = torch.zeros(1, 1, cfg.N, cfg.W, dtype=torch.int32, device=DEV).expand(cfg.B, cfg.Hkv, cfg.N, cfg.W)
    P = torch.zeros(cfg.Hkv, cfg.L, 128, device=DEV)
    out = torch.full((cfg.B, cfg.Hq, 128), 7.0, device=DEV)
    with pytest.raises(bpc.BPCError) as e:
        bpc.decode_attention_noalloc(q, K, K, codes, P, cfg.k, out)
    assert e.value.status == -4 and "static scratch" in str(e.value)
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)  # nothing launched
