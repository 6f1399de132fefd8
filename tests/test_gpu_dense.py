"""Dense decode attention (the full-attention comparison point) on the GPU
against the oracle's full attention (itself pinned to torch's scaled
dot-product attention): within 2e-3 relative error per row."""

import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2608_04405_amd as bpc
else:  # pragma: no cover
    bpc = None

DEV = "cuda"
TOL = 2e-3


def bits(t):
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


@pytest.mark.parametrize("B,Hq,Hkv,N,Ncap", [(1, 8, 8, 4096, 4096), (2, 32, 8, 20000, 20000), (1, 16, 1, 16385, 16400),
                                             (1, 2, 2, 1, 8), (1, 32, 4, 40000, 40000)])
def test_dense_matches_full_attention(B, Hq, Hkv, N, Ncap):
    print(f"[dense] B={B} Hq={Hq} Hkv={Hkv} N={N}", flush=True)
    rng = np.random.default_rng(N)
    q = torch.from_numpy(rng.standard_normal((B, Hq, 128)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    K = torch.from_numpy(3 * rng.standard_normal((B, Hkv, Ncap, 128)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    V = torch.from_numpy(rng.standard_normal((B, Hkv, Ncap, 128)).astype(np.float32)).to(torch.bfloat16).to(DEV)
    out = bpc.dense_attention(q, K, V, N=N)
    torch.cuda.synchronize()
    G = Hq // Hkv
    qb, Kb, Vb = bits(q), bits(K), bits(V)
    sm = 1.0 / np.sqrt(128)
    for b in range(B):
        for h in range(Hkv):
            ref = oracle.full_attention(qb[b, h * G:(h + 1) * G], Kb[b, h, :N], Vb[b, h, :N], sm)
            o = out[b, h * G:(h + 1) * G].cpu().numpy().astype(np.float64)
            e = np.max(np.abs(o - ref), axis=-1) / np.max(np.abs(ref), axis=-1)
            assert np.all(e <= TOL), f"output error {e.max():.3g} at {(b, h)}"
