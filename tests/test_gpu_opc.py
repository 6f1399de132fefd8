"""Offline projection calibration (OPC) on the GPU against the oracle.

OPC (Sec. 3.2, "Offline Projection Calibration") computes P once per KV
head with Algorithm 1 over keys of a calibration set, and every sequence
then hashes its keys against that shared P (Algorithm 2).  The calibration
corpus of the paper is not available; keys of held-out synthetic sequences
of the same layer stand in for it.  Checked: the calibrated P bit for bit,
the batch's codes under the shared P bit for bit, and a decode step that
reads the shared P (zero batch stride) against the oracle.  Recall of the
planted needles, which the calibration keys never contain, is reported.
"""

import numpy as np
import pytest
import torch

import oracle
from workloads import CONFIGS, make_calibration_keys, make_layer

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2608_04405_amd as bpc
else:  # pragma: no cover
    bpc = None

DEV = "cuda"
TOL = 2e-3


def bits(t):
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def u32(t):
    return t.detach().cpu().contiguous().numpy().view(np.uint32)


def rel_err(o, ref):
    o = np.asarray(o, np.float64)
    return np.max(np.abs(o - ref), axis=-1) / np.max(np.abs(ref), axis=-1)


def announce(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("name,B,N,n_cal", [("tiny_mha_4k", 2, 4096, 3), ("llama8b_32k", 2, 6000, 2)])
def test_opc_calibrate_hash_decode(name, B, N, n_cal):
    cfg = next(c for c in CONFIGS if c.name == name).replace(B=B, N=N)
    announce(f"[opc] {cfg} calibration sequences {n_cal}")
    d = make_layer(cfg, device=DEV)
    Kcal = make_calibration_keys(cfg, n_seq=n_cal, device=DEV)
    G = d["G"].to(DEV)
    # calibration: Algorithm 1 over the held-out keys, one P per KV head
    Pcal = bpc.build_hash(Kcal, G)[0][0]  # [Hkv, L, 128]
    # prefill under OPC: Algorithm 2 of every sequence's keys against the shared P
    codes, _ = bpc.hash_keys(d["K"], Pcal)
    idx = torch.empty(cfg.B, cfg.Hkv, cfg.k, dtype=torch.int32, device=DEV)
    out = bpc.decode_attention(d["q"], d["K"], d["V"], codes, Pcal, cfg.k, idx_out=idx)
    torch.cuda.synchronize()
    sm = 1.0 / np.sqrt(cfg.D)
    Gn = d["G"].numpy()
    Kb, Vb, qb, cn = bits(d["K"]), bits(d["V"]), bits(d["q"]), u32(codes)
    for h in range(cfg.Hkv):
        P_ref = oracle.build_binary_pcs(bits(Kcal[0, h]), Gn)[0]
        assert np.array_equal(Pcal[h].cpu().numpy(), P_ref), f"calibrated P differs at head {h}"
        for b in range(cfg.B):
            c_ref, _, _ = oracle.hash_keys(Kb[b, h], P_ref)
            assert np.array_equal(cn[b, h], c_ref), f"codes under the shared P differ at {(b, h)}"
            ref = oracle.decode_head(qb[b, h * cfg.G:(h + 1) * cfg.G], Kb[b, h], Vb[b, h], c_ref, P_ref, cfg.k, sm)
            assert np.array_equal(idx[b, h].cpu().numpy(), ref["idx"]), f"indices differ at {(b, h)}"
            e = rel_err(out[b, h * cfg.G:(h + 1) * cfg.G].cpu().numpy(), ref["out"])
            assert np.all(e <= TOL), f"output error {e.max():.3g} at {(b, h)}"
    # method quality, reported (not parity): recall of the batch's planted
    # needles under the calibrated projection, which never saw them
    if cfg.needles:
        pos = d["needle_pos"].cpu().numpy()
        idn = idx.cpu().numpy()
        rec = np.mean([np.isin(pos[b, h], idn[b, h]).mean() for b in range(cfg.B) for h in range(cfg.Hkv)])
        announce(f"[opc] {name}: needle recall under the calibrated projection {rec:.3f}")
        # the same budget with the error-aware safeguard: the needles are far
        # from every calibrated component, so their reconstruction errors are
        # large and the hard-to-hash set picks them up
        err = torch.empty(cfg.B, cfg.Hkv, cfg.N, device=DEV)
        bpc.hash_keys(d["K"], Pcal, codes_out=torch.empty_like(codes), err_out=err)
        k_hash, m = oracle.eas_budget(cfg.k)
        serr = bpc.select_hard(err, m)
        idx2 = torch.empty(cfg.B, cfg.Hkv, k_hash, dtype=torch.int32, device=DEV)
        bpc.decode_attention(d["q"], d["K"], d["V"], codes, Pcal, k_hash, idx_out=idx2, serr=serr)
        torch.cuda.synchronize()
        sel = [np.union1d(idx2[b, h].cpu().numpy(), serr[b, h].cpu().numpy()) for b in range(cfg.B)
               for h in range(cfg.Hkv)]
        rec2 = np.mean([np.isin(pos[b, h], sel[b * cfg.Hkv + h]).mean() for b in range(cfg.B) for h in range(cfg.Hkv)])
        announce(f"[opc] {name}: needle recall with the safeguard (k_hash={k_hash}, m={m}) {rec2:.3f}")
