"""Full-size parity: every workload's own pipeline on the GPU (Algorithm 1
build, Algorithm 2 hashing, the decode step), launched as the benchmark
launches it (the whole batch or layer in one call, the library's own
workspace sizing), against the oracle's records of sampled heads.

The records (tests/golden/fullsize_oracle.json) are written by
tests/golden/write_fullsize_digests.py, which calls only the oracle and the
input generators.  Each sampled head is generated on the CPU (the generator
gives the same values on any host) and copied into the GPU-generated batch;
its input digests are checked first, so an input mismatch is told apart
from a kernel mismatch.  Then, bit for bit: P, the codes, the float32
reconstruction errors and the fragile count of Algorithm 1, Algorithm 2's
codes and errors where recorded, the packed query planes, the scores and
the selected indices; the attention output within 2e-3 per row.

* tiny_mha_4k and llama8b_32k: all 8 KV heads.
* batch16_128k: 8 of the 128 (sequence, KV head) pairs; two of them also with
  the error-aware safeguard, fixed budgets of 1024 and 2048 keys and one
  selection per query head.
* stack32_b8_64k: all 32 layers end to end (build, then decode, per layer);
  2 heads of each of layers 0, 10, 21 and 31 against the records.
* million_1m: the GPU's own Algorithm 1 over all 1 048 576 keys at L = 128,
  then the decode on those codes; 2 KV heads against the records, including
  the recall of the 64 planted needles.

Every head, sampled or not, is checked for the selection property: indices
strictly ascending, the selected keys the k best by score, equal scores going
to the lower index.
"""

import hashlib
import json
import os

import numpy as np
import pytest
import torch

from workloads import config_by_name, make_layer
from workloads.synth import make_head, make_query

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    import paper_2608_04405_amd as bpc
else:  # pragma: no cover
    bpc = None

DEV = "cuda"
TOL = 2e-3
RECORDS = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "fullsize_oracle.json")


def records(name, layer=None):
    recs = [r for r in json.load(open(RECORDS))["records"] if r["config"] == name]
    return [r for r in recs if layer is None or r["layer"] == layer]


def sha(a) -> str:
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def bits(t):
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def u32(t):
    return t.detach().cpu().contiguous().numpy().view(np.uint32)


def i32(t):
    return t.detach().cpu().contiguous().numpy().astype(np.int32)


def rel_err(o, ref):
    o = np.asarray(o, np.float64)
    return np.max(np.abs(o - ref), axis=-1) / np.max(np.abs(ref), axis=-1)


def announce(msg):
    print(msg, flush=True)


def check_selection_property(scores: np.ndarray, idx: np.ndarray, k: int, where: str) -> None:
    """idx ascending, unique, in range; {scores[idx]} are the k largest with
    ties at the threshold resolved towards the lower index."""
    N = scores.shape[0]
    assert idx.shape == (k,), where
    assert idx[0] >= 0 and idx[-1] < N and np.all(np.diff(idx) > 0), f"{where}: indices not ascending/in range"
    if k == N:
        return
    sel = np.zeros(N, bool)
    sel[idx] = True
    s_min = scores[sel].min()
    u_max = scores[~sel].max()
    assert s_min >= u_max, f"{where}: an unselected key outscores a selected one"
    if s_min == u_max:
        tied_sel = np.flatnonzero(sel & (scores == s_min))
        tied_uns = np.flatnonzero(~sel & (scores == s_min))
        assert tied_sel.max() < tied_uns.min(), f"{where}: tie at the threshold not broken by lowest index"


def all_heads_property(sc, idx, k, label):
    scn, idn = sc.cpu().numpy(), idx.cpu().numpy()
    for b in range(idn.shape[0]):
        for h in range(idn.shape[1]):
            check_selection_property(scn[b, h], idn[b, h], k, f"{label} head {(b, h)}")


def layer_with_recorded_heads(cfg, layer, recs):
    """The layer generated on the GPU, with the recorded heads replaced by
    their CPU-generated values and the CPU query (what the oracle saw); the
    recorded input digests are checked."""
    d = make_layer(cfg, layer=layer, device=DEV)
    qc = make_query(cfg, layer, "cpu")
    d["q"] = qc.to(DEV)
    d["G"] = d["G"].to(DEV)
    for r in recs:
        b, h = r["b"], r["h"]
        Kh, Vh, pos = make_head(cfg, qc, layer, b, h, "cpu")
        assert sha(bits(Kh)) == r["inputs"]["K"], f"generated keys of {(layer, b, h)} differ from the recorded ones"
        assert sha(bits(Vh)) == r["inputs"]["V"], f"generated values of {(layer, b, h)} differ"
        assert sha(bits(qc[b, h * cfg.G:(h + 1) * cfg.G])) == r["inputs"]["q_group"], "generated query differs"
        assert sha(d["G"].cpu().numpy()) == r["inputs"]["G"], "Gaussian directions differ"
        d["K"][b, h, :cfg.N] = Kh.to(DEV)
        d["V"][b, h, :cfg.N] = Vh.to(DEV)
    torch.cuda.synchronize()
    return d


def build_layer(cfg, d):
    # the whole layer with the residual checkpoint; check_build rebuilds one
    # head without it
    err = torch.empty(cfg.B, cfg.Hkv, cfg.N, device=DEV)
    frag = torch.zeros(1, dtype=torch.int64, device=DEV)
    P, codes, _ = bpc.build_hash(d["K"], d["G"], err_out=err, fragile=frag, checkpoint=True)
    return P, codes, err, frag


def check_build(cfg, d, P, codes, err, rec, label):
    b, h = rec["b"], rec["h"]
    assert sha(P[b, h].cpu().numpy()) == rec["build"]["P"], f"{label}: projection differs"
    assert sha(u32(codes[b, h])) == rec["build"]["codes"], f"{label}: codes differ"
    e = err[b, h].cpu().numpy()
    pick = np.linspace(0, cfg.N - 1, 16).astype(np.int64)
    np.testing.assert_allclose(e[pick], rec["build"]["err_sample"], rtol=0, atol=0)
    assert sha(e) == rec["build"]["err_f32"], f"{label}: reconstruction errors differ"
    # the fragile count of this head alone, from a build of just this head
    frag = torch.zeros(1, dtype=torch.int64, device=DEV)
    P1, c1, _ = bpc.build_hash(d["K"][b:b + 1, h:h + 1], d["G"], N=cfg.N, fragile=frag)
    torch.cuda.synchronize()
    assert torch.equal(P1[0, 0], P[b, h]) and torch.equal(c1[0, 0, :cfg.N], codes[b, h, :cfg.N])
    assert int(frag.item()) == rec["build"]["fragile"], f"{label}: fragile count differs"


def decode_batch(cfg, d, codes, P, k):
    B, Hkv, L = cfg.B, cfg.Hkv, cfg.L
    idx = torch.empty(B, Hkv, k, dtype=torch.int32, device=DEV)
    sc = torch.empty(B, Hkv, cfg.N, dtype=torch.int32, device=DEV)
    qc = torch.empty(B, Hkv, 8, L // 32, dtype=torch.int32, device=DEV)
    out = bpc.decode_attention(d["q"], d["K"], d["V"], codes, P, k, N=cfg.N, idx_out=idx, score_out=sc,
                               qcode_out=qc)
    torch.cuda.synchronize()
    assert torch.isfinite(out).all()
    return out, idx, sc, qc


def check_decode(cfg, rec_dec, b, h, out, idx, sc, qc, label, needles=None):
    G = cfg.G
    assert u32(qc[b, h]).ravel().tolist() == rec_dec["qcode"], f"{label}: query planes differ"
    assert sha(i32(sc[b, h])) == rec_dec["scores"], f"{label}: scores differ"
    got = i32(idx[b, h])
    assert got[:8].tolist() == rec_dec["idx_first"] and sha(got) == rec_dec["idx"], f"{label}: indices differ"
    e = rel_err(out[b, h * G:(h + 1) * G].cpu().numpy(), np.asarray(rec_dec["out"]))
    msg = f"{label}: max relative output error {e.max():.3g}"
    if needles is not None:
        recall = float(np.isin(np.asarray(needles), got).mean())
        assert recall == rec_dec["needle_recall"]
        msg += f", needle recall {recall:.3f}"
    announce(msg)
    assert np.all(e <= TOL), msg


def check_hash(cfg, d, P, rec, label):
    b, h = rec["b"], rec["h"]
    frag = torch.zeros(1, dtype=torch.int64, device=DEV)
    err = torch.empty(1, 1, cfg.N, device=DEV)
    c2, _ = bpc.hash_keys(d["K"][b:b + 1, h:h + 1], P[b:b + 1, h:h + 1].contiguous(), N=cfg.N, err_out=err,
                          fragile=frag)
    torch.cuda.synchronize()
    assert sha(u32(c2[0, 0, :cfg.N])) == rec["hash"]["codes"], f"{label}: Algorithm 2 codes differ"
    assert sha(err[0, 0].cpu().numpy()) == rec["hash"]["err_f32"], f"{label}: Algorithm 2 errors differ"
    assert int(frag.item()) == rec["hash"]["fragile"], f"{label}: Algorithm 2 fragile count differs"
    # the matrix-core path with certified signs: the same codes and count
    frag.zero_()
    fall = torch.zeros(1, dtype=torch.int64, device=DEV)
    c3 = bpc.hash_keys_mm(d["K"][b:b + 1, h:h + 1], P[b:b + 1, h:h + 1].contiguous(), N=cfg.N, fragile=frag,
                          fallbacks=fall)
    torch.cuda.synchronize()
    assert sha(u32(c3[0, 0, :cfg.N])) == rec["hash"]["codes"], f"{label}: matrix-core Algorithm 2 codes differ"
    assert int(frag.item()) == rec["hash"]["fragile"], f"{label}: matrix-core fragile count differs"
    announce(f"{label}: matrix-core Algorithm 2 bit-exact, {int(fall.item())} of {cfg.N * cfg.L} decisions "
             f"recomputed in fp64")


def check_variants(cfg, d, P, codes, err, rec, label):
    b, h = rec["b"], rec["h"]
    G = cfg.G
    rows = slice(h * G, (h + 1) * G)
    ev = rec["eas"]
    serr = bpc.select_hard(err, ev["m"])
    idx2 = torch.empty(cfg.B, cfg.Hkv, ev["k_hash"], dtype=torch.int32, device=DEV)
    added = torch.empty(cfg.B, cfg.Hkv, ev["m"], dtype=torch.int32, device=DEV)
    out2 = bpc.decode_attention(d["q"], d["K"], d["V"], codes, P, ev["k_hash"], N=cfg.N, idx_out=idx2, serr=serr,
                                added_out=added)
    torch.cuda.synchronize()
    assert sha(i32(serr[b, h])) == ev["serr"], f"{label}: hard-to-hash set differs"
    assert sha(i32(idx2[b, h])) == ev["idx"], f"{label}: safeguard S_hash differs"
    assert sha(i32(added[b, h])) == ev["added"], f"{label}: safeguard flags differ"
    e = rel_err(out2[b, rows].cpu().numpy(), np.asarray(ev["out"]))
    announce(f"{label} with the safeguard ({ev['n_added']} of {ev['m']} added): max relative output error {e.max():.3g}")
    assert np.all(e <= TOL)
    for fx in rec["fixed"]:
        out_b, idx_b, sc_b, qc_b = decode_batch(cfg, d, codes, P, fx["k"])
        all_heads_property(sc_b, idx_b, fx["k"], f"{label} k={fx['k']}")
        check_decode(cfg, fx, b, h, out_b, idx_b, sc_b, qc_b, f"{label} fixed budget k={fx['k']}")
    ph = rec["per_head"]
    idx_p = torch.empty(cfg.B, cfg.Hq, cfg.k, dtype=torch.int32, device=DEV)
    sc_p = torch.empty(cfg.B, cfg.Hq, cfg.N, dtype=torch.int32, device=DEV)
    out_p = bpc.decode_attention_per_head(d["q"], d["K"], d["V"], codes, P, cfg.k, N=cfg.N, idx_out=idx_p,
                                          score_out=sc_p)
    torch.cuda.synchronize()
    scn, idn = sc_p.cpu().numpy(), idx_p.cpu().numpy()
    for bb in range(cfg.B):
        for j in range(cfg.Hq):
            check_selection_property(scn[bb, j], idn[bb, j], cfg.k, f"per head {(bb, j)}")
    for g in range(G):
        assert sha(scn[b, h * G + g].astype(np.int32)) == ph["scores"][g], f"{label}: per-head scores differ"
        assert sha(idn[b, h * G + g].astype(np.int32)) == ph["idx"][g], f"{label}: per-head indices differ"
    e = rel_err(out_p[b, rows].cpu().numpy(), np.asarray(ph["out"]))
    announce(f"{label} per query head: max relative output error {e.max():.3g}")
    assert np.all(e <= TOL)


def run_layer(cfg, layer, recs, label):
    """Build and decode one layer on the GPU; the recorded heads against the
    oracle, every head for the selection property."""
    d = layer_with_recorded_heads(cfg, layer, recs)
    P, codes, err, frag = build_layer(cfg, d)
    out, idx, sc, qc = decode_batch(cfg, d, codes, P, cfg.k)
    all_heads_property(sc, idx, cfg.k, label)
    for r in recs:
        where = f"{label} head {(r['b'], r['h'])}"
        check_build(cfg, d, P, codes, err, r, where)
        check_decode(cfg, r["decode"], r["b"], r["h"], out, idx, sc, qc, where, r.get("needles"))
        if "hash" in r:
            check_hash(cfg, d, P, r, where)
        if "eas" in r:
            check_variants(cfg, d, P, codes, err, r, where)
    return int(frag.item())


@pytest.mark.timeout(300)
@pytest.mark.parametrize("name", ["tiny_mha_4k", "llama8b_32k"])
def test_fullsize_all_heads(name):
    cfg = config_by_name(name)
    recs = records(name)
    announce(f"[full size] {cfg}: {len(recs)} recorded heads")
    total = run_layer(cfg, 0, recs, name)
    # every head is recorded: the batch's fragile count is their sum
    assert len(recs) == cfg.B * cfg.Hkv
    assert total == sum(r["build"]["fragile"] for r in recs)


@pytest.mark.timeout(600)
def test_fullsize_batch16_128k():
    cfg = config_by_name("batch16_128k")
    recs = records(cfg.name)
    announce(f"[full size] {cfg}: {len(recs)} recorded heads")
    run_layer(cfg, 0, recs, cfg.name)


@pytest.mark.timeout(900)
def test_fullsize_stack_all_layers_b8_64k():
    cfg = config_by_name("stack32_b8_64k")
    announce(f"[full size] {cfg}: all {cfg.layers} layers")
    checked = 0
    for layer in range(cfg.layers):
        recs = records(cfg.name, layer)
        frag = run_layer(cfg, layer, recs, f"{cfg.name} layer {layer}")
        checked += len(recs)
        announce(f"layer {layer}: built, hashed and decoded; {len(recs)} heads against the oracle; "
                 f"{frag} fragile sign decisions")
        torch.cuda.empty_cache()
    assert checked == len(records(cfg.name)) >= 8


@pytest.mark.timeout(900)
def test_fullsize_million_1m():
    cfg = config_by_name("million_1m")
    recs = records(cfg.name)
    announce(f"[full size] {cfg}: {len(recs)} recorded heads")
    assert len(recs) >= 2
    run_layer(cfg, 0, recs, cfg.name)
