"""Write tests/golden/fullsize_oracle.json: the oracle's results on sampled
heads of every workload at full size.

The GPU tests of the full-size pipelines (tests/test_gpu_fullsize.py) compare
the library's build, hashing and decode of whole batches against these
records, head by head, so the oracle does not have to run at test time (at a
million keys its Algorithm 1 takes minutes per head).  This script calls only
the oracle and the seeded input generators; nothing here comes from the HIP
library.  Each record holds:

* digests of the generated inputs (so a test can tell an input mismatch from a
  kernel mismatch), SHA-256 of the little-endian array bytes;
* Algorithm 1 ("Constructing hash codes and corresponding hashing
  projection", Sec. 3.2): digests of P (float32), the codes (uint32 words)
  and the reconstruction errors rounded to float32, and the fragile count;
* optionally Algorithm 2 ("Given projection, computing hashcode") of every
  key of the head under that P: code and error digests, fragile count;
* the decode step (Sec. 3.2 "Retrieval Phase", Algorithm "Computing hashing
  score", Sec. 4.2): the packed query planes, digests of the scores and the
  selected indices (int32), the attention output (float64 values), and for
  workloads with planted needles the needle recall; optionally the same with
  the error-aware safeguard (Sec. 3.2, Eq. safeguard_union; 10 % of the
  budget, Sec. 4.1), with fixed budgets of 1024 and 2048 keys, and with one
  selection per query head.

Usage: python tests/golden/write_fullsize_digests.py [--jobs 4] [--only NAME]
(about 25 minutes on 4 cores, most of it the million-key builds).
"""

from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import multiprocessing as mp
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
OUT = os.path.join(HERE, "fullsize_oracle.json")

# (config, layer, b, h, extras); extras: "hash" = Algorithm 2 over the head,
# "variants" = safeguard, fixed budgets and per-query-head selection
JOBS = (
    [("tiny_mha_4k", 0, 0, h, ("hash",)) for h in range(8)]
    + [("llama8b_32k", 0, 0, h, ("hash",) if h == 3 else ()) for h in range(8)]
    + [("batch16_128k", 0, b, h, ("variants",) if (b, h) in ((11, 6), (2, 7)) else ())
       for b, h in ((0, 0), (2, 7), (5, 3), (7, 6), (9, 1), (11, 6), (13, 4), (15, 2))]
    + [("stack32_b8_64k", layer, b, h, ("hash",) if j == 0 else ())
       for layer in (0, 10, 21, 31)
       for j, (b, h) in enumerate((((3 * layer) % 8, (5 * layer + 1) % 8), ((3 * layer + 4) % 8, (5 * layer + 6) % 8)))]
    + [("million_1m", 0, 0, 0, ("hash",)), ("million_1m", 0, 0, 5, ())]
)


def sha(a) -> str:
    import numpy as np
    a = np.ascontiguousarray(a)
    return hashlib.sha256(a.tobytes()).hexdigest()


def _reuse_heap() -> None:
    """Keep large freed blocks in the heap (glibc M_MMAP_MAX = 0, M_TRIM_THRESHOLD
    huge): the oracle's arrays of a million keys are freed and reallocated every
    bit, and fresh mappings would fault in every page again."""
    try:
        libc = ctypes.CDLL("libc.so.6")
        libc.mallopt(-4, 0)            # M_MMAP_MAX
        libc.mallopt(-1, 1 << 30)      # M_TRIM_THRESHOLD
    except OSError:
        pass


def run_job(job):
    _reuse_heap()
    sys.path.insert(0, ROOT)
    import numpy as np
    import torch

    import oracle
    from workloads import config_by_name
    from workloads.synth import make_gaussian_directions, make_head, make_query

    torch.set_num_threads(2)
    name, layer, b, h, extras = job
    cfg = config_by_name(name)
    t0 = time.time()
    q = make_query(cfg, layer, "cpu")
    K, V, pos = make_head(cfg, q, layer, b, h, "cpu")
    G = make_gaussian_directions(cfg).numpy()
    bits = lambda t: t.contiguous().view(torch.int16).numpy().view(np.uint16)  # noqa: E731
    Kb, Vb = bits(K), bits(V)
    qg = bits(q[b, h * cfg.G:(h + 1) * cfg.G])
    rec = {"config": name, "layer": layer, "b": b, "h": h, "N": cfg.N, "L": cfg.L, "k": cfg.k,
           "inputs": {"K": sha(Kb), "V": sha(Vb), "q_group": sha(qg), "G": sha(G.astype(np.float32))}}
    if cfg.needles:
        rec["needles"] = sorted(int(x) for x in pos.tolist())

    P, codes, err, frag = oracle.build_binary_pcs(Kb, G)
    err32 = err.astype(np.float32)
    rec["build"] = {"P": sha(P), "codes": sha(codes), "err_f32": sha(err32), "fragile": int(frag),
                    "err_sample": [float(err32[i]) for i in np.linspace(0, cfg.N - 1, 16).astype(np.int64)]}
    if "hash" in extras:
        c2, e2, f2 = oracle.hash_keys(Kb, P)
        rec["hash"] = {"codes": sha(c2), "err_f32": sha(e2.astype(np.float32)), "fragile": int(f2)}

    sm = 1.0 / np.sqrt(cfg.D)

    def decode_record(k):
        r = oracle.decode_head(qg, Kb, Vb, codes, P, k, sm)
        d = {"k": k, "qcode": [int(x) for x in r["qcode"].ravel()], "T": int(r["T"]),
             "scores": sha(r["scores"].astype(np.int32)), "idx": sha(r["idx"].astype(np.int32)),
             "idx_first": [int(x) for x in r["idx"][:8]], "out": r["out"].tolist()}
        if cfg.needles:
            d["needle_recall"] = float(np.isin(pos.numpy(), r["idx"]).mean())
        return d

    rec["decode"] = decode_record(cfg.k)
    if "variants" in extras:
        k_hash, m = oracle.eas_budget(cfg.k)
        serr = oracle.select_hard(err32, m)
        r = oracle.decode_head_eas(qg, Kb, Vb, codes, P, k_hash, serr, sm)
        rec["eas"] = {"k_hash": k_hash, "m": m, "serr": sha(serr.astype(np.int32)), "idx": sha(r["idx"].astype(np.int32)),
                      "added": sha(r["added"].astype(np.int32)), "n_added": int(r["added"].sum()),
                      "out": r["out"].tolist()}
        rec["fixed"] = [decode_record(kb) for kb in (1024, 2048)]
        r = oracle.decode_per_query_head(qg, Kb, Vb, codes, P, cfg.k, sm)
        rec["per_head"] = {"scores": [sha(s.astype(np.int32)) for s in r["scores"]],
                           "idx": [sha(i.astype(np.int32)) for i in r["idx"]], "out": r["out"].tolist()}
    rec["oracle_seconds"] = round(time.time() - t0, 1)
    print(f"done {name} layer {layer} head {(b, h)} in {rec['oracle_seconds']} s", flush=True)
    return rec


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=4)
    ap.add_argument("--only", default=None, help="recompute only this workload and keep the other records")
    args = ap.parse_args()
    todo = [j for j in JOBS if args.only is None or j[0] == args.only]
    # the longest jobs first, so that they overlap the short ones
    todo.sort(key=lambda j: -{"million_1m": 100, "batch16_128k": 10, "stack32_b8_64k": 5}.get(j[0], 1))
    keep = []
    if args.only is not None and os.path.exists(OUT):
        keep = [r for r in json.load(open(OUT))["records"] if r["config"] != args.only]
    with mp.get_context("spawn").Pool(args.jobs, maxtasksperchild=1) as pool:
        recs = pool.map(run_job, todo, chunksize=1)
    recs = keep + recs
    recs.sort(key=lambda r: (r["config"], r["layer"], r["b"], r["h"]))
    doc = {"what": "the oracle's results on sampled heads of the full-size workloads (see this script's docstring)",
           "written_by": "tests/golden/write_fullsize_digests.py",
           "digest": "SHA-256 of the little-endian bytes of the C-ordered array",
           "records": recs}
    with open(OUT, "w") as f:
        json.dump(doc, f, indent=1)
        f.write("\n")
    print(f"wrote {OUT} ({len(recs)} records)")


if __name__ == "__main__":
    main()
