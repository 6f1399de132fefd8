"""Benchmark of the BinaryPC decode hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

Workload: batch 16, 32 query / 8 KV heads, head_dim 128, 131072 cached keys
per sequence (bf16 K/V), 64-bit codes, 2 % budget (k = 2622 per KV head).
A step is one full decode step (query packing, XOR/popcount scan of every
cached code, exact top-k, gathered sparse attention, merge) for the whole
batch.  Four independent instances of the workload (different seeds) are
used in turn so that consecutive steps do not re-read each other's data from
the 256 MB last-level cache; all inputs are resident in HBM before timing.

Prints one JSON line with the metric (decode keys/s = B * Hkv * N / step
time), the stage breakdown, the roofline of the dominant kernel, the
prefill (binary-PC build and key hashing) timings and the CPU oracle's
throughput on a bounded sample.
"""

from __future__ import annotations

import argparse
import hashlib
import numpy as np
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode attention keys/sec/GPU at 128K ctx (hash+top-k+sparse attn); % HBM peak"
HBM_PEAK_GBS = 8000.0
PMC_FILE = os.path.join(ROOT, "profiles", "pmc_decode_batch16_128k.json")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_04405_amd", "csrc", f)
                  for f in ("decode_kernels.hip", "bpc_internal.h")]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=300)
    ap.add_argument("--instances", type=int, default=4)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--no-configs", action="store_true", help="measure only batch16_128k (skip the other workloads)")
    ap.add_argument("--decode-only", action="store_true",
                    help="skip the context measurements after the timed region (safeguard, fixed budgets, per "
                         "query head, dense, offline calibration), so that a profile holds only the decode step")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain 1 GiB device copy (counter calibration for rocprofv3 --pmc)")
    ap.add_argument("--cpu-sample-heads", type=int, default=128)
    ap.add_argument("--decode-path", choices=("auto", "three-launch"), default="auto",
                    help="auto: one fused launch when the step's workgroups fit on the GPU at once")
    ap.add_argument("--summarize", metavar="DIR", nargs="+", default=None,
                    help="summarize rocprofv3 csv output under each DIR (kernel stats and counters per dispatch) "
                         "instead of benchmarking")
    ap.add_argument("--prefill-only", metavar="WORKLOAD", default=None,
                    help="time only the prefill of one layer of WORKLOAD: Algorithm 1 recomputing its residual, "
                         "then with the residual checkpoint, then Algorithm 2 on both kernels; print one JSON line")
    ap.add_argument("--pmc-json", metavar="PATH", default=None,
                    help="with --summarize over a FETCH_SIZE and a WRITE_SIZE run: write HBM bytes per launch")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def source_sha() -> str:
    """Hash of the decode kernels' source with comments and blank lines
    removed: counter readings stay valid across comment-only edits."""
    import re
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        for line in open(p).read().splitlines():
            line = re.sub(r"//.*", "", line).strip()
            if line:
                h.update(line.encode() + b"\n")
    return h.hexdigest()[:16]


def _build_passes(path, root):
    """The Algorithm 1 builds of a kernel trace, one line each: the passes
    (build_bit launches, one per bit and a last one for the errors) and the
    time of the bit passes by range of bits."""
    import csv
    rows = []
    for r in csv.DictReader(open(path)):
        n = r["Kernel_Name"]
        if "bpc::build_" in n:
            rows.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), _short(n)))
    rows.sort()
    builds, cur = [], None
    for t0, t1, n in rows:
        if "build_prep" in n:
            cur = {"bit": [], "finish": [], "t0": t0, "t1": t1}
            builds.append(cur)
        elif cur is not None:
            cur["bit" if "build_bit" in n else "finish"].append((t1 - t0) / 1e3)
            cur["t1"] = t1
    out = []
    if builds:
        out.append(f"Algorithm 1 builds ({os.path.relpath(path, root)}), durations in us:")
    for i, b in enumerate(builds):
        bit = b["bit"]
        nb = len(bit)
        rng = [(a, min(e, nb - 1)) for a, e in ((0, 16), (16, 32), (32, 64), (64, nb - 1))] + [(nb - 1, nb)]
        parts = ", ".join(f"passes {a}-{e - 1}: mean {sum(bit[a:e]) / (e - a):.1f}" for a, e in rng if e > a)
        out.append(f"  build {i}: {len(bit)} bit passes, {sum(bit) / 1e3:.2f} ms in them, {sum(b['finish']) / 1e3:.2f} ms "
                   f"in {len(b['finish'])} fold and finish launches, {(b['t1'] - b['t0']) / 1e6:.2f} ms first to last; {parts}")
    return out


def _short(name: str) -> str:
    return name.split("(")[0].replace("void ", "").strip()


def _is_copy(name: str) -> bool:
    return "copyBuffer" in name


def _stage_of(name: str):
    import re
    m = re.search(r"bpc::(\w+?)_kernel", name)
    return m.group(1) if m else None


def summarize(roots, pmc_json=None) -> None:
    """Per-kernel summary of rocprofv3 csv output under each of `roots`
    (kernel stats, and the mean of every collected counter per dispatch).

    With `pmc_json`, the FETCH_SIZE / WRITE_SIZE means (KiB per dispatch) of
    the library's kernels are converted to HBM bytes per launch and written
    there.  Each counter is scaled by the factor that makes it read the
    known size of the 1 GiB device copies that `--copy-probe` adds to the
    run (the largest copy dispatches of the run; their read and their write
    are 1 GiB each)."""
    import csv
    import glob
    from collections import defaultdict

    lines = []
    kernels = defaultdict(dict)   # stage -> counter -> mean KiB per dispatch
    calib = {}                    # counter -> (mean KiB of the 1 GiB copies, n)
    for root in roots:
        for f in sorted(glob.glob(os.path.join(root, "**", "*kernel_stats.csv"), recursive=True)):
            lines.append(f"kernel stats ({os.path.relpath(f, root)}):")
            lines.append(f"{'kernel':<48}{'calls':>8}{'avg_us':>12}{'min_us':>10}{'max_us':>10}{'total_ms':>12}")
            for r in csv.DictReader(open(f)):
                if "bpc::" in r["Name"] or _is_copy(r["Name"]):
                    lines.append(f"{_short(r['Name'])[:47]:<48}{int(r['Calls']):>8}"
                                 f"{float(r['AverageNs']) / 1e3:>12.2f}{float(r.get('MinNs', 'nan')) / 1e3:>10.2f}"
                                 f"{float(r.get('MaxNs', 'nan')) / 1e3:>10.2f}{float(r['TotalDurationNs']) / 1e6:>12.3f}")
        for f in sorted(glob.glob(os.path.join(root, "**", "*kernel_trace.csv"), recursive=True)):
            lines.extend(_build_passes(f, root))
        for f in sorted(glob.glob(os.path.join(root, "**", "*counter_collection.csv"), recursive=True)):
            acc = defaultdict(lambda: defaultdict(list))
            copies = defaultdict(list)
            for r in csv.DictReader(open(f)):
                name = r.get("Kernel_Name", "")
                val = float(r["Counter_Value"])
                if _is_copy(name):
                    copies[r["Counter_Name"]].append(val)
                elif "bpc::" in name:
                    acc[_short(name)][r["Counter_Name"]].append(val)
            lines.append(f"counters, mean per dispatch ({os.path.relpath(f, root)}):")
            for cname, vals in sorted(copies.items()):
                # the calibration copies are by far the largest copies of the run
                big = [v for v in vals if v >= 0.5 * max(vals)]
                calib[cname] = (sum(big) / len(big), len(big))
                lines.append(f"  1 GiB device copy: {cname}={calib[cname][0]:.6g} (n={len(big)})")
            for kname in sorted(acc):
                vals = ", ".join(f"{c}={sum(v) / len(v):.6g} (n={len(v)})" for c, v in sorted(acc[kname].items()))
                lines.append(f"  {kname}: {vals}")
                st = _stage_of(kname)
                if st:
                    for c, v in acc[kname].items():
                        kernels[st][c] = sum(v) / len(v)
    print("\n".join(lines))
    if pmc_json:
        need = ("FETCH_SIZE", "WRITE_SIZE")
        if not all(c in calib for c in need):
            raise SystemExit("FETCH_SIZE and WRITE_SIZE runs with --copy-probe are both needed")
        factor = {c: float(1 << 30) / (calib[c][0] * 1024.0) for c in need}
        out = {"source_sha": source_sha(),
               "counter_unit": "KiB per dispatch",
               "copy_calibration": {c: {"copy_bytes": 1 << 30, "counter_kib": calib[c][0], "dispatches": calib[c][1],
                                        "bytes_per_counted_kib": factor[c] * 1024.0} for c in need},
               "kernels": {}}
        for st, cs in sorted(kernels.items()):
            if all(c in cs for c in need):
                fb = cs["FETCH_SIZE"] * 1024.0 * factor["FETCH_SIZE"]
                wb = cs["WRITE_SIZE"] * 1024.0 * factor["WRITE_SIZE"]
                out["kernels"][st] = {"fetch_kib": cs["FETCH_SIZE"], "write_kib": cs["WRITE_SIZE"],
                                      "read_bytes": round(fb), "write_bytes": round(wb),
                                      "hbm_bytes_per_launch": round(fb + wb)}
        with open(pmc_json, "w") as fh:
            json.dump(out, fh, indent=1)
            fh.write("\n")
        print(f"wrote {pmc_json}")


def host_info():
    """CPU model and the cores this process may use (the CPU baseline's host)."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"cpu_model": model, "usable_cores": len(os.sched_getaffinity(0))}


def step_bytes(B, Hq, Hkv, N, D, L, k, layers=1):
    """Algorithmic bytes of a decode step: codes read, gathered K+V rows, P,
    q read and out written (scores and selections are not counted)."""
    BH = B * Hkv
    return layers * (BH * N * (L // 8) + BH * k * 2 * D * 2 + BH * L * D * 4 + B * Hq * D * (2 + 4))


def time_steps(fn, steps, warmup, runs=1):
    """Mean us per step of `runs` timed regions of `steps` calls each, after
    `warmup` untimed calls; every region is bracketed by synchronizations."""
    import torch
    for j in range(warmup):
        fn(j)
    torch.cuda.synchronize()
    res = []
    for r in range(runs):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for j in range(steps):
            fn(j)
        e1.record()
        torch.cuda.synchronize()
        res.append(e0.elapsed_time(e1) / steps * 1e3)
    return res


def measure_config(bpc, cfg, dev, n_inst, steps, warmup, log_name):
    """One workload end to end: inputs generated on the GPU, the prefill
    (Algorithm 1 build with its fragile count, Algorithm 2 hashing of every
    key), then the decode step timed.  A step is one decode of every layer
    (the 32 layers of the stack one after another); single-layer workloads
    rotate `n_inst` independent instances so that steps do not share data
    through the 256 MB last-level cache."""
    import torch
    from workloads import make_layer
    B, Hq, Hkv, D, N, L, k = cfg.B, cfg.Hq, cfg.Hkv, cfg.D, cfg.N, cfg.L, cfg.k
    sm = 1.0 / math.sqrt(D)
    layers = cfg.layers
    n_data = layers if layers > 1 else n_inst
    frag = torch.zeros(1, dtype=torch.int64, device=dev)
    fall = torch.zeros(1, dtype=torch.int64, device=dev)
    ws_build = torch.empty(bpc.build_workspace_bytes(B, Hkv, N, L), dtype=torch.uint8, device=dev)
    ws_ck = torch.empty(bpc.build_checkpoint_workspace_bytes(B, Hkv, N, L), dtype=torch.uint8, device=dev)
    build_ms = build_ck_ms = hash_ms = hash_mm_ms = 0.0
    data = []
    t0 = time.time()
    for i in range(n_data):
        d = make_layer(cfg, layer=i, device=dev)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
        ev[0].record()
        P, codes, _ = bpc.build_hash(d["K"], d["G"].to(dev), fragile=frag if i == 0 or layers > 1 else None,
                                     workspace=ws_build)
        ev[1].record()
        if i == 0 or layers > 1:
            c2, _ = bpc.hash_keys(d["K"], P)
        ev[2].record()
        if i == 0 or layers > 1:
            c3 = bpc.hash_keys_mm(d["K"], P, fallbacks=fall)
        ev[3].record()
        if i == 0 or layers > 1:
            P4, c4, _ = bpc.build_hash(d["K"], d["G"].to(dev), workspace=ws_ck)
        ev[4].record()
        torch.cuda.synchronize()
        if i == 0 or layers > 1:
            build_ms += ev[0].elapsed_time(ev[1])
            hash_ms += ev[1].elapsed_time(ev[2])
            hash_mm_ms += ev[2].elapsed_time(ev[3])
            build_ck_ms += ev[3].elapsed_time(ev[4])
            if not torch.equal(c2, c3):
                raise RuntimeError(f"{log_name}: matrix-core Algorithm 2 codes differ from the fp64 kernel's")
            if not (torch.equal(P4, P) and torch.equal(c4, codes)):
                raise RuntimeError(f"{log_name}: the checkpointed Algorithm 1 build differs from the recomputing one")
            del c2, c3, P4, c4
        data.append({"q": d["q"], "K": d["K"], "V": d["V"], "codes": codes, "P": P})
        del d
    del ws_build, ws_ck
    torch.cuda.empty_cache()
    keys_pf = B * Hkv * N * (layers if layers > 1 else 1)
    log(f"{log_name}: {n_data} layers/instances generated and built in {time.time() - t0:.1f}s")
    ws = torch.zeros(bpc.decode_workspace_bytes(B, Hq, Hkv, N, L, k), dtype=torch.uint8, device=dev)
    outs = [torch.empty(B, Hq, D, dtype=torch.float32, device=dev) for _ in range(min(n_data, 4))]

    def step(j):
        if layers > 1:  # every layer of the stack in turn
            for i, it in enumerate(data):
                bpc.decode_attention(it["q"], it["K"], it["V"], it["codes"], it["P"], k, sm, out=outs[i % 4],
                                     workspace=ws)
        else:
            it = data[j % len(data)]
            bpc.decode_attention(it["q"], it["K"], it["V"], it["codes"], it["P"], k, sm, out=outs[j % len(outs)],
                                 workspace=ws)

    runs = time_steps(step, steps, warmup, runs=3)
    us = float(np.median(runs))
    nbytes = step_bytes(B, Hq, Hkv, N, D, L, k, layers)
    keys = B * Hkv * N * layers
    res = {"workload": cfg.name, "B": B, "Hq": Hq, "Hkv": Hkv, "N": N, "L": L, "k": k, "layers": layers,
           "us_per_step": round(us, 2), "runs_us_per_step": [round(x, 2) for x in runs],
           "mean_us_per_step": round(float(np.mean(runs)), 2),
           "keys_per_s": keys / (us * 1e-6), "token_positions_per_s": B * N * layers / (us * 1e-6),
           "step_algorithmic_bytes": nbytes, "hbm_frac": round(nbytes / (us * 1e-6) / (HBM_PEAK_GBS * 1e9), 4),
           "decode_path": "fused single launch" if bpc.decode_path_taken(B, Hq, Hkv, N, L) == 0 else "three launches",
           "slice_keys": bpc.decode_slice_keys(B, Hq, Hkv, N, L),
           "prefill": {"build_ms": round(build_ms, 2), "hash_ms": round(hash_ms, 2),
                       "build_keys_per_s": keys_pf / (build_ms * 1e-3), "hash_keys_per_s": keys_pf / (hash_ms * 1e-3),
                       "build_checkpoint_ms": round(build_ck_ms, 2),
                       "hash_mm_ms": round(hash_mm_ms, 2), "hash_mm_keys_per_s": keys_pf / (hash_mm_ms * 1e-3),
                       "hash_mm_recomputed_decisions": int(fall.item()),
                       "fragile_sign_decisions": int(frag.item()),
                       "covers": "all layers" if layers > 1 else "one instance"}}
    log(f"{log_name}: {res['us_per_step']} us/step, {res['keys_per_s']:.3g} keys/s, {res['hbm_frac'] * 100:.1f} % of "
        f"8 TB/s; prefill {res['prefill']}")
    del data, ws, outs
    torch.cuda.empty_cache()
    return res


def copy_ceiling(dev):
    """A plain 1 GiB device-to-device copy (read + write), the reference
    rate of a streaming kernel on this GPU."""
    import torch
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    us = time_steps(lambda j: dst.copy_(src), 10, 3)[0]
    del src, dst
    torch.cuda.empty_cache()
    return {"bytes_per_copy": 2 << 30, "us": round(us, 1), "GBps": round((2 << 30) / (us * 1e-6) / 1e9, 1),
            "what": "torch copy of 1 GiB (1 GiB read + 1 GiB written), mean of 10"}


def prefill_only(name):
    """Prefill of one layer of a workload, each kernel path once after a
    warm-up build: Algorithm 1 recomputing the residual, Algorithm 1 with
    the residual checkpoint (results compared), Algorithm 2 fp64 and on the
    matrix cores (codes compared)."""
    import torch

    import paper_2608_04405_amd as bpc
    from workloads import config_by_name, make_layer
    cfg = config_by_name(name)
    dev = torch.device("cuda:0")
    B, Hkv, N, L = cfg.B, cfg.Hkv, cfg.N, cfg.L
    d = make_layer(cfg, layer=0, device=dev)
    K, G = d["K"], d["G"].to(dev)
    del d
    ws = torch.empty(bpc.build_checkpoint_workspace_bytes(B, Hkv, N, L), dtype=torch.uint8, device=dev)
    small = ws[:bpc.build_workspace_bytes(B, Hkv, N, L)]
    bpc.build_hash(K, G, workspace=small)  # warm-up
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
    ev[0].record()
    P1, c1, _ = bpc.build_hash(K, G, workspace=small)
    ev[1].record()
    P2, c2, _ = bpc.build_hash(K, G, workspace=ws)
    ev[2].record()
    h1, _ = bpc.hash_keys(K, P1)
    ev[3].record()
    h2 = bpc.hash_keys_mm(K, P1)
    ev[4].record()
    torch.cuda.synchronize()
    if not (torch.equal(P1, P2) and torch.equal(c1, c2) and torch.equal(h1, h2)):
        raise RuntimeError(f"{name}: the prefill paths disagree")
    t = [ev[i].elapsed_time(ev[i + 1]) for i in range(4)]
    print(json.dumps({"workload": name, "keys": B * Hkv * N, "L": L, "build_ms": round(t[0], 3),
                      "build_checkpoint_ms": round(t[1], 3), "hash_ms": round(t[2], 3), "hash_mm_ms": round(t[3], 3),
                      "checkpoint_workspace_bytes": int(ws.numel())}), flush=True)


def main():
    args = parse()
    if args.summarize:
        summarize(args.summarize, args.pmc_json)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (the decode step of every "
              "(sequence, KV head) is independent; see DESIGN.md for how it would shard).", file=sys.stderr)
        sys.exit(2)
    if args.prefill_only:
        prefill_only(args.prefill_only)
        return

    import torch

    import paper_2608_04405_amd as bpc
    from workloads import config_by_name, make_calibration_keys, make_layer

    cfg = config_by_name("batch16_128k")
    dev = torch.device("cuda:0")
    bpc.set_decode_path(0 if args.decode_path == "auto" else 1)
    B, Hq, Hkv, D, N, L, k = cfg.B, cfg.Hq, cfg.Hkv, cfg.D, cfg.N, cfg.L, cfg.k
    sm = 1.0 / math.sqrt(D)
    W = L // 32
    host = host_info()

    # ---------------------------------------------------------------- inputs
    insts = []
    t0 = time.time()
    for i in range(args.instances):
        d = make_layer(cfg, layer=i, device=dev)
        insts.append({"q": d["q"], "K": d["K"], "V": d["V"], "G": d["G"].to(dev)})
        del d
    torch.cuda.synchronize()
    log(f"generated {args.instances} instances in {time.time() - t0:.1f}s")

    # ---------------------------------------------------------------- prefill
    ws_build = torch.empty(bpc.build_workspace_bytes(B, Hkv, N, L), dtype=torch.uint8, device=dev)
    prefill = {}
    frag = torch.zeros(1, dtype=torch.int64, device=dev)
    frag2 = torch.zeros(1, dtype=torch.int64, device=dev)
    frag3 = torch.zeros(1, dtype=torch.int64, device=dev)
    fall3 = torch.zeros(1, dtype=torch.int64, device=dev)
    for i, it in enumerate(insts):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
        ev[0].record()
        err = torch.empty(B, Hkv, N, dtype=torch.float32, device=dev)
        P, codes, _ = bpc.build_hash(it["K"], it["G"], err_out=err, fragile=frag if i == 0 else None,
                                     workspace=ws_build)
        ev[1].record()
        if i == 0 and not args.no_prefill:
            err2 = torch.empty(B, Hkv, N, dtype=torch.float32, device=dev)
            codes2, _ = bpc.hash_keys(it["K"], P, err_out=err2, fragile=frag2)
            ev[2].record()
            codes3 = bpc.hash_keys_mm(it["K"], P, fragile=frag3, fallbacks=fall3)
            ev[3].record()
            codes4, _ = bpc.hash_keys(it["K"], P)
            ev[4].record()
            # Algorithm 1 again, keeping the fp64 residual every 16 bits
            del ws_build
            ws_ck = torch.empty(bpc.build_checkpoint_workspace_bytes(B, Hkv, N, L), dtype=torch.uint8, device=dev)
            err5 = torch.empty(B, Hkv, N, dtype=torch.float32, device=dev)
            frag5 = torch.zeros(1, dtype=torch.int64, device=dev)
            ev5 = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            ev5[0].record()
            P5, codes5, _ = bpc.build_hash(it["K"], it["G"], err_out=err5, fragile=frag5, workspace=ws_ck)
            ev5[1].record()
        torch.cuda.synchronize()
        it["P"], it["codes"], it["err"] = P, codes, err
        if i == 0 and not args.no_prefill:
            build_ms = ev[0].elapsed_time(ev[1])
            hash_ms = ev[1].elapsed_time(ev[2])
            hash_mm_ms = ev[2].elapsed_time(ev[3])
            hash_codes_ms = ev[3].elapsed_time(ev[4])
            build_ck_ms = ev5[0].elapsed_time(ev5[1])
            if not (torch.equal(codes2, codes3) and torch.equal(codes2, codes4)) or int(frag2.item()) != int(frag3.item()):
                raise RuntimeError("matrix-core Algorithm 2 differs from the fp64 kernel")
            if not (torch.equal(P5, P) and torch.equal(codes5, codes) and torch.equal(err5, err)
                    and int(frag5.item()) == int(frag.item())):
                raise RuntimeError("the checkpointed Algorithm 1 build differs from the recomputing one")
            keys = B * Hkv * N
            prefill = {"build_ms": round(build_ms, 3), "hash_ms": round(hash_ms, 3),
                       "build_keys_per_s": keys / (build_ms / 1e3), "hash_keys_per_s": keys / (hash_ms / 1e3),
                       "build_checkpoint_ms": round(build_ck_ms, 3),
                       "build_checkpoint_workspace_bytes": int(ws_ck.numel()),
                       "hash_codes_only_ms": round(hash_codes_ms, 3),
                       "hash_mm_ms": round(hash_mm_ms, 3), "hash_mm_keys_per_s": keys / (hash_mm_ms / 1e3),
                       "hash_mm_speedup": round(hash_codes_ms / hash_mm_ms, 2),
                       "hash_mm_recomputed_decisions": int(fall3.item()),
                       "fragile_sign_decisions_build": int(frag.item()),
                       "fragile_sign_decisions_hash": int(frag2.item()),
                       "what": "Algorithm 1 (build P, codes and errors) and Algorithm 2 (hash every key, with "
                               "errors) for the whole batch, fp64 fixed-order arithmetic; build_checkpoint: the same "
                               "build keeping each key's fp64 residual every 16 bits (same results); hash_codes_only: the same "
                               "kernel without the errors; hash_mm: the same codes with the projections on the "
                               "matrix cores and certified signs (recomputed = decisions redone in fp64); fragile = "
                               "sign decisions with |a| < 1e-6"}
            del codes2, codes3, codes4, err2, ws_ck, P5, codes5, err5
            ws_build = None
    del ws_build
    torch.cuda.empty_cache()
    log(f"prefill {prefill}")

    ws = torch.zeros(bpc.decode_workspace_bytes(B, Hq, Hkv, N, L, k), dtype=torch.uint8, device=dev)
    outs = [torch.empty(B, Hq, D, dtype=torch.float32, device=dev) for _ in insts]

    def step(j, events=None):
        it = insts[j % len(insts)]
        bpc.decode_attention(it["q"], it["K"], it["V"], it["codes"], it["P"], k, sm, out=outs[j % len(insts)],
                             workspace=ws, events=events)

    if args.copy_probe:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # ---------------------------------------------------------------- timed region
    for j in range(args.warmup):
        step(j)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    start.record()
    for j in range(args.steps):
        step(j)
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_per_step = start.elapsed_time(end) / args.steps
    keys_per_step = B * Hkv * N
    value = keys_per_step / (ms_per_step / 1e3)
    log(f"{ms_per_step * 1e3:.1f} us/step, {value:.4g} keys/s (wall {wall:.3f}s)")
    # two more timed regions of the same length: three runs, median and mean
    runs = [ms_per_step * 1e3] + time_steps(step, args.steps, 0, runs=2)
    log(f"three runs: {[round(x, 2) for x in runs]} us/step")

    # ---------------------------------------------------------------- stage breakdown (same steps, with events)
    nst = bpc.DECODE_STAGES
    prof_steps = max(10, min(args.steps, 100))

    def stage_times():
        t = np.zeros(nst)
        evsets = [[torch.cuda.Event(enable_timing=True) for _ in range(nst + 1)] for _ in range(prof_steps)]
        for j in range(prof_steps):
            step(j, events=evsets[j])
        torch.cuda.synchronize()
        for evs in evsets:
            for s in range(nst):
                t[s] += evs[s].elapsed_time(evs[s + 1])
        return {n: round(float(x) / prof_steps * 1e3, 2) for n, x in zip(bpc.DECODE_STAGE_NAMES, t)}

    fused = bpc.decode_path_taken(B, Hq, Hkv, N, L) == 0
    stages = stage_times()  # on the fused path the whole step is the first stage (one launch)
    bpc.set_decode_path(1)
    ws3 = torch.zeros(bpc.decode_workspace_bytes(B, Hq, Hkv, N, L, k), dtype=torch.uint8, device=dev)
    ws_keep, ws = ws, ws3
    for j in range(args.warmup):
        step(j)
    three = stage_times()
    three_us = time_steps(step, prof_steps, 0)[0]
    ws = ws_keep
    del ws3
    torch.cuda.empty_cache()
    bpc.set_decode_path(0 if args.decode_path == "auto" else 1)
    log(f"stages (us): {stages}; three-launch path: {three}, {three_us:.1f} us/step")

    eas, fixed, per_head, dense, opc = {}, {}, {}, {}, {}
    if not args.decode_only:
        # ---------------------------------------------------------------- the error-aware safeguard (context)
        # the same step with 10 % of the 2 % budget reserved for the hard-to-hash
        # set: k_hash = 2359 by hash score, union with the 263 keys of largest
        # reconstruction error chosen once at prefill
        k_hash = k - (k + 9) // 10
        m_eas = k - k_hash
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        for it in insts:
            it["serr"] = bpc.select_hard(it["err"], m_eas)
        ev[1].record()
        torch.cuda.synchronize()
        select_ms = ev[0].elapsed_time(ev[1]) / len(insts)

        def eas_step(j):
            it = insts[j % len(insts)]
            bpc.decode_attention(it["q"], it["K"], it["V"], it["codes"], it["P"], k_hash, sm, out=outs[j % len(insts)],
                                 serr=it["serr"], workspace=ws)

        eas = {"us_per_step": round(time_steps(eas_step, prof_steps, args.warmup)[0], 2), "k_hash": k_hash,
               "m": m_eas, "select_hard_ms": round(select_ms, 3),
               "what": "decode step over S_hash (top-2359 by hash score) united with S_err (263 keys of largest "
                       "reconstruction error, chosen per (b, h) at prefill by select_hard)"}
        log(f"safeguard: {eas}")

        # ---------------------------------------------------------------- fixed-count budgets (context)
        fixed = {}
        for kb in (1024, 2048):
            ws_b = torch.zeros(bpc.decode_workspace_bytes(B, Hq, Hkv, N, L, kb), dtype=torch.uint8, device=dev)

            def fixed_step(j, kb=kb, ws_b=ws_b):
                it = insts[j % len(insts)]
                bpc.decode_attention(it["q"], it["K"], it["V"], it["codes"], it["P"], kb, sm, out=outs[j % len(insts)],
                                     workspace=ws_b)

            fixed[f"k{kb}_us_per_step"] = round(time_steps(fixed_step, prof_steps, args.warmup)[0], 2)
            del ws_b
        fixed["what"] = "the decode step with a fixed budget of 1024 or 2048 keys per (b, h)"
        log(f"fixed budgets: {fixed}")

        # ---------------------------------------------------------------- per-query-head selection (context)
        ws_ph = torch.zeros(bpc.decode_per_head_workspace_bytes(B, Hq, Hkv, N, L, k), dtype=torch.uint8, device=dev)

        def per_head_step(j):
            it = insts[j % len(insts)]
            bpc.decode_attention_per_head(it["q"], it["K"], it["V"], it["codes"], it["P"], k, sm,
                                          out=outs[j % len(insts)], workspace=ws_ph)

        ph_us = time_steps(per_head_step, prof_steps, args.warmup)[0]
        ph_bytes = B * Hq * N * W * 4 + B * Hq * k * 2 * D * 2 + B * Hq * L * D * 4 + B * Hq * D * (2 + 4)
        per_head = {"us_per_step": round(ph_us, 2), "GBps": round(ph_bytes / (ph_us * 1e-6) / 1e9, 1),
                    "what": f"one selection of {k} keys per query head ({Hq // Hkv} scans of each KV head's codes and "
                            f"{Hq // Hkv} gathers per (b, h))"}
        del ws_ph
        log(f"per query head: {per_head}")

        # ---------------------------------------------------------------- dense decode attention (context)
        ws_dense = torch.empty(int(bpc._lib.bpc_dense_workspace_bytes(B, Hq, Hkv, N, D)), dtype=torch.uint8, device=dev)

        def dense_step(j):
            it = insts[j % len(insts)]
            bpc.dense_attention(it["q"], it["K"], it["V"], sm, out=outs[j % len(insts)], workspace=ws_dense)

        dense_us = time_steps(dense_step, 10, 3)[0]
        dense_bytes = B * Hkv * N * 2 * D * 2 + B * Hq * D * (2 + 4)
        dense = {"us_per_step": round(dense_us, 1), "GBps": round(dense_bytes / (dense_us * 1e-6) / 1e9, 1),
                 "sparse_speedup": round(dense_us / (ms_per_step * 1e3), 2),
                 "what": "dense decode attention over all keys (every K and V row read), the comparison point"}
        del ws_dense
        log(f"dense: {dense}")

        # ---------------------------------------------------------------- offline projection calibration (context)
        if not args.no_prefill:
            Kcal = make_calibration_keys(cfg, layer=0, n_seq=1, device=dev)
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            ev[0].record()
            Pcal = bpc.build_hash(Kcal, insts[0]["G"])[0][0]
            ev[1].record()
            codes_opc = bpc.hash_keys_mm(insts[0]["K"], Pcal)
            ev[2].record()
            torch.cuda.synchronize()
            del Kcal
            it = insts[0]
            opc_us = time_steps(lambda j: bpc.decode_attention(it["q"], it["K"], it["V"], codes_opc, Pcal, k, sm,
                                                               out=outs[0], workspace=ws), 50, 5)[0]
            opc = {"calibration_build_ms": round(ev[0].elapsed_time(ev[1]), 3),
                   "prefill_hash_ms": round(ev[1].elapsed_time(ev[2]), 3),
                   "decode_us_per_step_same_instance": round(opc_us, 2),
                   "what": "P per KV head from Algorithm 1 over 131072 held-out keys; prefill = Algorithm 2 of the "
                           "whole batch against it (matrix-core path); decode with the shared P, one instance repeated (its data "
                           "partly stays in the 256 MB last-level cache)"}
            del codes_opc
            log(f"offline calibration: {opc}")

    # algorithmic bytes (per step): codes read, gathered K+V rows, P, q and out
    BH = B * Hkv
    code_bytes = BH * N * W * 4
    gather_bytes = BH * k * 2 * D * 2
    p_bytes = BH * L * D * 4
    qo_bytes = B * Hq * D * (2 + 4)
    sbytes = code_bytes + gather_bytes + p_bytes + qo_bytes
    if fused:
        # one launch per step moves every algorithmic byte of the step: its
        # average duration is the timed regions' step time (back-to-back
        # launches; the event-bracketed stage timing adds each launch's
        # end-of-kernel flush and is kept only as a breakdown)
        dom, dom_us, dom_bytes = "fused_decode", float(np.median(runs)), sbytes
    else:
        per_kernel_bytes = {"score": code_bytes + p_bytes + B * Hq * D * 2, "attend": gather_bytes + B * Hq * D * 2}
        dom = max(("score", "attend"), key=lambda n: stages[n])
        dom_us, dom_bytes = stages[dom], per_kernel_bytes[dom]
    achieved = dom_bytes / (dom_us * 1e-6) / 1e9
    traffic = None
    if os.path.exists(PMC_FILE):
        pmc = json.load(open(PMC_FILE))
        if pmc.get("source_sha") == source_sha() and dom in pmc.get("kernels", {}):
            traffic = pmc["kernels"][dom]["hbm_bytes_per_launch"]
    roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "algorithmic_bytes_per_launch": dom_bytes, "avg_launch_us": round(dom_us, 2)}
    step_gbs = sbytes / (ms_per_step * 1e-3) / 1e9

    # ---------------------------------------------------------------- the other workloads
    del insts, ws, outs
    torch.cuda.empty_cache()
    configs = {}
    if not args.no_configs:
        for name, n_inst, steps in (("tiny_mha_4k", 4, 200), ("llama8b_32k", 4, 200), ("stack32_b8_64k", 1, 10),
                                    ("million_1m", 3, 60)):
            configs[name] = measure_config(bpc, config_by_name(name), dev, n_inst, steps, 5, name)
    ceiling = copy_ceiling(dev)
    log(f"copy ceiling: {ceiling}")

    # ---------------------------------------------------------------- CPU oracle baseline
    cpu = None
    if not args.no_cpu_baseline:
        d0 = make_layer(cfg, layer=0, device=dev)
        cpu = cpu_baseline(cfg, d0, args.cpu_sample_heads, host)
        del d0

    line = {
        "metric": METRIC,
        "value": value,
        "unit": "keys/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 K/V/q, u32 codes, f32 accumulation",
        "data": "synthetic",
        "config": {"workload": cfg.name, "B": B, "Hq": Hq, "Hkv": Hkv, "head_dim": D, "N": N, "code_bits": L,
                   "k": k, "budget": "2%", "instances": args.instances,
                   "decode_path": "fused single launch" if fused else "three launches",
                   "slice_keys": bpc.decode_slice_keys(B, Hq, Hkv, N, L)},
        "runs_us_per_step": [round(x, 2) for x in runs],
        "median_us_per_step": round(float(np.median(runs)), 2),
        "mean_us_per_step": round(float(np.mean(runs)), 2),
        "hbm_frac_step": round(step_gbs / HBM_PEAK_GBS, 4),
        "step_algorithmic_bytes": sbytes,
        "step_GBps": round(step_gbs, 1),
        "token_positions_per_s": B * N / (ms_per_step * 1e-3),
        "stages_us": stages,
        "three_launch_path": {"us_per_step": round(three_us, 2), "stages_us": three},
        "roofline": roofline,
        "copy_ceiling": ceiling,
        "prefill": prefill,
        "configs": configs,
        "eas": eas,
        "fixed_budget": fixed,
        "per_query_head": per_head,
        "dense": dense,
        "opc": opc,
        "cpu_baseline": cpu,
        "host": host,
        "wall_s_timed": round(wall, 4),
    }
    print(json.dumps(line), flush=True)


def cpu_baseline(cfg, inst, heads: int, host):
    """The oracle's decode step, timed on host cores for `heads` (b, h) pairs
    of the same workload.  Codes are drawn uniformly by the input generator
    (the oracle's running time does not depend on their values); P comes from
    the oracle's own build on the first 256 keys of the head."""
    import numpy as np
    import torch
    from threadpoolctl import threadpool_limits

    import oracle

    def bits(t):
        return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)

    rng = np.random.default_rng(7)
    sm = 1.0 / math.sqrt(cfg.D)
    G = inst["G"].cpu().numpy()
    total = 0.0
    pairs = [(b, h) for b in range(cfg.B) for h in range(cfg.Hkv)][:heads]
    with threadpool_limits(1):
        for b, h in pairs:
            K = bits(inst["K"][b, h])
            V = bits(inst["V"][b, h])
            q = bits(inst["q"][b, h * cfg.G:(h + 1) * cfg.G])
            codes = rng.integers(0, 1 << 32, size=(cfg.N, cfg.L // 32), dtype=np.uint64).astype(np.uint32)
            P = oracle.build_binary_pcs(K[:256], G)[0]
            t0 = time.perf_counter()
            oracle.decode_head(q, K, V, codes, P, cfg.k, sm)
            total += time.perf_counter() - t0
    keys = len(pairs) * cfg.N
    return {"value": keys / total, "unit": "keys/s", "cores": 1, "kind": "oracle",
            "sample": f"decode step of {len(pairs)} of the {cfg.B * cfg.Hkv} (sequence, KV head) pairs "
                      f"({keys} keys) of {cfg.name}, numpy fp64 oracle on one thread, {total:.1f} s",
            "cpu_model": host["cpu_model"], "usable_cores": host["usable_cores"]}


if __name__ == "__main__":
    main()
