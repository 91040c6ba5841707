#!/usr/bin/env python3
"""Benchmark of the MSV -> Viterbi -> Forward profile-HMM search on one MI355X.

One step = one hmm_search of the workload's profile against its whole
database (every stage of the cascade, on the GPU, inputs resident in HBM).
Prints one JSON line on stdout; progress goes to stderr.

Metric: GCUPS = M x (database residues) / (seconds per step) / 1e9.
Default workload: M = 734 profile against 1,000,000 synthetic sequences
(~348M residues, 0.5 % planted homologs), MSV P < 0.02 -> Viterbi
P < 1e-3 -> Forward on survivors.

Roofline of the dominant kernel (MSV): plain packed-int16 VALU arithmetic,
4 element-ops per cell (max, saturating add, saturating subtract, max), so
achieved = 4 x cells / (average MSV duration), against the MI355X packed
16-bit VALU peak 256 CU x 64 lanes x 2 elements x 2.4 GHz = 78.64 Tops/s.
The MSV duration is measured with HIP events that the library records on
the search stream around the stage.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_PK16_TOPS = 256 * 64 * 2 * 2.4e9 / 1e12      # 78.64
MSV_OPS_PER_CELL = 4
VIT_OPS_PER_CELL = 18


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def cpu_baseline(prof, db, F, budget_s: float, threads: int) -> dict:
    """The CPU oracle (scalar C, threaded) on a stride sample of the same
    database, sized to roughly `budget_s` seconds."""
    import numpy as np

    import oracle
    op = oracle.OracleProfile(prof)
    calib = oracle.calibrate(op, nthreads=threads)
    lengths = np.diff(db.offsets)

    def run(stride):
        idx = np.arange(0, db.n, stride)
        seqs = [db.residues[db.offsets[i]:db.offsets[i + 1]] for i in idx]
        off = np.zeros(idx.size + 1, np.int64)
        off[1:] = np.cumsum(lengths[idx])
        res = np.concatenate(seqs)
        t = time.perf_counter()
        oracle.search(op, res, off, calib, F, nthreads=threads)
        return time.perf_counter() - t, int(res.size), int(idx.size)

    probe_stride = max(1, db.n // 2000)
    t, nres, nseq = run(probe_stride)
    rate = nres / max(t, 1e-6)
    stride = max(1, int(math.ceil(db.n * float(lengths.mean()) / (rate * budget_s))))
    t, nres, nseq = run(stride)
    gcups = prof.M * nres / t / 1e9
    return {"value": round(gcups, 4), "unit": "GCUPS", "cores": threads, "kind": "oracle",
            "sample": f"every {stride}th target of the same database ({nseq} targets, {nres} residues), "
                      f"same cutoffs, oracle's own calibration; {t:.1f} s wall",
            "seconds": round(t, 2)}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="C3", choices=["C1", "C2", "C3", "C5"])
    ap.add_argument("--cpu-seconds", type=float, default=20.0, help="budget of the CPU-oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib", default=None,
                    help="mu_msv,mu_vit,tau to use instead of calibrating on the GPU (profiling runs)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MB",
                    help="run one plain device copy of MB MiB first (scales rocprofv3 byte counters)")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "msv_traffic_C3.json"),
                    help="HBM traffic per MSV launch measured by rocprofv3 counters (JSON), if present")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the search shards by database bins across GPUs "
              "without communication, and only the single-GPU path is built and measured.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2111_06340_amd as hg
    from paper_2111_06340_amd.calibrate import calibrate
    from synth import gen

    assert torch.cuda.is_available(), "bench.py needs the GPU"
    w = gen.WORKLOADS[args.workload]
    t = time.perf_counter()
    prof = gen.workload_profile(w)
    db = gen.workload_database(w, prof=prof)
    log(f"generated {w.name}: M={prof.M}, {db.n} targets, {db.residues.size} residues "
        f"in {time.perf_counter() - t:.1f}s")
    t = time.perf_counter()
    if args.calib:
        calib = tuple(float(v) for v in args.calib.split(","))
    else:
        calib = calibrate(prof)
    log(f"calibration mu_msv={calib[0]!r} mu_vit={calib[1]!r} tau={calib[2]!r} "
        f"({'given' if args.calib else 'on the GPU'}, {time.perf_counter() - t:.1f}s)")
    P = hg.Profile(prof, *calib)
    t = time.perf_counter()
    D = hg.Database(db.residues, db.offsets)
    upload_s = time.perf_counter() - t
    log(f"database packed and uploaded in {upload_s:.2f}s (host buffers, PCIe included; not timed below)")
    out = hg.alloc_results(D.n)
    stream = torch.cuda.current_stream()
    if args.copy_probe:
        src = torch.ones(args.copy_probe << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy probe: {src.numel()} bytes read and written once")
        del src, dst
    for _ in range(args.warmup):
        hg.search(P, D, w.F, out, stream=stream)
    torch.cuda.synchronize()
    hg.hmm_db_stage_timing(D.handle, args.steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        hg.search(P, D, w.F, out, stream=stream)
    torch.cuda.synchronize()
    total = time.perf_counter() - t0
    stages = hg.hmm_db_stage_times(D.handle, args.steps)
    hg.hmm_db_stage_timing(D.handle, 0)
    ms_step = total / args.steps * 1e3
    cells = prof.M * D.n_residues
    gcups = cells / (ms_step / 1e3) / 1e9
    counts = out["counts"].cpu().numpy().tolist()
    fl = out["flags"].cpu().numpy()
    vit_cells = prof.M * int(np.diff(db.offsets)[(fl & hg.HMM_VIT_RAN) != 0].sum())
    st_ms = stages.mean(axis=0) if stages.size else np.zeros(4)
    msv_ms = float(st_ms[0])
    achieved = MSV_OPS_PER_CELL * cells / (msv_ms / 1e3) / 1e12
    log(f"{ms_step:.3f} ms/step, {gcups:.1f} GCUPS; stages ms: MSV {st_ms[0]:.3f} Viterbi {st_ms[1]:.3f} "
        f"rescore {st_ms[2]:.3f} (concurrent with) Forward {st_ms[3]:.3f}; counts {counts}")
    traffic = None
    if os.path.exists(args.traffic):
        with open(args.traffic) as f:
            tr = json.load(f)
        if tr.get("workload") == w.name and tr.get("kernel_source_sha") == kernel_source_sha():
            traffic = tr.get("bytes_per_launch")
    rec = {
        "metric": "GCUPS (profile cols x DB residues /s), MSV+Viterbi+Forward, M=734 vs 1M seqs",
        "value": round(gcups, 2),
        "unit": "GCUPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8/i16/i32/f32",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: Plan7 profile M={prof.M} vs {D.n} synthetic sequences "
                               f"({D.n_residues} residues, {w.planted * 100:g}% planted homologs), "
                               f"MSV P<{w.F[0]:g} -> Viterbi P<{w.F[1]:g} -> Forward",
                   "M": prof.M, "n_seqs": D.n, "residues": D.n_residues, "cutoffs": list(w.F)},
        # rescore and Forward run concurrently after Viterbi: both are timed
        # from Viterbi's end, Forward until both are done
        "stage_ms": {"msv": round(float(st_ms[0]), 4), "viterbi": round(float(st_ms[1]), 4),
                     "rescore": round(float(st_ms[2]), 4), "forward_and_rescore": round(float(st_ms[3]), 4)},
        "survivors": {"msv_pass": counts[0], "vit_overflow": counts[1], "vit_pass": counts[2],
                      "fwd_pass": counts[3], "viterbi_cells": vit_cells},
        "roofline": {"bound": "alu", "kernel": "msv_kernel", "achieved": round(achieved, 3),
                     "peak": round(PEAK_PK16_TOPS, 2), "unit": "Tops/s (packed 16-bit VALU element-ops)",
                     "frac": round(achieved / PEAK_PK16_TOPS, 4), "traffic": traffic,
                     "ops_per_cell": MSV_OPS_PER_CELL, "cells_per_launch": cells},
        "upload_s": round(upload_s, 3),
    }
    P.close()
    D.close()
    if not args.no_cpu_baseline:
        threads = min(16, len(os.sched_getaffinity(0)))
        log(f"CPU oracle baseline on {threads} threads ...")
        rec["cpu_baseline"] = cpu_baseline(prof, db, w.F, args.cpu_seconds, threads)
        log(f"CPU oracle: {rec['cpu_baseline']['value']} GCUPS")
    print(json.dumps(rec), flush=True)


def kernel_source_sha() -> str:
    import hashlib
    p = os.path.join(ROOT, "paper_2111_06340_amd", "csrc", "hmm_kernels.hip")
    with open(p, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


if __name__ == "__main__":
    main()
