#!/usr/bin/env python3
"""Benchmark of the MSV -> Viterbi -> Forward profile-HMM search on one MI355X.

One step = one hmm_search of the workload's profile against its whole
database (every stage of the cascade, on the GPU, inputs resident in HBM).
Prints one JSON line on stdout; progress goes to stderr.

Metric: GCUPS = M x (database residues) / (seconds per step) / 1e9.
Default workload: M = 734 profile against 1,000,000 synthetic sequences
(~348M residues, 0.5 % planted homologs), MSV P < 0.02 -> Viterbi
P < 1e-3 -> Forward on survivors.  Other modes: --workload C1/C2/C5 (the
other single-profile configurations), --workload C4 (64 profiles, M 50-400,
against the C3 database; one step searches all 64, reported as aggregate
GCUPS and queries/hour), --cutoffs F1,F2,F3 (e.g. 1,1e-3,1 runs Viterbi on
every target).

Roofline of the dominant kernel (MSV): plain packed 16-bit VALU work, bound
by instruction issue.  `frac` is the launch's VALU issue against the
datasheet: the wave64 VALU instructions of one MSV launch (rocprofv3
SQ_INSTS_VALU, recorded in profiles/msv_traffic_C3.json for the same
kernel source) over the launch's live duration, against one wave
instruction per CU per clock (256 x 2.4 GHz); `achieved` and `peak` are the
same rate in packed 16-bit element-ops (x 128 per instruction, peak 256 CU x
64 lanes x 2 elements x 2.4 GHz = 78.64 Tops/s).  The MSV launches of a
search (one per pipelined chunk) run back to back on the search stream,
between HIP events that the library records there, so the live launch
duration is the stage's time divided by the launches.  Beside it,
`algorithmic_frac` counts the nominal 4 element-ops per cell (max,
saturating add, saturating subtract, running max) over the same time; the
fp16 rewrite needs fewer instructions than that (one packed add and one
packed 3-way maximum per two cells, plus its running maximum), so that
figure can pass 1 while the issue fraction cannot.  `traffic` is the HBM
bytes per MSV launch that rocprofv3's FETCH_SIZE and WRITE_SIZE counters
measured for the same kernel source (scaled by a plain 1 GiB copy), beside
the launch's algorithmic bytes; `valu_issue` is the same instruction count
against the sustained rate a probe kernel measures in the run.
`stage_roofline` gives the algorithmic fraction of every stage (Viterbi 18
ops/cell, rescore 17 int32 ops/cell against 39.32 Tops/s, Forward 18
flops/cell against 157.3 TFLOP/s).
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
PEAK_I32_TOPS = 256 * 64 * 2.4e9 / 1e12           # 39.32
PEAK_FP32_TFLOPS = 157.3                          # datasheet (packed fp32 FMA)
PEAK_WAVE_INSTS = 256 * 2.4e9                     # VALU wave64 instructions per second (one per CU per clock)
MSV_OPS_PER_CELL = 4
VIT_OPS_PER_CELL = 18
RESCORE_OPS_PER_CELL = 17
FWD_FLOPS_PER_CELL = 18
BWD_FLOPS_PER_CELL = 26
OA_FLOPS_PER_CELL = 20


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def host_cpus() -> dict:
    """The host the CPU baseline runs on: logical CPUs, the CPUs this
    process may use, and the CPU model."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"nproc": os.cpu_count(), "affinity": len(os.sched_getaffinity(0)), "cpu_model": model}


def oracle_threads() -> int:
    """Threads of the CPU baseline: the host CPUs allotted to this GPU
    (OMP_NUM_THREADS where the job scheduler sets it, else 16), within the
    CPUs this process may use."""
    share = int(os.environ.get("OMP_NUM_THREADS") or 16)
    return max(1, min(share, len(os.sched_getaffinity(0))))


def cpu_baseline(profs, db, F, budget_s: float, threads: int) -> dict:
    """The CPU oracle (scalar C, threaded) on a stride sample of the same
    database, every profile of the workload on the same sample, sized to
    roughly `budget_s` seconds; GCUPS = sum over profiles of M x sampled
    residues / seconds."""
    import numpy as np

    import oracle
    ops = [oracle.OracleProfile(p) for p in profs]
    calibs = [oracle.calibrate(op, nthreads=threads) for op in ops]
    lengths = np.diff(db.offsets)

    def run(stride):
        idx = np.arange(0, db.n, stride)
        seqs = [db.residues[db.offsets[i]:db.offsets[i + 1]] for i in idx]
        off = np.zeros(idx.size + 1, np.int64)
        off[1:] = np.cumsum(lengths[idx])
        res = np.concatenate(seqs)
        t = time.perf_counter()
        for op, calib in zip(ops, calibs):
            oracle.search(op, res, off, calib, F, nthreads=threads)
        return time.perf_counter() - t, int(res.size), int(idx.size)

    probe_stride = max(1, db.n * len(profs) // 2000)
    t, nres, nseq = run(probe_stride)
    rate = nres / max(t, 1e-6)
    stride = max(1, int(math.ceil(db.n * float(lengths.mean()) / (rate * budget_s))))
    t, nres, nseq = run(stride)
    gcups = sum(p.M for p in profs) * nres / t / 1e9
    what = "every profile on " if len(profs) > 1 else ""
    return {"value": round(gcups, 4), "unit": "GCUPS", "cores": threads, "kind": "oracle",
            "sample": f"{what}one target in {stride} of the same database ({nseq} targets, {nres} residues), "
                      f"same cutoffs, oracle's own calibration; {t:.1f} s wall on {threads} threads",
            "seconds": round(t, 2), "host": host_cpus(),
            "threads_note": "one oracle thread per host CPU allotted to this GPU (16 on a one-GPU share)"}


def issue_roofline(insts_per_launch, ms_per_launch) -> dict:
    """VALU issue of a launch against the datasheet: its wave64 VALU
    instructions (rocprofv3 SQ_INSTS_VALU, same kernel source) over its
    live duration, against one wave instruction per CU per clock (4 SIMD16
    each issue a wave64 instruction per 4 clocks): 256 x 2.4e9 = 6.144e11
    per second.  In packed 16-bit element-ops (x 128 per instruction) the
    peak is 78.64 Tops/s.  Cannot exceed 1."""
    rate = insts_per_launch / (ms_per_launch / 1e3)
    return {"achieved": round(rate * 128 / 1e12, 3), "peak": round(PEAK_PK16_TOPS, 2),
            "frac": round(rate / PEAK_WAVE_INSTS, 4), "insts_per_launch": insts_per_launch}


def valu_issue(insts_per_launch, ms_per_launch, probe_ops_per_s):
    """Share of the sustained VALU issue rate a launch used: its wave64 VALU
    instructions (rocprofv3 SQ_INSTS_VALU, for the same kernel source) over
    its duration times the chip's sustained rate of wave instructions (the
    packed 16-bit probe's element-ops / 128: 64 lanes x 2 halves each).
    Unlike the algorithmic fraction this cannot exceed 1."""
    rate = probe_ops_per_s / 128.0
    return {"insts_per_launch": insts_per_launch, "sustained_insts_per_s": round(rate, 1),
            "frac": round(insts_per_launch / (ms_per_launch / 1e3 * rate), 4)}


def stage_roofline(M_list, res_total, ran_cells, st_ms, chunks=1, fused=False):
    """Per-stage fractions of the relevant VALU peak: algorithmic ops of the
    cells each stage processed, over its measured time (HIP events).  With
    a pipelined search (chunks > 1) the later stages overlap the MSV of the
    next chunk and only their exposed time is measured, so only MSV's
    fraction is given (run with --pipeline 1 for the others).  With the
    fused tail (Viterbi, rescore and Forward as one kernel) the three have
    one time, given as `tail` (run with --tail 1 for the separate ones)."""
    msv_ops = MSV_OPS_PER_CELL * sum(M * res_total for M in M_list)
    out = {}

    def entry(ops, ms, peak, unit):
        ach = ops / (ms / 1e3) / 1e12 if ms > 0 else 0.0
        return {"algorithmic_achieved": round(ach, 3), "peak": peak, "unit": unit,
                "algorithmic_frac": round(ach / peak, 4)}

    out["msv"] = entry(msv_ops, st_ms[0], round(PEAK_PK16_TOPS, 2), "Tops/s packed 16-bit, 4 ops/cell")
    if chunks > 1:
        out["note"] = (f"{chunks} pipelined chunks: Viterbi, rescore and Forward overlap the next chunk's MSV; "
                       f"stage_ms holds their exposed time after the last MSV")
        return out
    if fused:
        out["tail"] = {"ms": round(st_ms[1], 4),
                       "note": "Viterbi, rescore and Forward as one kernel (hmm_db_fused_tail mode 2): one time "
                               "for the three stages; --tail 1 times them one by one"}
        return out
    out["viterbi"] = entry(VIT_OPS_PER_CELL * ran_cells["viterbi"], st_ms[1], round(PEAK_PK16_TOPS, 2),
                           "Tops/s packed 16-bit, 18 ops/cell, cells of the targets scored to their last row "
                           "(int16 overflows, which stop early, left out: a lower bound)")
    out["rescore"] = entry(RESCORE_OPS_PER_CELL * ran_cells["rescore"], st_ms[2], round(PEAK_I32_TOPS, 2),
                           "Tops/s 32-bit, 17 ops/cell")
    # Forward runs beside the rescore; its figure here uses the time both take
    out["forward"] = entry(FWD_FLOPS_PER_CELL * ran_cells["forward"], st_ms[3], PEAK_FP32_TFLOPS,
                           "TFLOP/s fp32, 18 flops/cell (datasheet peak counts packed fp32)")
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="C3", choices=["C1", "C2", "C3", "C4", "C5"],
                    help="C4 = 64 profiles (M 50-400) against the C3 database; one step searches all 64")
    ap.add_argument("--cutoffs", default=None, metavar="F1,F2,F3",
                    help="P-value cutoffs instead of the workload's (1,1e-3,1 runs Viterbi on every target)")
    ap.add_argument("--cpu-seconds", type=float, default=20.0, help="budget of the CPU-oracle baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib", default=None,
                    help="mu_msv,mu_vit,tau to use instead of calibrating on the GPU (profiling runs)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MB",
                    help="run one plain device copy of MB MiB first (scales rocprofv3 byte counters)")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "msv_traffic_C3.json"),
                    help="HBM traffic per MSV launch measured by rocprofv3 counters (JSON), if present")
    ap.add_argument("--streams", type=int, default=0,
                    help="spread the searches of a step over this many database handles (hmm_db_share) "
                         "and streams, so that they run concurrently (0 = 4 for C4, else 1)")
    ap.add_argument("--dbs", type=int, default=1,
                    help="search this many databases of the workload's recipe (different seeds) per step; "
                         "with --streams 2, one profile against two databases models the paper's "
                         "side-by-side MSA searches")
    ap.add_argument("--pipeline", type=int, default=-1,
                    help="chunks a search is pipelined in (hmm_db_pipeline; 0 = the library's default, "
                         "1 = sequential stages, whose per-stage times give per-stage roofline fractions; "
                         "-1 = 1 for C4, whose 64 searches overlap through --streams, else the default)")
    ap.add_argument("--tail", type=int, default=0, choices=[0, 1, 2, 3],
                    help="stages after MSV (hmm_db_fused_tail): 1 = one kernel per stage, 2 = one fused kernel "
                         "for profiles of up to 384 nodes, 3 = fused when the Viterbi cutoff is 1, "
                         "0 = the library's default (3)")
    ap.add_argument("--group", type=int, default=-1,
                    help="C4: searches per hmm_search_group call, each through its own database handle "
                         "(default: all 64 in one call; 0: separate hmm_search calls spread over --streams)")
    ap.add_argument("--bias", action="store_true",
                    help="run the cascade with the composition-bias filter between MSV and Viterbi")
    ap.add_argument("--iterations", type=int, default=1,
                    help="iterate the search this many times (search, decode the Forward passes, count their "
                         "alignments, re-estimate the profile, calibrate it, search again); reported under "
                         "'iterations', never in value")
    ap.add_argument("--decode", action="store_true",
                    help="also time posterior decoding (hmm_decode) of the Forward survivors of the last "
                         "search: Forward with rows kept, Backward, regions and alignments (reported "
                         "under 'decode', not in value)")
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
    batched = args.workload == "C4"
    if args.group < 0:
        args.group = 64 if batched and args.dbs == 1 else 0
    if args.group and (not batched or args.dbs != 1):
        print("--group applies to C4 with one database", file=sys.stderr)
        sys.exit(2)
    if args.group:
        args.streams = 1
    if args.streams <= 0:
        args.streams = 4 if batched else 1
    if args.pipeline < 0:
        args.pipeline = 1 if batched else 0
    w = gen.WORKLOADS["C3" if batched else args.workload]
    F = tuple(float(v) for v in args.cutoffs.split(",")) if args.cutoffs else w.F
    t = time.perf_counter()
    dbprof = gen.workload_profile(w)
    profs = gen.c4_profiles() if batched else [dbprof]
    dbs = [gen.workload_database(w, prof=dbprof, seed_offset=j) for j in range(args.dbs)]
    db = dbs[0]
    log(f"generated {args.workload}: {len(profs)} profile(s), M={[p.M for p in profs][:8]}"
        f"{'...' if len(profs) > 8 else ''}, {len(dbs)} database(s) of {db.n} targets, "
        f"{sum(d.residues.size for d in dbs)} residues in {time.perf_counter() - t:.1f}s")
    t = time.perf_counter()
    if args.calib:
        assert not batched, "--calib gives one profile's calibration"
        calibs = [tuple(float(v) for v in args.calib.split(","))]
    else:
        calibs = [calibrate(p) for p in profs]
    log(f"calibration {'given' if args.calib else 'on the GPU'} ({time.perf_counter() - t:.1f}s): "
        f"{calibs[0]!r}{' ...' if batched else ''}")
    Ps = [hg.Profile(p, *c) for p, c in zip(profs, calibs)]
    t = time.perf_counter()
    Ds = [hg.Database(d.residues, d.offsets) for d in dbs]
    D = Ds[0]
    chunks = [hg.hmm_db_pipeline(Dx.handle, args.pipeline) for Dx in Ds][0]
    tail_mode = [hg.hmm_db_fused_tail(Dx.handle, args.tail) for Dx in Ds][0]   # shared handles inherit it
    upload_s = time.perf_counter() - t
    log(f"database(s) packed and uploaded in {upload_s:.2f}s (host buffers, PCIe included; not timed below)")
    # search jobs (profile, database) spread round-robin over `streams` lanes;
    # lane j searches through its own handle of every database, on its own stream
    S = max(1, args.streams)
    lanes = [[Dx if j == 0 else Dx.share() for Dx in Ds] for j in range(S)]
    for lane in lanes[1:]:
        for h in lane:
            hg.hmm_db_pipeline(h.handle, chunks)
    streams = [torch.cuda.current_stream()] + [torch.cuda.Stream() for _ in range(S - 1)]
    jobs = [(pi, di) for pi in range(len(Ps)) for di in range(len(Ds))]
    outs = [hg.alloc_results(Ds[di].n) for _, di in jobs]
    stream = streams[0]
    if args.copy_probe:
        src = torch.ones(args.copy_probe << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy probe: {src.numel()} bytes read and written once")
        del src, dst

    # group mode: search i through handle i of the database, `group` searches per call
    ghandles = [D] + [D.share() for _ in range(len(Ps) - 1)] if args.group else []

    def step():
        if args.group:
            for a in range(0, len(Ps), args.group):
                b = min(len(Ps), a + args.group)
                hg.search_group(Ps[a:b], ghandles[a:b], F, outs[a:b], stream=stream, bias_filter=args.bias)
            return
        for i, ((pi, di), out) in enumerate(zip(jobs, outs)):
            j = i % S
            hg.search(Ps[pi], lanes[j][di], F, out, stream=streams[j], bias_filter=args.bias)

    timed_stages = S == 1 and len(Ds) == 1 and not args.group
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if timed_stages:
        hg.hmm_db_stage_timing(D.handle, args.steps * len(Ps))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    total = time.perf_counter() - t0
    if timed_stages:
        stages = hg.hmm_db_stage_times(D.handle, args.steps * len(Ps))
        hg.hmm_db_stage_timing(D.handle, 0)
    else:
        stages = np.zeros((0, 4))
    ms_step = total / args.steps * 1e3
    M_list = [p.M for p in profs]
    cells = sum(M_list) * sum(Dx.n_residues for Dx in Ds)
    gcups = cells / (ms_step / 1e3) / 1e9
    counts = np.zeros(4, np.int64)
    # cells each stage processed.  The int16 Viterbi pass (and MSV) stop at
    # the row where a target overflows, so Viterbi counts only the targets
    # it scored to the end (a lower bound of its work); the cells of the
    # overflowed targets, whose rows past the overflow are never computed,
    # are reported apart.
    ran = {"viterbi": 0, "viterbi_overflow": 0, "msv_overflow": 0, "rescore": 0, "forward": 0}
    for (pi, di), out in zip(jobs, outs):
        p = profs[pi]
        lengths = np.diff(dbs[di].offsets)
        counts += out["counts"].cpu().numpy()
        fl = out["flags"].cpu().numpy()
        vit_ran = (fl & hg.HMM_VIT_RAN) != 0
        vit_ovf = (fl & hg.HMM_VIT_OVF) != 0
        ran["viterbi"] += p.M * int(lengths[vit_ran & ~vit_ovf].sum())
        ran["viterbi_overflow"] += p.M * int(lengths[vit_ran & vit_ovf].sum())
        ran["msv_overflow"] += p.M * int(lengths[(fl & hg.HMM_MSV_OVF) != 0].sum())
        ran["rescore"] += p.M * int(lengths[(fl & hg.HMM_VIT_OVF) != 0].sum())
        ran["forward"] += p.M * int(lengths[(fl & hg.HMM_FWD_RAN) != 0].sum())
    counts = counts.tolist()
    # stage times summed over the profiles of one step
    st_ms = [float(v) for v in
             (stages.reshape(-1, len(Ps), 4).sum(axis=1).mean(axis=0) if stages.size else np.zeros(4))]
    msv_ms = float(st_ms[0])
    # the fused tail has instances for profiles of up to 384 nodes (3 int16
    # vectors per lane); longer ones run the staged kernels in either mode
    tail_fused = (tail_mode == 2 or (tail_mode == 3 and F[1] >= 1.0)) and max(M_list) <= 384
    achieved = MSV_OPS_PER_CELL * cells / (msv_ms / 1e3) / 1e12 if msv_ms > 0 else 0.0
    log(f"{ms_step:.3f} ms/step, {gcups:.1f} GCUPS; stages ms: MSV {st_ms[0]:.3f} Viterbi {st_ms[1]:.3f} "
        f"rescore {st_ms[2]:.3f} (concurrent with) Forward {st_ms[3]:.3f}; counts {counts}")
    # the packed 16-bit VALU rate this device sustains (a timed kernel of
    # independent chains of the MSV recurrence's instructions)
    probe_ops, _ = hg.hmm_probe_pk16(stream)
    probe_tops = probe_ops / 1e12
    log(f"packed 16-bit VALU probe: {probe_tops:.2f} Tops/s sustained (datasheet peak {PEAK_PK16_TOPS:.2f})")
    traffic = None
    if os.path.exists(args.traffic) and not batched and not args.cutoffs:
        with open(args.traffic) as f:
            tr = json.load(f)
        # the MSV stage's HBM bytes per search (all of its launches), while
        # the kernel source and the launches per search are the measured ones
        if (tr.get("workload") == w.name and tr.get("kernel_source_sha") == kernel_source_sha()
                and tr.get("header_sha", kernel_source_sha("hmm_device.h")) == kernel_source_sha("hmm_device.h")
                and tr.get("launches_per_search") == chunks):
            traffic = (tr.get("bytes_per_launch"), tr.get("algorithmic_bytes_per_launch"),
                       tr.get("valu_insts_per_launch"), tr.get("kernel_source_sha"))
    issue = issue_roofline(traffic[2], msv_ms / chunks) if traffic and traffic[2] and msv_ms > 0 else None
    if batched:
        wl = (f"C4: {len(profs)} Plan7 profiles, M {min(M_list)}-{max(M_list)} (sum {sum(M_list)}), each searched "
              f"against {D.n} synthetic sequences ({D.n_residues} residues, the C3 database)")
    else:
        wl = (f"{w.name}: Plan7 profile M={profs[0].M} vs {D.n} synthetic sequences ({D.n_residues} residues, "
              f"{w.planted * 100:g}% planted homologs)")
    if len(Ds) > 1:
        wl += (f", against {len(Ds)} databases of this recipe (different seeds; "
               f"{sum(Dx.n_residues for Dx in Ds)} residues in all)")
    if S > 1:
        wl += f", searches spread over {S} concurrent streams and database handles"
    if args.group:
        wl += f", hmm_search_group of {args.group} searches per call (one handle each)"
    wl += f", MSV P<{F[0]:g}{' -> composition-bias filter' if args.bias else ''} -> Viterbi P<{F[1]:g} -> Forward"
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
        "config": {"workload": wl, "M": M_list if batched else M_list[0], "n_seqs": D.n,
                   "residues": D.n_residues, "cutoffs": list(F), "databases": len(Ds), "streams": S},
        # rescore and Forward run concurrently after Viterbi: both are timed
        # from Viterbi's end, Forward until both are done (with the fused
        # tail, "viterbi" holds all three)
        "stage_ms": {"msv": round(float(st_ms[0]), 4), "viterbi": round(float(st_ms[1]), 4),
                     "rescore": round(float(st_ms[2]), 4), "forward_and_rescore": round(float(st_ms[3]), 4)},
        "survivors": {"msv_pass": counts[0],
                      "bias_pass": (int(sum(int(((o["flags"].cpu().numpy() & hg.HMM_BIAS_PASS) != 0).sum())
                                            for o in outs)) if args.bias else None),
                      "vit_overflow": counts[1], "vit_pass": counts[2],
                      "fwd_pass": counts[3], "viterbi_cells": ran["viterbi"],
                      "viterbi_overflow_cells": ran["viterbi_overflow"], "msv_overflow_cells": ran["msv_overflow"],
                      "rescore_cells": ran["rescore"],
                      "forward_cells": ran["forward"]},
        "roofline": {"bound": "alu", "kernel": "msv_kernel",
                     "achieved": issue["achieved"] if issue else None,
                     "peak": round(PEAK_PK16_TOPS, 2),
                     "unit": "Tops/s packed 16-bit VALU issue (SQ_INSTS_VALU x 128 per launch / launch time)",
                     "frac": issue["frac"] if issue else None,
                     "frac_note": ("wave64 VALU instructions per MSV launch (rocprofv3 counter record of the "
                                   "kernel source whose sha256[:16] is counter_source_sha, the one built here) / "
                                   "live launch time / (256 CU x 2.4 GHz); null when the record is for another "
                                   "source"),
                     "valu_insts_per_launch": issue["insts_per_launch"] if issue else None,
                     "counter_source_sha": traffic[3] if traffic else None,
                     "algorithmic_achieved": round(achieved, 3),
                     "algorithmic_frac": round(achieved / PEAK_PK16_TOPS, 4),
                     "algorithmic_note": ("4 packed 16-bit ops per cell (max, saturating add, saturating subtract, "
                                          "running max) x M x residues of a launch / launch time; the fp16 rewrite "
                                          "needs fewer instructions than that, so this can pass 1"),
                     "traffic": traffic[0] if traffic else None,
                     "traffic_note": ("HBM bytes per MSV launch (FETCH_SIZE + WRITE_SIZE, rocprofv3 counters "
                                      "scaled by a 1 GiB copy); algorithmic_bytes = residues of the launch's chunk "
                                      "+ 15 bytes of index and results per target"),
                     "algorithmic_bytes": traffic[1] if traffic else None,
                     "ms_per_launch": round(msv_ms / chunks, 4),
                     "peak_measured": round(probe_tops, 3),
                     "algorithmic_frac_of_measured": round(achieved / probe_tops, 4),
                     "valu_issue": (valu_issue(traffic[2], msv_ms / chunks, probe_ops)
                                    if traffic and traffic[2] else None),
                     "ops_per_cell": MSV_OPS_PER_CELL, "cells_per_search": cells // len(jobs),
                     "msv_launches_per_search": chunks}
        if timed_stages else None,
        "stage_roofline": (stage_roofline(M_list, D.n_residues, ran, st_ms, chunks, fused=tail_fused)
                           if timed_stages else None),
        "pipeline_chunks": chunks,
        "tail_mode": tail_mode,
        "upload_s": round(upload_s, 3),
        "calib": list(calibs[0]),
    }
    if batched:
        rec["queries_per_hour"] = round(len(Ps) / (ms_step / 1e3) * 3600.0, 1)
    if args.decode:
        pi, di = jobs[-1]
        rec["decode"] = bench_decode(hg, Ps[pi], profs[pi], Ds[di], outs[-1], stream, args)
    if args.iterations > 1 and not batched:
        rec["iterations"] = bench_iterations(hg, profs[0], calibs[0], D, F, stream, args)
    for P in Ps:
        P.close()
    for lane in lanes[1:]:
        for h in lane:
            h.close()
    for h in ghandles[1:]:
        h.close()
    for Dx in Ds:
        Dx.close()
    if not args.no_cpu_baseline and len(Ds) == 1:
        threads = oracle_threads()
        log(f"CPU oracle baseline on {threads} threads ...")
        rec["cpu_baseline"] = cpu_baseline(profs, db, F, args.cpu_seconds, threads)
        log(f"CPU oracle: {rec['cpu_baseline']['value']} GCUPS")
    print(json.dumps(rec), flush=True)


def bench_decode(hg, P, prof, D, out, stream, args) -> dict:
    """Time hmm_decode of the Forward passes of the last search on the
    search stream (HIP events on that stream bracket exactly its kernels)."""
    import numpy as np
    import torch
    flags = out["flags"]
    fl = flags.cpu().numpy()
    lengths = np.asarray(D.lengths_caller())
    sel = (fl & hg.HMM_FWD_PASS) != 0
    n_dec = int(sel.sum())
    cells = prof.M * int(lengths[sel].sum())
    dec = None
    for _ in range(max(1, args.warmup)):
        dec = hg.decode(P, D, flags=flags, mask=hg.HMM_FWD_PASS, stream=stream)
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record(stream)
    for _ in range(args.steps):
        dec = hg.decode(P, D, flags=flags, mask=hg.HMM_FWD_PASS, stream=stream)
    ev[1].record(stream)
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / args.steps
    doms = hg.domains_table(dec)
    region_cells = prof.M * sum(d["e"] - d["s"] + 1 for d in doms)
    # fp32 work of the three passes (FMA = 2 flops): Forward 18 and Backward
    # 26 flops per cell of every decoded target, alignment 20 per cell of
    # the regions (adds and maxima of its three states)
    flops = (FWD_FLOPS_PER_CELL + BWD_FLOPS_PER_CELL) * cells + OA_FLOPS_PER_CELL * region_cells
    # HBM traffic the design needs: every kept Forward row (M and I, 8 bytes
    # per cell) written once and read back once by the Backward pass, plus
    # the 0.5-byte traceback code of every region cell written (the
    # traceback reads a few of them again)
    traffic = 16 * cells + region_cells // 2
    s = ms / 1e3
    log(f"decode: {n_dec} targets, {len(doms)} regions, {ms:.3f} ms, {cells / s / 1e9:.1f} GCUPS")
    return {"ms": round(ms, 4), "targets": n_dec, "regions": len(doms), "cells": cells,
            "region_cells": region_cells, "gcups": round(cells / s / 1e9, 2),
            "roofline": {"fp32": {"achieved": round(flops / s / 1e12, 3), "peak": PEAK_FP32_TFLOPS,
                                  "unit": "TFLOP/s", "frac": round(flops / s / 1e12 / PEAK_FP32_TFLOPS, 4)},
                         "hbm": {"achieved": round(traffic / s / 1e9, 1), "peak": 8000.0, "unit": "GB/s",
                                 "frac": round(traffic / s / 8e12, 4), "design_bytes": traffic,
                                 "traffic": measured_traffic(args, "decode_traffic_C3.json", "hmm_decode.hip")}}}


def bench_iterations(hg, prof, calib, D, F, stream, args) -> list:
    """jackhmmer-style iterations on the GPU: each one searches with the
    current profile, decodes its Forward passes, counts their alignments
    and re-estimates the profile (prior weights 20 and 10) for the next.
    Times: the GPU part (search + decode + count, HIP events on the search
    stream) and the host part (re-estimate, upload, calibration searches)."""
    import numpy as np
    import torch
    from paper_2111_06340_amd.calibrate import calibrate
    out = []
    cur, cal = prof, calib
    for it in range(args.iterations):
        P = hg.Profile(cur, *cal)
        res = hg.alloc_results(D.n)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        torch.cuda.synchronize()
        ev[0].record(stream)
        hg.search(P, D, F, res, stream=stream)
        ev[1].record(stream)
        dec = hg.decode(P, D, flags=res["flags"], mask=hg.HMM_FWD_PASS, aln=True, stream=stream)
        ev[2].record(stream)
        counts = torch.zeros(hg.count_size(cur.M), dtype=torch.int32, device="cuda")
        hg.hmm_count(P.handle, D.handle, dec, counts, stream=stream)
        ev[3].record(stream)
        torch.cuda.synchronize()
        t = time.perf_counter()
        c = counts.cpu().numpy().astype(np.uint32)
        nxt = hg.hmm_rebuild(cur, c, 20.0, 10.0)
        ncal = calibrate(nxt)
        host_s = time.perf_counter() - t
        n_pass = int(res["counts"].cpu()[2])
        rec = {"iteration": it + 1, "vit_pass": n_pass, "regions": int(dec["n_dom"].cpu()[0]),
               "search_ms": round(ev[0].elapsed_time(ev[1]), 3), "decode_ms": round(ev[1].elapsed_time(ev[2]), 3),
               "count_ms": round(ev[2].elapsed_time(ev[3]), 3), "host_rebuild_and_calibrate_s": round(host_s, 3)}
        log(f"iteration {it + 1}: {rec}")
        out.append(rec)
        P.close()
        cur, cal = nxt, ncal
    return out


def measured_traffic(args, name: str, source: str):
    """HBM bytes per launch from committed rocprofv3 counter passes, while
    the kernel source is the one they were taken on (C3 only)."""
    path = os.path.join(ROOT, "profiles", name)
    if args.workload != "C3" or args.cutoffs or not os.path.exists(path):
        return None
    with open(path) as f:
        tr = json.load(f)
    same = (tr.get("kernel_source_sha") == kernel_source_sha(source)
            and tr.get("header_sha", kernel_source_sha("hmm_device.h")) == kernel_source_sha("hmm_device.h"))
    return tr.get("bytes_per_launch") if same else None


def kernel_source_sha(source: str = "hmm_kernels.hip") -> str:
    import hashlib
    p = os.path.join(ROOT, "paper_2111_06340_amd", "csrc", source)
    with open(p, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


if __name__ == "__main__":
    main()
