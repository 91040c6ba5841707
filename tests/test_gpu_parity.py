"""GPU parity: the HIP search (through the C ABI) against the CPU oracle on
the same seeded inputs.

Bar: MSV scores, Viterbi scores (int16, and exact int32 after overflow) and
all flag bits bit-exact; Forward within 1e-3 + 1e-5 |x| nats of the fp64
oracle.  Sizes: whole workloads where the oracle finishes in seconds;
sampled targets (random plus every kind of planted homolog) at the full
workload sizes, in the same launch configuration the benchmark times.
"""
import math
import sys
import time

import numpy as np
import pytest

import oracle
import paper_2111_06340_amd as hg
from conftest import random_profile
from synth import gen

pytestmark = pytest.mark.gpu

FWD_ABS, FWD_REL = 1e-3, 1e-5
NTHREADS = 16


def announce(msg):
    print(f"[gpu-parity] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    hg.lib()
    return torch


def run_gpu(prof, residues, offsets, calib, F, stream=None, tail_mode=0):
    import torch
    P = hg.Profile(prof, *calib)
    D = hg.Database(residues, offsets)
    out = hg.alloc_results(D.n)
    mode = hg.hmm_db_fused_tail(D.handle, tail_mode)
    announce(f"search M={prof.M} n={D.n} residues={D.n_residues} max_len={D.max_len} F={F} tail mode {mode}")
    hg.search(P, D, F, out, stream=stream)
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in out.items()}
    P.close()
    D.close()
    return res


def compare(g, o, idx=None, what=""):
    """g: GPU results (caller order), o: oracle results for targets idx."""
    if idx is None:
        idx = np.arange(o["msv"].size)
    gm, gv, gf, gl = g["msv"][idx], g["vit"][idx], g["fwd"][idx], g["flags"][idx]
    bad = np.nonzero(gm != o["msv"])[0]
    assert bad.size == 0, f"{what} msv mismatch at {idx[bad[:5]]}: gpu {gm[bad[:5]]} oracle {o['msv'][bad[:5]]}"
    bad = np.nonzero(gl != o["flags"])[0]
    assert bad.size == 0, f"{what} flags mismatch at {idx[bad[:5]]}: gpu {gl[bad[:5]]} oracle {o['flags'][bad[:5]]}"
    bad = np.nonzero(gv != o["vit"])[0]
    assert bad.size == 0, f"{what} vit mismatch at {idx[bad[:5]]}: gpu {gv[bad[:5]]} oracle {o['vit'][bad[:5]]}"
    ran = ~np.isnan(o["fwd"])
    assert np.array_equal(ran, ~np.isnan(gf)), f"{what} Forward ran on different targets"
    err = np.abs(gf[ran].astype(np.float64) - o["fwd"][ran])
    tol = FWD_ABS + FWD_REL * np.abs(o["fwd"][ran])
    if err.size:
        worst = int(np.argmax(err - tol))
        assert np.all(err <= tol), (f"{what} fwd off by {err[worst]:.3g} (tol {tol[worst]:.3g}) at "
                                    f"{idx[ran][worst]}: gpu {gf[ran][worst]} oracle {o['fwd'][ran][worst]}")
    return dict(n=idx.size, fwd_ran=int(ran.sum()), fwd_max_err=float(err.max()) if err.size else 0.0,
                vit_ovf=int(np.sum((o["flags"] & oracle.F_VIT_OVF) != 0)),
                msv_ovf=int(np.sum((o["flags"] & oracle.F_MSV_OVF) != 0)))


def oracle_search(prof, residues, offsets, calib, F):
    op = oracle.OracleProfile(prof)
    return oracle.search(op, residues, offsets, calib, F, nthreads=NTHREADS)


def sub_db(db, idx):
    seqs = [db.seq(int(i)) for i in idx]
    off = np.zeros(len(seqs) + 1, np.int64)
    off[1:] = np.cumsum([s.size for s in seqs])
    return np.concatenate(seqs) if seqs else np.zeros(0, np.uint8), off


# ------------------------------------------------------------ whole workloads

def test_c1_all_stages_on_every_target():
    w = gen.WORKLOADS["C1"]
    prof = gen.workload_profile(w)
    db = gen.workload_database(w)
    calib = oracle.calibrate(oracle.OracleProfile(prof), nthreads=NTHREADS)
    g = run_gpu(prof, db.residues, db.offsets, calib, w.F)
    o = oracle_search(prof, db.residues, db.offsets, calib, w.F)
    st = compare(g, o, what="C1")
    assert st["fwd_ran"] == db.n            # F = 1: every target reaches Forward
    announce(f"C1 ok {st}")


@pytest.mark.parametrize("name,n", [("C2", 20000), ("C3", 3000), ("C5", 600)])
def test_reduced_workload_filter_pipeline(name, n):
    w = gen.WORKLOADS[name]
    prof = gen.workload_profile(w)
    db = gen.workload_database(w, n=n, prof=prof)
    calib = oracle.calibrate(oracle.OracleProfile(prof), nthreads=NTHREADS)
    g = run_gpu(prof, db.residues, db.offsets, calib, w.F)
    o = oracle_search(prof, db.residues, db.offsets, calib, w.F)
    st = compare(g, o, what=name)
    assert st["fwd_ran"] > 0
    announce(f"{name} reduced n={n} ok {st}")


@pytest.mark.parametrize("name,n", [("C1", 5000), ("C3", 2000)])
def test_reduced_workload_every_stage(name, n):
    # thresholds at 1: Viterbi, rescore and Forward on every target
    w = gen.WORKLOADS[name]
    prof = gen.workload_profile(w)
    db = gen.workload_database(w, n=n, prof=prof)
    calib = (0.0, 0.0, 0.0)
    g = run_gpu(prof, db.residues, db.offsets, calib, (1.0, 1.0, 1.0))
    o = oracle_search(prof, db.residues, db.offsets, calib, (1.0, 1.0, 1.0))
    st = compare(g, o, what=name)
    assert st["fwd_ran"] == db.n
    announce(f"{name} all-stages ok {st}")


# ------------------------------------------------------------ full sizes, sampled

_DB_CACHE = {}


def full_db(name):
    if name not in _DB_CACHE:
        w = gen.WORKLOADS[name]
        t = time.time()
        prof = gen.workload_profile(w)
        _DB_CACHE.clear()
        _DB_CACHE[name] = (prof, gen.workload_database(w, prof=prof))
        announce(f"generated {name} in {time.time() - t:.1f}s")
    return _DB_CACHE[name]


def sample_ids(db, n_random, n_planted, seed):
    rng = np.random.default_rng(seed)
    r = rng.choice(db.n, size=min(n_random, db.n), replace=False)
    p = db.planted[rng.choice(db.planted.size, size=min(n_planted, db.planted.size), replace=False)] \
        if db.planted.size else np.zeros(0, np.int64)
    return np.unique(np.concatenate([r, p]).astype(np.int64))


def whole_db_properties(g, what=""):
    """Properties of a full-database result that need no oracle."""
    fl = g["flags"]
    assert np.all((fl & hg.HMM_VIT_RAN != 0) == (fl & hg.HMM_MSV_PASS != 0)), what
    assert np.all((fl & hg.HMM_FWD_RAN != 0) == (fl & hg.HMM_VIT_PASS != 0)), what
    assert np.all(g["vit"][(fl & hg.HMM_VIT_RAN) == 0] == np.iinfo(np.int32).min), what
    assert np.all(np.isnan(g["fwd"][(fl & hg.HMM_FWD_RAN) == 0])), what
    return float(np.mean((fl & hg.HMM_MSV_PASS) != 0))


@pytest.mark.parametrize("name,stride", [("C2", 1), ("C3", 1), ("C5", 50)])
def test_full_size(name, stride):
    """The whole workload database in the benchmark's launch configuration
    (default pipeline); every target (C2, C3) or every 50th target in
    caller order (C5, where the oracle would need about six minutes for
    all 2M) compared with the oracle, element by element."""
    w = gen.WORKLOADS[name]
    prof, db = full_db(name)
    calib = oracle.calibrate(oracle.OracleProfile(prof), nthreads=NTHREADS)
    g = run_gpu(prof, db.residues, db.offsets, calib, w.F)
    t = time.time()
    if stride == 1:
        idx = np.arange(db.n, dtype=np.int64)
        o = oracle_search(prof, db.residues, db.offsets, calib, w.F)
    else:
        idx = np.arange(0, db.n, stride, dtype=np.int64)
        res, off = sub_db(db, idx)
        o = oracle_search(prof, res, off, calib, w.F)
    announce(f"{name} oracle on {idx.size} of {db.n} targets in {time.time() - t:.1f}s")
    st = compare(g, o, idx, what=name)
    announce(f"{name} full n={db.n}: {idx.size} targets compared ok {st}")
    msv_pass = whole_db_properties(g, name)
    assert 0.005 < msv_pass < 0.06, msv_pass


def test_c4_group_full_size():
    """C4 exactly as the benchmark times it: one hmm_search_group call of
    the 64 profiles (M 50-400) against the full C3 database, each through
    its own handle, on the current stream.  The group MSV kernels then
    score about 120 targets per wave.  For every profile 150 random and 30
    planted targets are compared with the oracle; for one profile of each
    group size (1, 2 and 3 vectors per lane) every target is compared, bit
    for bit, with a single hmm_search of the same profile, whose MSV kernel
    the whole-database C3 test checks against the oracle."""
    import torch
    _, db = full_db("C3")
    profiles = gen.c4_profiles()
    F = gen.WORKLOADS["C3"].F
    t = time.time()
    calibs = [oracle.calibrate(oracle.OracleProfile(p), nthreads=NTHREADS) for p in profiles]
    announce(f"C4: {len(profiles)} profiles calibrated by the oracle in {time.time() - t:.1f}s")
    Ps = [hg.Profile(p, *c) for p, c in zip(profiles, calibs)]
    D = hg.Database(db.residues, db.offsets)
    handles = [D] + [D.share() for _ in profiles[1:]]
    announce(f"C4 group search: {len(Ps)} profiles, n={D.n}, residues={D.n_residues}")
    outs = hg.search_group(Ps, handles, F)
    torch.cuda.synchronize()
    firsts = {}
    for i, p in enumerate(profiles):
        firsts.setdefault((p.M + 127) // 128, i)
    for i, (p, c, out) in enumerate(zip(profiles, calibs, outs)):
        g = {k: v.cpu().numpy() for k, v in out.items()}
        idx = sample_ids(db, 150, 30, seed=200 + i)
        res, off = sub_db(db, idx)
        o = oracle_search(p, res, off, c, F)
        st = compare(g, o, idx, what=f"C4 group profile {i} M={p.M}")
        whole_db_properties(g, f"C4 profile {i}")
        counts = g["counts"]
        fl = g["flags"]
        assert counts[0] == np.sum((fl & hg.HMM_MSV_PASS) != 0)
        assert counts[2] == np.sum((fl & hg.HMM_VIT_PASS) != 0)
        if i in firsts.values():
            single = hg.alloc_results(D.n)
            H = D.share()
            hg.search(Ps[i], H, F, single)
            torch.cuda.synchronize()
            H.close()
            s1 = {k: v.cpu().numpy() for k, v in single.items()}
            for k in ("msv", "vit", "flags", "counts"):
                assert np.array_equal(g[k], s1[k]), f"C4 group vs single {k} differ, profile {i} M={p.M}"
            ran = ~np.isnan(s1["fwd"])
            assert np.array_equal(ran, ~np.isnan(g["fwd"]))
            assert np.array_equal(g["fwd"][ran], s1["fwd"][ran])
            announce(f"C4 profile {i} M={p.M}: all {D.n} targets equal the single search")
        announce(f"C4 group profile {i} M={p.M} ok {st}")
    for H in handles:
        H.close()
    for P in Ps:
        P.close()


# ------------------------------------------------------------ edge cases

EDGE_LENGTHS = [1, 2, 3, 4, 5, 7, 15, 16, 17, 63, 64, 65, 255, 256, 257, 511, 512, 513, 767, 768, 769,
                1023, 1024, 1025, 2047, 4096, 7000]


def _ragged_db(prof, seed, lengths=EDGE_LENGTHS, homolog_every=3):
    rng = np.random.default_rng(seed)
    seqs = []
    homs = gen.sample_homologs(rng, prof, len(lengths)) if homolog_every <= len(lengths) else []
    for i, L in enumerate(lengths):
        s = gen.background_residues(rng, L)
        if homs and i % homolog_every == 0:
            h = homs[i][:L]
            o = int(rng.integers(0, L - h.size + 1))
            s[o:o + h.size] = h
        seqs.append(s)
    off = np.zeros(len(seqs) + 1, np.int64)
    off[1:] = np.cumsum([s.size for s in seqs])
    return np.concatenate(seqs), off


@pytest.mark.parametrize("M", [1, 2, 3, 77, 127, 128, 129, 255, 256, 257, 733, 734, 800, 1000, 1100, 1281,
                               1700, 2000])
def test_edge_lengths_and_profile_sizes(M):
    prof = gen.make_profile(M, 500 + M)
    res, off = _ragged_db(prof, M)
    calib = (0.0, 0.0, 0.0)
    F = (1.0, 1.0, 1.0)
    g = run_gpu(prof, res, off, calib, F)
    o = oracle_search(prof, res, off, calib, F)
    st = compare(g, o, what=f"edge M={M}")
    announce(f"edge M={M} ok {st}")


def test_largest_profile():
    M = hg.HMM_MAX_M
    prof = gen.make_profile(M, 77)
    res, off = _ragged_db(prof, 1, lengths=[1, 31, 300, 3100, 600], homolog_every=3)
    g = run_gpu(prof, res, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0))
    o = oracle_search(prof, res, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0))
    announce(f"M={M} ok {compare(g, o, what='max M')}")


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_random_transitions_exercise_insert_and_delete_paths(seed):
    prof = random_profile(300, 40 + seed, alpha=0.3, talpha=0.6)
    res, off = _ragged_db(prof, seed, lengths=[50, 300, 301, 700, 1200, 90, 2000, 5, 333] * 3,
                          homolog_every=2)
    g = run_gpu(prof, res, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0))
    o = oracle_search(prof, res, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0))
    announce(f"random transitions seed={seed} ok {compare(g, o, what='random-trans')}")


@pytest.mark.parametrize("M", [1990, 2047, 2300, 2560])
def test_random_transitions_long_profiles(M):
    # 16 and 20 vectors per lane: the Viterbi instances that read their
    # transition planes from LDS every row; per-node transitions, so that a
    # plane or vector read at the wrong place changes some score
    prof = random_profile(M, 90 + M, alpha=0.3, talpha=0.6)
    res, off = _ragged_db(prof, M, lengths=[50, 300, 700, 1200, 90, 5, 333, 2600], homolog_every=2)
    g = run_gpu(prof, res, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0))
    o = oracle_search(prof, res, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0))
    announce(f"random transitions M={M} ok {compare(g, o, what='random-trans long')}")


def _peaked(M, seed, p_top=0.81):
    rng = np.random.default_rng(seed)
    c = rng.integers(0, 19, size=M)
    bg = np.full(20, 0.05)
    match = np.full((M, 20), (1 - p_top) / 19)
    match[np.arange(M), c] = p_top
    insert = np.tile(bg, (M - 1, 1))
    trans = np.tile([0.9, 0.05, 0.05, 0.6, 0.4, 0.5, 0.5], (M - 1, 1))
    return gen.Profile(M, bg, match, insert, trans), c.astype(np.uint8)


@pytest.mark.parametrize("M", [40, 200, 700, 800, 1000, 2500])
def test_overflow_and_rescore(M):
    prof, c = _peaked(M, M)
    rng = np.random.default_rng(M)
    seqs = [c, np.concatenate([gen.background_residues(rng, 50), c, gen.background_residues(rng, 30)])]
    for d in (0.05, 0.2, 0.4, 0.6):
        mut = c.copy()
        m = rng.random(M) < d
        mut[m] = rng.integers(0, 20, size=int(m.sum()))
        seqs.append(mut)
    seqs.append(np.concatenate([c[: M // 2], c[M // 3:]]))           # repeat: two hits
    seqs.append(gen.background_residues(rng, 400))
    off = np.zeros(len(seqs) + 1, np.int64)
    off[1:] = np.cumsum([s.size for s in seqs])
    res = np.concatenate(seqs)
    for F in ((1.0, 1.0, 1.0), (0.02, 1e-3, 1.0)):
        calib = (-8.0, -9.0, -4.0)
        g = run_gpu(prof, res, off, calib, F)
        o = oracle_search(prof, res, off, calib, F)
        st = compare(g, o, what=f"peaked M={M}")
        assert st["vit_ovf"] >= 1 and st["msv_ovf"] >= 1
        announce(f"overflow M={M} F={F} ok {st}")


@pytest.mark.parametrize("M", [40, 64, 65, 77, 128, 129, 200, 256, 257, 320, 384, 385])
def test_fused_and_staged_tails_agree(M):
    """Profiles up to 384 nodes can run Viterbi, rescore and Forward as one
    kernel (hmm_db_fused_tail mode 2; by default when F2 = 1); the staged
    kernels (mode 1) must give the same results, bit for bit, and both the
    oracle's.  A
    peaked profile against its planted homologs (int16 overflows, several
    hits), mutated copies and background, and a profile with random per-node
    transitions; open cutoffs and the filter cutoffs; the counts as well."""
    import torch
    peaked, c = _peaked(M, 1000 + M)
    rng = np.random.default_rng(M)
    seqs = [c, np.concatenate([gen.background_residues(rng, 60), c, gen.background_residues(rng, 700)])]
    for d in (0.1, 0.3, 0.5):
        mut = c.copy()
        m = rng.random(M) < d
        mut[m] = rng.integers(0, 20, size=int(m.sum()))
        seqs.append(mut)
    seqs.append(np.concatenate([c[: M // 2], c[M // 3:]]))
    seqs += [gen.background_residues(rng, int(n)) for n in rng.integers(1, 1500, size=40)]
    off = np.zeros(len(seqs) + 1, np.int64)
    off[1:] = np.cumsum([s.size for s in seqs])
    res = np.concatenate(seqs)
    rand = random_profile(M, 300 + M, alpha=0.3, talpha=0.6)
    for prof, calib in ((peaked, (-8.0, -9.0, -4.0)), (rand, (0.0, 0.0, 0.0))):
        for F in ((1.0, 1.0, 1.0), (0.02, 1e-3, 1.0)):
            o = oracle_search(prof, res, off, calib, F)
            got = {}
            for mode in (1, 2):
                P = hg.Profile(prof, *calib)
                D = hg.Database(res, off)
                assert hg.hmm_db_fused_tail(D.handle) == 3    # the default: fused when F2 = 1
                assert hg.hmm_db_fused_tail(D.handle, mode) == mode
                out = hg.alloc_results(D.n)
                announce(f"tails M={M} mode={mode} F={F}")
                hg.search(P, D, F, out)
                torch.cuda.synchronize()
                got[mode] = {k: v.cpu().numpy() for k, v in out.items()}
                P.close()
                D.close()
                st = compare(got[mode], o, what=f"tail mode {mode} M={M} F={F}")
                fl = o["flags"]
                assert got[mode]["counts"][1] == np.sum((fl & hg.HMM_VIT_OVF) != 0)
                assert got[mode]["counts"][2] == np.sum((fl & hg.HMM_VIT_PASS) != 0)
                assert got[mode]["counts"][3] == np.sum((fl & hg.HMM_FWD_PASS) != 0)
            for k in ("msv", "vit", "flags", "counts"):
                assert np.array_equal(got[1][k], got[2][k]), k
            assert np.array_equal(got[1]["fwd"].view(np.uint32), got[2]["fwd"].view(np.uint32))
            announce(f"tails M={M} F={F} agree {st}")
    # with the composition-bias filter between MSV and Viterbi (its own
    # parity test covers the oracle side): the two tails agree bit for bit
    got = {}
    for mode in (1, 2):
        P = hg.Profile(peaked, -8.0, -9.0, -4.0)
        D = hg.Database(res, off)
        hg.hmm_db_fused_tail(D.handle, mode)
        out = hg.alloc_results(D.n)
        hg.search(P, D, (0.5, 1.0, 1.0), out, bias_filter=True)
        torch.cuda.synchronize()
        got[mode] = {k: v.cpu().numpy() for k, v in out.items()}
        P.close()
        D.close()
    for k in ("msv", "vit", "flags", "counts"):
        assert np.array_equal(got[1][k], got[2][k]), f"bias filter: {k}"
    assert np.array_equal(got[1]["fwd"].view(np.uint32), got[2]["fwd"].view(np.uint32))
    assert np.array_equal(got[1]["bias"].view(np.uint32), got[2]["bias"].view(np.uint32))
    assert np.any((got[2]["flags"] & hg.HMM_FWD_RAN) != 0)


@pytest.mark.parametrize("M", [700, 900, 1500, 2600])
def test_long_delete_runs(M):
    """A peaked profile whose middle half is skipped by a cheap delete run,
    searched with the consensus minus that block: the best path (and much
    of the Forward mass) runs through hundreds of consecutive delete
    states, across many lanes of the profile layout and, for long
    profiles, across the waves that share one target."""
    prof, c = _peaked(M, 7 * M)
    a, b = M // 4, 3 * M // 4
    tr = prof.trans.copy()
    tr[a - 1] = [0.6, 0.05, 0.35, 0.6, 0.4, 0.5, 0.5]      # M_a -> D_{a+1} likely
    tr[a:b, 5], tr[a:b, 6] = 0.01, 0.99                    # D -> D runs cheap
    prof = gen.Profile(M, prof.bg, prof.match, prof.insert, tr)
    rng = np.random.default_rng(M)
    seqs = [np.concatenate([c[:a], c[b:]]),
            np.concatenate([gen.background_residues(rng, 40), c[:a], c[b + M // 8:],
                            gen.background_residues(rng, 25)]),
            np.concatenate([c[:a // 2], c[b:]]),
            gen.background_residues(rng, 300)]
    off = np.zeros(len(seqs) + 1, np.int64)
    off[1:] = np.cumsum([s.size for s in seqs])
    res = np.concatenate(seqs)
    calib = (-8.0, -9.0, -4.0)
    F = (1.0, 1.0, 1.0)
    g = run_gpu(prof, res, off, calib, F)
    o = oracle_search(prof, res, off, calib, F)
    st = compare(g, o, what=f"delete runs M={M}")
    announce(f"delete runs M={M} ok {st}")


def _high_bias_profiles():
    """Small profiles whose BIAS8 is pushed up by one near-impossible
    residue, so that xB - ENTRY8 + BIAS8 exceeds 255 on short targets: the
    uint8 add of BIAS8 then saturates before COST8 is subtracted (the MSV
    corner where the saturation order matters)."""
    out = []
    for seed in range(12):
        rng = np.random.default_rng(1000 + seed)
        M = int(rng.integers(1, 12))
        prof = gen.make_profile(M, 1000 + seed)
        k, r = int(rng.integers(0, M)), int(rng.integers(0, 20))
        prof.match[k, r] = 10.0 ** (-float(rng.uniform(9, 14)))
        prof.match[k] /= prof.match[k].sum()
        out.append((prof, r))
    return out


def test_msv_biased_entry_saturates_before_cost():
    hit = 0
    for i, (prof, rare) in enumerate(_high_bias_profiles()):
        sc = oracle.OracleProfile(prof).scalars()
        hit += oracle.BASE8 - 1 - sc["entry8"] + sc["bias8"] > 255   # xB - ENTRY8 at L = 1
        rng = np.random.default_rng(77 + i)
        lengths = rng.integers(1, 31, 500)
        res = rng.integers(0, 20, int(lengths.sum())).astype(np.uint8)
        res[rng.random(res.size) < 0.3] = rare
        off = np.zeros(lengths.size + 1, np.int64)
        off[1:] = np.cumsum(lengths)
        g = run_gpu(prof, res, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0))
        o = oracle_search(prof, res, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0))
        announce(f"high-bias profile {i} M={prof.M} bias8={sc['bias8']} entry8={sc['entry8']} "
                 f"ok {compare(g, o, what=f'high-bias {i}')}")
    assert hit >= 4, "too few profiles reach the saturation corner"


def test_degenerate_and_extreme_profiles():
    rng = np.random.default_rng(5)
    # BIAS8 clamps at 255: MSV overflows on every target
    bg = np.full(20, 0.05)
    match = np.full((30, 20), 0.05)
    match[7, 0] = 1e-300
    match[7, 1] += 0.05 - 1e-300
    deg = gen.Profile(30, bg, match, np.tile(bg, (29, 1)), np.tile([0.9, 0.05, 0.05, 0.6, 0.4, 0.5, 0.5], (29, 1)))
    # extreme: score -32768 in int16, zero inserts and zero transitions
    ext = gen.make_profile(60, 9)
    ext.match[3, 0] = 1e-30
    ext.match[3, 1] += 0.5
    ext.match[3] /= ext.match[3].sum()
    ext.insert[2, :] = 0.0
    ext.insert[2, 5] = 1.0
    ext.trans[4] = [1.0, 0.0, 0.0, 1.0, 0.0, 0.0, 1.0]
    ext.trans[10] = [0.0, 0.5, 0.5, 0.0, 1.0, 1.0, 0.0]
    # BIAS8 between 128 and 254: the MSV kernel's unsigned (two-step) path
    mid = gen.make_profile(80, 10)
    mid.match[5, 0] = 1e-15
    mid.match[5, 1] += 0.3
    mid.match[5] /= mid.match[5].sum()
    assert 128 <= hg.hmm_debug_tables(mid)["bias8"] <= 254
    assert hg.hmm_debug_tables(gen.make_profile(80, 10))["bias8"] <= 127
    # (ext has I->I = 1 at node 3: no finite path can be sampled from it, so
    # its targets are background sequences with the rare residue injected)
    for name, prof, every in (("degenerate", deg, 2), ("extreme", ext, 10**9), ("bias128+", mid, 2)):
        res, off = _ragged_db(prof, 3, lengths=[1, 10, 60, 61, 300, 1000, 64, 128, 129], homolog_every=every)
        res = res.copy()
        res[::7] = 0                                  # many copies of the near-impossible residue
        g = run_gpu(prof, res, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0))
        o = oracle_search(prof, res, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0))
        announce(f"{name} ok {compare(g, o, what=name)}")
    assert rng is not None


@pytest.mark.parametrize("M", [734, 1000, 2500])
def test_zero_probabilities_in_long_profiles(M):
    """Impossible insert emissions (probability exactly 0: score minus
    infinity), zero transitions and near-impossible match emissions
    (1e-30; a match probability of 0 is rejected at upload) in profiles of
    12, 16 and 40 vectors per lane (the one-wave int32 rescore and Forward,
    and the cooperative ones), against homologs that overflow int16 and
    targets full of the rare residue: the int32 rescore meets insert values
    far below its -2^30 floor and must still equal the oracle."""
    rng = np.random.default_rng(M)
    prof = gen.make_profile(M, 3100 + M)
    match, insert, trans = prof.match.copy(), prof.insert.copy(), prof.trans.copy()
    for k in rng.choice(M, size=M // 5, replace=False):       # residue 0 near-impossible at a fifth of the nodes
        match[k, 0] = 1e-30
        match[k] /= match[k].sum()
    for k in rng.choice(M - 1, size=M // 10, replace=False):  # inserts that emit one residue only
        insert[k] = 0.0
        insert[k, int(rng.integers(1, 20))] = 1.0
    for k in rng.choice(M - 1, size=M // 10, replace=False):  # no M->D, no I->I, no D->D at some nodes
        trans[k] = [0.9, 0.1, 0.0, 1.0, 0.0, 1.0, 0.0]
    prof = gen.Profile(M, prof.bg, match, insert, trans)
    homs = gen.sample_homologs(rng, prof, 4)
    seqs = [np.concatenate([gen.background_residues(rng, 30), h, gen.background_residues(rng, 20)]) for h in homs]
    seqs += [np.zeros(400, np.uint8), gen.background_residues(rng, 900)]
    mixed = gen.background_residues(rng, 1500)
    mixed[::3] = 0
    seqs.append(mixed)
    off = np.zeros(len(seqs) + 1, np.int64)
    off[1:] = np.cumsum([x.size for x in seqs])
    res = np.concatenate(seqs)
    F = (1.0, 1.0, 1.0)
    g = run_gpu(prof, res, off, (0.0, 0.0, 0.0), F)
    o = oracle_search(prof, res, off, (0.0, 0.0, 0.0), F)
    st = compare(g, o, what=f"zero probabilities M={M}")
    assert st["vit_ovf"] >= 1
    announce(f"zero probabilities M={M} ok {st}")


def _rare_residue_profile(M, seed):
    """Residue 0 has background frequency 1e-9 and match probability 1/2 at
    every node: each match of it scores about 14,400 units (1/500 bit), so
    a run of it drives the Viterbi score towards the int32 rescore's bound."""
    prof = gen.make_profile(M, seed)
    bg = prof.bg.copy()
    bg[1:] *= (1.0 - 1e-9) / bg[1:].sum()
    bg[0] = 1e-9
    match = prof.match.copy()
    match[:, 1:] *= 0.5 / match[:, 1:].sum(axis=1, keepdims=True)
    match[:, 0] = 0.5
    insert = np.tile(bg, (M - 1, 1))
    return gen.Profile(M, bg, match, insert, prof.trans)


def test_scores_near_the_int32_bound_and_beyond():
    """hmm_search is exact up to the bound (longest target x largest
    emission score < 2^29), here with targets whose best score lies within
    a factor 1.3 of it through the cooperative long-profile kernels, and
    rejects a database one step past it with HMM_ERANGE before enqueuing
    anything."""
    import torch
    M = 2000
    prof = _rare_residue_profile(M, 31)
    tab = hg.hmm_debug_tables(prof)
    s_max = int(max(tab["msc16"].max(), tab["isc16"].max(), 0))
    limit = -(-(1 << 29) // s_max)                # shortest length the bound rejects
    assert 30000 < limit < 40000, (s_max, limit)
    rng = np.random.default_rng(8)
    L = limit - 1
    run = np.zeros(L, np.uint8)                   # residue 0 throughout: about L * s_max
    mixed = gen.background_residues(rng, L)
    mixed[rng.random(L) < 0.7] = 0
    seqs = [run, mixed, gen.background_residues(rng, 500), np.zeros(3, np.uint8)]
    off = np.zeros(len(seqs) + 1, np.int64)
    off[1:] = np.cumsum([x.size for x in seqs])
    res = np.concatenate(seqs)
    g = run_gpu(prof, res, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0))
    o = oracle_search(prof, res, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0))
    st = compare(g, o, what="near the int32 bound")
    assert g["vit"][0] > (1 << 29) // 2, g["vit"][0]
    announce(f"int32 bound: s_max={s_max} L={L} vit={g['vit'][0]} ok {st}")
    # one residue longer: rejected by hmm_search and hmm_search_group
    P = hg.Profile(prof, 0.0, 0.0, 0.0)
    D = hg.Database(np.zeros(limit, np.uint8), np.array([0, limit], np.int64))
    out = hg.alloc_results(D.n)
    with pytest.raises(hg.HmmError) as e:
        hg.search(P, D, (1.0, 1.0, 1.0), out)
    assert e.value.status == hg.HMM_ERANGE
    with pytest.raises(hg.HmmError) as e:
        hg.hmm_search_group([P.handle], [D.handle], [(1.0, 1.0, 1.0)], [out])
    assert e.value.status == hg.HMM_ERANGE
    torch.cuda.synchronize()
    D.close()
    P.close()


def test_empty_and_single_target_databases():
    import torch
    prof = gen.make_profile(50, 1)
    P = hg.Profile(prof, 0.0, 0.0, 0.0)
    D0 = hg.Database(np.zeros(0, np.uint8), np.zeros(1, np.int64))
    assert D0.n == 0
    out = hg.alloc_results(0)
    hg.search(P, D0, (1.0, 1.0, 1.0), out)
    torch.cuda.synchronize()
    for L in (1, 2, 777):
        x = gen.background_residues(np.random.default_rng(L), L)
        off = np.array([0, L], np.int64)
        g = run_gpu(prof, x, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0))
        o = oracle_search(prof, x, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0))
        compare(g, o, what=f"single L={L}")
    D0.close()
    P.close()


def test_repeated_searches_streams_and_threshold_changes():
    import torch
    w = gen.WORKLOADS["C2"]
    prof = gen.workload_profile(w)
    db = gen.workload_database(w, n=5000, prof=prof)
    calib = oracle.calibrate(oracle.OracleProfile(prof), nthreads=NTHREADS)
    P = hg.Profile(prof, *calib)
    D = hg.Database(db.residues, db.offsets)
    s = torch.cuda.Stream()
    outs = []
    for F in ((0.02, 1e-3, 1.0), (1.0, 1.0, 1.0), (0.02, 1e-3, 1.0), (0.1, 0.01, 0.5)):
        out = hg.alloc_results(D.n)
        with torch.cuda.stream(s):
            hg.search(P, D, F, out)
        outs.append((F, out))
    torch.cuda.synchronize()
    for F, out in outs:
        g = {k: v.cpu().numpy() for k, v in out.items()}
        o = oracle_search(prof, db.residues, db.offsets, calib, F)
        if F[2] < 1.0:
            # FWD_PASS is an fp32 compare: check it only away from the cutoff
            _, _, ft = np.vectorize(lambda L: oracle.thresholds(calib, F, int(L)), otypes=[int, int, float])(
                np.diff(db.offsets))
            close = np.abs(o["fwd"] - ft) <= FWD_ABS + FWD_REL * np.abs(o["fwd"])
            g["flags"] = np.where(close, (g["flags"] & ~np.uint8(hg.HMM_FWD_PASS)) |
                                  (o["flags"] & np.uint8(hg.HMM_FWD_PASS)), g["flags"])
        st = compare(g, o, what=f"repeat F={F}")
        counts = out["counts"].cpu().numpy()
        fl = o["flags"]
        assert counts[0] == np.sum((fl & hg.HMM_MSV_PASS) != 0)
        assert counts[1] == np.sum((fl & hg.HMM_VIT_OVF) != 0)
        assert counts[2] == np.sum((fl & hg.HMM_VIT_PASS) != 0)
        announce(f"repeat F={F} ok {st} counts={counts.tolist()}")
    P.close()
    D.close()


def test_stages_that_receive_no_target():
    """Searches whose later stages get no target -- nothing passes MSV; then
    MSV passes but none passes Viterbi or overflows int16 -- between full
    searches on the same handle: the empty Viterbi, rescore and Forward
    launches return before staging their tables, the counters of the
    previous search do not leak, and every result equals the oracle's."""
    import torch
    prof = gen.make_profile(200, 31)
    db = gen.random_sequences(4321, 3000, 300)
    calib = oracle.calibrate(oracle.OracleProfile(prof), nthreads=NTHREADS)
    P = hg.Profile(prof, *calib)
    D = hg.Database(db.residues, db.offsets)
    for F in ((1.0, 1.0, 1.0), (1e-30, 1.0, 1.0), (0.05, 1e-30, 1.0), (1.0, 1.0, 1.0)):
        out = hg.alloc_results(D.n)
        hg.search(P, D, F, out)
        torch.cuda.synchronize()
        g = {k: v.cpu().numpy() for k, v in out.items()}
        o = oracle_search(prof, db.residues, db.offsets, calib, F)
        st = compare(g, o, what=f"empty stages F={F}")
        fl = o["flags"]
        counts = out["counts"].cpu().numpy()
        assert counts[0] == np.sum((fl & hg.HMM_MSV_PASS) != 0)
        assert counts[1] == np.sum((fl & hg.HMM_VIT_OVF) != 0)
        assert counts[2] == np.sum((fl & hg.HMM_VIT_PASS) != 0)
        if F[0] < 1e-20:
            assert counts[0] == 0 and np.all(g["vit"] == np.iinfo(np.int32).min) and np.all(np.isnan(g["fwd"]))
        if F[1] < 1e-20:
            assert counts[0] > 0 and counts[1] == 0 and counts[2] == 0 and np.all(np.isnan(g["fwd"]))
        announce(f"empty stages F={F} ok {st} counts={counts.tolist()}")
    P.close()
    D.close()


def test_concurrent_searches_on_shared_database_handles():
    """hmm_db_share: four profiles searched at once on four streams through
    four handles of one uploaded database; every result equals the oracle's,
    and the shared residues outlive the handle that uploaded them."""
    import torch
    w = gen.WORKLOADS["C2"]
    db = gen.workload_database(w, n=6000, prof=gen.workload_profile(w))
    profs = [gen.make_profile(M, 900 + M) for M in (60, 200, 450, 801)]
    calibs = [oracle.calibrate(oracle.OracleProfile(p), nthreads=NTHREADS) for p in profs]
    Ps = [hg.Profile(p, *c) for p, c in zip(profs, calibs)]
    D = hg.Database(db.residues, db.offsets)
    handles = [D.share() for _ in range(4)]
    D.close()                                   # the shares keep the data alive
    streams = [torch.cuda.Stream() for _ in handles]
    F = (0.05, 0.01, 1.0)
    outs = [hg.alloc_results(db.n) for _ in handles]
    for _ in range(2):                          # twice: the second round reuses every scratch
        for P, H, s, o in zip(Ps, handles, streams, outs):
            hg.search(P, H, F, o, stream=s)
    torch.cuda.synchronize()
    for p, c, o in zip(profs, calibs, outs):
        g = {k: v.cpu().numpy() for k, v in o.items()}
        ref = oracle_search(p, db.residues, db.offsets, c, F)
        st = compare(g, ref, what=f"shared M={p.M}")
        announce(f"shared handle M={p.M} ok {st}")
    for H in handles:
        H.close()
    for P in Ps:
        P.close()


@pytest.mark.parametrize("chunks", [1, 3, 8])
def test_pipelined_chunks_give_identical_results(chunks):
    """The search is split into pipelined chunks of the sorted database;
    results (and counts) do not depend on how many."""
    import torch
    w = gen.WORKLOADS["C2"]
    prof = gen.workload_profile(w)
    db = gen.workload_database(w, n=9000, prof=prof)
    calib = oracle.calibrate(oracle.OracleProfile(prof), nthreads=NTHREADS)
    P = hg.Profile(prof, *calib)
    D = hg.Database(db.residues, db.offsets)
    assert hg.hmm_db_pipeline(D.handle, chunks) == chunks
    F = (0.05, 0.01, 1.0)
    out = hg.alloc_results(D.n)
    hg.search(P, D, F, out)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in out.items()}
    o = oracle_search(prof, db.residues, db.offsets, calib, F)
    st = compare(g, o, what=f"chunks={chunks}")
    fl = o["flags"]
    assert list(g["counts"][:3]) == [np.sum((fl & m) != 0) for m in (hg.HMM_MSV_PASS, hg.HMM_VIT_OVF, hg.HMM_VIT_PASS)]
    announce(f"pipelined chunks={chunks} ok {st}")
    P.close()
    D.close()


def _low_complexity_db(prof, base, seed):
    """A reduced workload database plus targets made of the residues the
    profile's mean composition favours most (they pass raw MSV but carry
    a large composition bias)."""
    rng = np.random.default_rng(seed)
    odds = prof.match.mean(axis=0) / prof.bg
    top = np.argsort(odds)[-3:]
    seqs = [base.seq(i) for i in range(base.n)]
    for L in (30, 60, 120, 250, 400, 800):
        seqs.append(rng.choice(top, size=L).astype(np.uint8))
        mix = gen.background_residues(rng, L)
        mix[rng.random(L) < 0.5] = top[0]
        seqs.append(mix)
    off = np.zeros(len(seqs) + 1, np.int64)
    off[1:] = np.cumsum([s.size for s in seqs])
    return np.concatenate(seqs), off


@pytest.mark.parametrize("name,n", [("C2", 8000), ("C3", 2000), ("C5", 300)])
def test_bias_filter(name, n):
    """The composition-bias filter between MSV and Viterbi: bias scores
    within their fp32 tolerance; the filter decision, and everything after
    it, exact except where the corrected MSV score lies within that
    tolerance of the cutoff (there the GPU's decision must follow its own
    bias score)."""
    import torch
    w = gen.WORKLOADS[name]
    prof = gen.workload_profile(w)
    base = gen.workload_database(w, n=n, prof=prof)
    res, off = _low_complexity_db(prof, base, 5)
    op = oracle.OracleProfile(prof)
    calib = oracle.calibrate(op, nthreads=NTHREADS)
    F = (0.05, 0.01, 1.0)
    P = hg.Profile(prof, *calib)
    D = hg.Database(res, off)
    out = hg.alloc_results(D.n)
    hg.search(P, D, F, out, bias_filter=True)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in out.items()}
    o = oracle.search(op, res, off, calib, F, nthreads=NTHREADS, bias_filter=True)
    lengths = np.diff(off)
    ran = ~np.isnan(o["beta"])
    assert np.array_equal(ran, ~np.isnan(g["bias"]))
    tol = 1e-5 + 4 * 2.0 ** -24 * lengths
    assert np.all(np.abs(g["bias"][ran] - o["beta"][ran]) <= tol[ran])
    thr8 = np.array([oracle.thresholds(calib, F, int(L))[0] for L in lengths])
    margin = o["msv"] - oracle.S8 * np.maximum(o["beta"], 0.0) - thr8
    amb = ran & (np.abs(margin) <= oracle.S8 * tol) & ((o["flags"] & oracle.F_MSV_OVF) == 0)
    for t in np.nonzero(amb)[0]:      # the GPU follows its own bias score
        keep = float(g["msv"][t]) - np.float32(oracle.S8) * max(float(g["bias"][t]), 0.0) >= thr8[t]
        assert bool(g["flags"][t] & hg.HMM_BIAS_PASS) == keep
    idx = np.nonzero(~amb)[0]
    sub = {k: v[idx] for k, v in o.items() if k in ("msv", "vit", "fwd", "flags")}
    st = compare(g, sub, idx, what=f"bias {name}")
    dropped = int(np.sum(((o["flags"] & oracle.F_MSV_PASS) != 0) & ((o["flags"] & oracle.F_BIAS_PASS) == 0)))
    assert dropped >= 6
    announce(f"bias filter {name} n={D.n}: {int(ran.sum())} scored, {dropped} dropped, {int(amb.sum())} near the "
             f"cutoff, max bias error {np.max(np.abs(g['bias'][ran] - o['beta'][ran])):.2e} ok {st}")
    P.close()
    D.close()


def _group_db(profs, seed, n_bg=2500):
    """Background targets of the C2 length law, the ragged edge lengths,
    and homologs of every profile (so that every profile overflows MSV
    somewhere and reaches its later stages)."""
    rng = np.random.default_rng(seed)
    w = gen.WORKLOADS["C2"]
    base = gen.workload_database(w, n=n_bg, prof=profs[0])
    seqs = [base.seq(i) for i in range(base.n)]
    seqs += [gen.background_residues(rng, L) for L in EDGE_LENGTHS]
    for p in profs:
        for h in gen.sample_homologs(rng, p, 3):
            L = int(h.size + rng.integers(0, 200))
            s = gen.background_residues(rng, L)
            o = int(rng.integers(0, L - h.size + 1))
            s[o:o + h.size] = h
            seqs.append(s)
    order = rng.permutation(len(seqs))
    seqs = [seqs[i] for i in order]
    off = np.zeros(len(seqs) + 1, np.int64)
    off[1:] = np.cumsum([s.size for s in seqs])
    return np.concatenate(seqs), off


def test_search_group_matches_oracle_and_single_searches():
    """hmm_search_group: profiles of every MSV group size (1-3 vectors per
    lane, grouped up to 4, 3 and 2 at a time) and larger ones that run
    alone, each with its own cutoffs (one with the composition-bias
    filter), against one database through distinct handles.  Every result
    equals the oracle's and, bit for bit, the single hmm_search's; a second
    group call (scratch reused, cutoffs changed) again matches."""
    import torch
    Ms = [50, 77, 100, 127, 128, 200, 255, 256, 300, 383, 384, 734, 60]
    profs = []
    for i, M in enumerate(Ms):
        if i % 3 == 2:   # peaked random transitions and emissions: many triggers and delete runs
            profs.append(random_profile(M, 4400 + M, alpha=0.3, talpha=0.5))
        else:
            profs.append(gen.make_profile(M, 4300 + M))
    res, off = _group_db(profs, 4500)
    calibs = [oracle.calibrate(oracle.OracleProfile(p), nthreads=NTHREADS, n=100) for p in profs]
    Ps = [hg.Profile(p, *c) for p, c in zip(profs, calibs)]
    D = hg.Database(res, off)
    handles = [D] + [D.share() for _ in profs[1:]]
    Fs = [(0.05, 0.01, 1.0), (0.2, 0.05, 1.0), (1.0, 1.0, 1.0)] * 5
    Fs = Fs[:len(profs)]
    bias = [i == 4 for i in range(len(profs))]
    for rnd in range(2):
        if rnd == 1:
            Fs = [(0.02, 1e-3, 1.0)] * len(profs)
        announce(f"group round {rnd}: {len(profs)} profiles M={Ms} n={D.n} residues={D.n_residues}")
        outs = hg.search_group(Ps, handles, Fs, bias_filter=bias)
        torch.cuda.synchronize()
        for i, (p, c, o) in enumerate(zip(profs, calibs, outs)):
            g = {k: v.cpu().numpy() for k, v in o.items()}
            single = hg.alloc_results(D.n)
            H = D.share()
            hg.search(Ps[i], H, Fs[i], single, bias_filter=bias[i])
            torch.cuda.synchronize()
            H.close()
            s1 = {k: v.cpu().numpy() for k, v in single.items()}
            for k in ("msv", "vit", "flags", "counts"):
                assert np.array_equal(g[k], s1[k]), f"group vs single {k} differ, profile {i} M={p.M}"
            assert np.array_equal(np.isnan(g["fwd"]), np.isnan(s1["fwd"]))
            ran = ~np.isnan(g["fwd"])
            assert np.array_equal(g["fwd"][ran], s1["fwd"][ran])
            if bias[i]:
                continue   # the bias filter's own parity test covers the oracle side
            ref = oracle_search(p, res, off, c, Fs[i])
            st = compare(g, ref, what=f"group M={p.M}")
            announce(f"group round {rnd} profile {i} M={p.M} ok {st}")
    for H in handles:
        H.close()
    for P in Ps:
        P.close()


def test_search_group_several_targets_per_wave():
    """Every group size of the group MSV kernels (4, 3 and 2 profiles at 1,
    2 and 3 vectors per lane, plus a profile left alone) against 60,000
    targets: the launch keeps 8,192 waves resident, so each wave scores
    about seven targets in turn (its next-target prefetch, per-target
    state reset and table reuse).  Every target of every profile is
    compared with the oracle, and with the single hmm_search."""
    import torch
    Ms = [50, 90, 127, 64, 100, 128, 200, 255, 256, 383]
    profs = [random_profile(M, 6100 + M, alpha=0.3, talpha=0.5) if i % 4 == 1 else gen.make_profile(M, 6000 + M)
             for i, M in enumerate(Ms)]
    rng = np.random.default_rng(6200)
    base = gen.make_database(60000, 6201, None, 0.0)
    seqs = [base.seq(i) for i in range(base.n)]
    for p in profs:                            # planted homologs of every profile
        for h in gen.sample_homologs(rng, p, 4):
            L = int(h.size + rng.integers(0, 150))
            s = gen.background_residues(rng, L)
            o = int(rng.integers(0, L - h.size + 1))
            s[o:o + h.size] = h
            seqs.append(s)
    order = rng.permutation(len(seqs))
    seqs = [seqs[i] for i in order]
    off = np.zeros(len(seqs) + 1, np.int64)
    off[1:] = np.cumsum([x.size for x in seqs])
    res = np.concatenate(seqs)
    calibs = [oracle.calibrate(oracle.OracleProfile(p), nthreads=NTHREADS, n=100) for p in profs]
    Ps = [hg.Profile(p, *c) for p, c in zip(profs, calibs)]
    D = hg.Database(res, off)
    handles = [D] + [D.share() for _ in profs[1:]]
    F = (0.05, 0.01, 1.0)
    announce(f"group of {len(profs)} profiles M={Ms} against n={D.n} residues={D.n_residues}")
    outs = hg.search_group(Ps, handles, F)
    torch.cuda.synchronize()
    for i, (p, c, o) in enumerate(zip(profs, calibs, outs)):
        g = {k: v.cpu().numpy() for k, v in o.items()}
        ref = oracle_search(p, res, off, c, F)
        st = compare(g, ref, what=f"group/multi-target M={p.M}")
        single = hg.alloc_results(D.n)
        H = D.share()
        hg.search(Ps[i], H, F, single)
        torch.cuda.synchronize()
        H.close()
        s1 = {k: v.cpu().numpy() for k, v in single.items()}
        for k in ("msv", "vit", "flags", "counts"):
            assert np.array_equal(g[k], s1[k]), f"group vs single {k} differ, profile {i} M={p.M}"
        assert st["msv_ovf"] >= 1
        announce(f"group/multi-target profile {i} M={p.M} ok {st}")
    for H in handles:
        H.close()
    for P in Ps:
        P.close()


def test_search_group_rejects_bad_groups():
    w = gen.WORKLOADS["C1"]
    prof = gen.workload_profile(w)
    db = gen.workload_database(w, n=200, prof=prof)
    P = hg.Profile(prof, 0.0, 0.0, 0.0)
    D = hg.Database(db.residues, db.offsets)
    S = D.share()
    E = hg.Database(db.residues, db.offsets)
    F = (0.5, 0.5, 1.0)
    outs = [hg.alloc_results(D.n) for _ in range(2)]

    def status(profiles, dbs, Fs, o):
        try:
            hg.hmm_search_group([p.handle for p in profiles], [d.handle for d in dbs], Fs, o)
        except hg.HmmError as e:
            return e.status
        return hg.HMM_OK

    assert status([P, P], [D, D], [F, F], outs) == hg.HMM_EINVAL        # one handle twice
    assert status([P, P], [D, E], [F, F], outs) == hg.HMM_EINVAL        # two databases
    assert status([P, P], [D, S], [F, (0.0, 0.5, 1.0)], outs) == hg.HMM_EINVAL
    assert status([], [], [], []) == hg.HMM_EINVAL
    assert status([P, P], [D, S], [F, F], outs) == hg.HMM_OK
    import torch
    torch.cuda.synchronize()
    for h in (S, D, E, P):
        h.close()


def test_packed16_probe_rate_is_plausible():
    """hmm_probe_pk16: the sustained packed 16-bit rate lies between a third
    of the datasheet peak and the peak at a 10 % higher clock."""
    import torch
    ops, ms = hg.hmm_probe_pk16(torch.cuda.current_stream())
    announce(f"packed 16-bit probe: {ops / 1e12:.2f} Tops/s in {ms:.3f} ms")
    assert ms > 0
    assert 26e12 < ops < 86.5e12
