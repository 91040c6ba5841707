"""GPU parity of posterior decoding (hmm_decode, through the C ABI) against
the CPU oracle on the same seeded inputs.

The GPU computes in fp32, the oracle in fp64, so the bar is a tolerance,
derived below, on every float; decisions taken from floats are compared
where they are unique:
  - core posterior of every residue of every decoded target and the
    expected number of domains: within the tolerance;
  - regions: identical, except for targets with a residue whose core
    posterior lies within the tolerance of a region threshold, where the
    GPU's regions must be the ones its own posteriors define;
  - alignment of each region: the GPU's path must be a valid path of the
    model, and its objective value, evaluated with the oracle's fp64
    posteriors, must be within the tolerance of the oracle's optimum (near-
    ties between different paths are both correct); the reported score and
    the expected domain count within the tolerance; residues outside every
    region carry code 0.

Tolerance: the posteriors are products of fp32 Forward and Backward values,
each the end of a chain of about L rows of a few roundings (unit 2^-24); the
error grows at most linearly, so |pp_gpu - pp| <= 2e-5 + 8 * 2^-24 * L
(about 5e-4 at L = 1000).  An objective value is a sum of at most R such
terms (R the region length) plus the fp32 sum itself: R times the
posterior tolerance.
"""
import numpy as np
import pytest

import oracle
import paper_2111_06340_amd as hg
from conftest import random_profile
from synth import gen
from test_gpu_parity import NTHREADS, _ragged_db, announce, full_db, sample_ids, sub_db
from test_oracle_decode import _zero_transition_profile

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


def tol_pp(L: int) -> float:
    return 2e-5 + 8 * U * L


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    hg.lib()
    return torch


def run(prof, residues, offsets, calib, F, decode_all=False, max_dom=None):
    """Search, then decode (the Forward passes, or every target); host copies."""
    import torch
    P = hg.Profile(prof, *calib)
    D = hg.Database(residues, offsets)
    announce(f"decode M={prof.M} n={D.n} residues={D.n_residues} max_len={D.max_len} F={F} all={decode_all}")
    out = hg.alloc_results(D.n)
    hg.search(P, D, F, out)
    dec = hg.decode(P, D, flags=None if decode_all else out["flags"], mask=hg.HMM_FWD_PASS, pp=True, aln=True,
                    max_dom=max_dom)
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in out.items()}
    g = dict(exp_dom=dec["exp_dom"].cpu().numpy(), pp=dec["pp"].cpu().numpy(), aln=dec["aln"].cpu().numpy(),
             doms=hg.domains_table(dec), n_dom=int(dec["n_dom"].cpu()[0]))
    P.close()
    D.close()
    return res, g


def compare_decode(prof, residues, offsets, g, ids, what=""):
    """Check the GPU's decoding of targets `ids` (caller indices) against
    the oracle; returns the largest errors seen."""
    op = oracle.OracleProfile(prof)
    by_t = {}
    for d in g["doms"]:
        by_t.setdefault(d["target"], []).append(d)
    st = dict(n=0, pp=0.0, exp=0.0, oa=0.0, score=0.0, nexp=0.0, regions=0, ambiguous=0)
    for t in ids:
        t = int(t)
        lo, hi = int(offsets[t]), int(offsets[t + 1])
        x = residues[lo:hi]
        L = x.size
        tp = tol_pp(L)
        dec, odoms = oracle.domains(op, x)
        pp = g["pp"][lo:hi].astype(np.float64)
        e_pp = float(np.max(np.abs(pp - dec["core"])))
        assert e_pp <= tp, f"{what} target {t} L={L}: core posterior off by {e_pp:.3g} (tol {tp:.3g})"
        e_exp = abs(float(g["exp_dom"][t]) - float(dec["end"].sum()))
        assert e_exp <= tp * L, f"{what} target {t}: expected domains off by {e_exp:.3g}"
        gd = by_t.get(t, [])
        amb = bool(np.any(np.abs(dec["core"] - oracle.RT1) <= tp) or np.any(np.abs(dec["core"] - oracle.RT2) <= tp))
        greg = [(d["s"], d["e"]) for d in gd]
        if not amb:
            assert greg == [(d["s"], d["e"]) for d in odoms], f"{what} target {t}: regions {greg} vs oracle"
        else:
            st["ambiguous"] += 1
            own = oracle.regions(g["pp"][lo:hi].astype(np.float32).astype(np.float64),
                                 float(np.float32(oracle.RT1)), float(np.float32(oracle.RT2)))
            assert greg == own, f"{what} target {t}: regions {greg} vs its own posteriors {own}"
        aln = g["aln"][lo:hi]
        covered = np.zeros(L, bool)
        for d in gd:
            s, e = d["s"], d["e"]
            covered[s - 1:e] = True
            code = aln[s - 1:e].astype(np.int16)
            sc, ok = oracle.oa_path_score(op, dec, s, e, code)
            assert ok, f"{what} target {t} region {(s, e)}: invalid alignment {code[:20]}..."
            best = oracle.oa_align(op, dec, s, e)["score"]
            R = e - s + 1
            tol = tp * R + 8 * U * R
            assert sc >= best - tol, f"{what} target {t} region {(s, e)}: path value {sc} < optimum {best}"
            assert abs(d["score"] - best) <= tol, f"{what} target {t}: score {d['score']} vs {best}"
            nz = np.nonzero(code)[0]
            assert d["a"] == s + nz[0] and d["b"] == s + nz[-1]
            assert d["k1"] == code[nz[0]] and d["k2"] == code[nz[-1]]
            e_nexp = abs(d["nexp"] - float(dec["end"][s - 1:e].sum()))
            assert e_nexp <= tp * R
            st["oa"] = max(st["oa"], best - sc)
            st["score"] = max(st["score"], abs(d["score"] - best))
            st["nexp"] = max(st["nexp"], e_nexp)
        assert np.all(aln[~covered] == 0), f"{what} target {t}: codes outside regions"
        st["n"] += 1
        st["pp"] = max(st["pp"], e_pp)
        st["exp"] = max(st["exp"], e_exp)
        st["regions"] += len(gd)
    return st


def _decoded(res, all_targets: bool):
    return np.arange(res["flags"].size) if all_targets else np.nonzero(res["flags"] & hg.HMM_FWD_PASS)[0]


def _check_selection(res, g, all_targets: bool):
    ids = _decoded(res, all_targets)
    sel = np.zeros(res["flags"].size, bool)
    sel[ids] = True
    assert np.all(np.isfinite(g["exp_dom"][sel])) and np.all(np.isnan(g["exp_dom"][~sel]))
    assert g["n_dom"] == len(g["doms"])
    return ids


# ------------------------------------------------------------ workloads

def test_decode_c1_sampled():
    w = gen.WORKLOADS["C1"]
    prof = gen.workload_profile(w)
    db = gen.workload_database(w)
    calib = oracle.calibrate(oracle.OracleProfile(prof), nthreads=NTHREADS)
    res, g = run(prof, db.residues, db.offsets, calib, w.F)
    ids = _check_selection(res, g, False)
    assert ids.size == db.n
    pick = sample_ids(db, 300, 60, seed=1)
    st = compare_decode(prof, db.residues, db.offsets, g, pick, "C1")
    announce(f"C1 decode: {g['n_dom']} regions over {ids.size} targets; sampled {st}")


@pytest.mark.parametrize("name,n", [("C2", 20000), ("C3", 3000), ("C5", 600)])
def test_decode_reduced_workload(name, n):
    w = gen.WORKLOADS[name]
    prof = gen.workload_profile(w)
    db = gen.workload_database(w, n=n, prof=prof)
    calib = oracle.calibrate(oracle.OracleProfile(prof), nthreads=NTHREADS)
    res, g = run(prof, db.residues, db.offsets, calib, w.F)
    ids = _check_selection(res, g, False)
    assert ids.size > 0
    st = compare_decode(prof, db.residues, db.offsets, g, ids, name)
    announce(f"{name} reduced n={n} decode: {ids.size} targets {st}")


def test_decode_c3_full_size_sampled():
    w = gen.WORKLOADS["C3"]
    prof, db = full_db("C3")
    calib = oracle.calibrate(oracle.OracleProfile(prof), nthreads=NTHREADS)
    res, g = run(prof, db.residues, db.offsets, calib, w.F)
    ids = _check_selection(res, g, False)
    rng = np.random.default_rng(7)
    pick = rng.choice(ids, size=min(40, ids.size), replace=False)
    res_s, off_s = sub_db(db, pick)
    # the sample's own arrays, with the GPU outputs of those targets
    gs = dict(pp=np.concatenate([g["pp"][db.offsets[t]:db.offsets[t + 1]] for t in pick]),
              aln=np.concatenate([g["aln"][db.offsets[t]:db.offsets[t + 1]] for t in pick]),
              exp_dom=g["exp_dom"][pick],
              doms=[dict(d, target=int(np.nonzero(pick == d["target"])[0][0])) for d in g["doms"]
                    if d["target"] in set(pick.tolist())])
    st = compare_decode(prof, res_s, off_s, gs, np.arange(pick.size), "C3 full")
    planted = np.intersect1d(db.planted, ids)
    with_region = {d["target"] for d in g["doms"]}
    frac = np.mean([t in with_region for t in planted]) if planted.size else 1.0
    announce(f"C3 full decode: {ids.size} targets, {g['n_dom']} regions, planted with a region {frac:.3f}; "
             f"sampled {st}")
    assert frac > 0.95


# ------------------------------------------------------------ edge cases

@pytest.mark.parametrize("M", [1, 2, 3, 63, 64, 65, 128, 129, 734, 1000, 2500])
def test_decode_edge_lengths_and_profile_sizes(M):
    prof = gen.make_profile(M, 700 + M)
    lengths = [1, 2, 3, 5, 63, 64, 65, 255, 256, 257, 600] if M < 2000 else [1, 2, 65, 257, 2600, 3000]
    res_, off = _ragged_db(prof, M, lengths=lengths, homolog_every=2)
    res, g = run(prof, res_, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0), decode_all=True)
    ids = _check_selection(res, g, True)
    st = compare_decode(prof, res_, off, g, ids, f"edge M={M}")
    announce(f"decode edge M={M}: {st}")


@pytest.mark.parametrize("seed", [0, 1])
def test_decode_zero_probability_transitions(seed):
    prof = _zero_transition_profile(150, 60 + seed)
    res_, off = _ragged_db(prof, 10 + seed, lengths=[40, 150, 300, 151, 500, 90] * 2, homolog_every=1)
    res, g = run(prof, res_, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0), decode_all=True)
    st = compare_decode(prof, res_, off, g, _check_selection(res, g, True), f"zero-trans {seed}")
    announce(f"decode zero transitions seed={seed}: {st}")


def test_decode_random_transitions():
    prof = random_profile(300, 41, alpha=0.3, talpha=0.6)
    res_, off = _ragged_db(prof, 5, lengths=[50, 300, 301, 700, 1200, 90, 5, 333] * 2, homolog_every=2)
    res, g = run(prof, res_, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0), decode_all=True)
    st = compare_decode(prof, res_, off, g, _check_selection(res, g, True), "random-trans")
    announce(f"decode random transitions: {st}")


def test_decode_two_domains_in_one_target():
    prof = gen.make_profile(90, 21)
    rng = np.random.default_rng(4)
    seqs = []
    for _ in range(6):
        h = gen.sample_homologs(rng, prof, 2)
        seqs.append(np.concatenate([gen.background_residues(rng, 60), h[0], gen.background_residues(rng, 120),
                                    h[1], gen.background_residues(rng, 40)]))
    off = np.zeros(len(seqs) + 1, np.int64)
    off[1:] = np.cumsum([s.size for s in seqs])
    res_ = np.concatenate(seqs)
    res, g = run(prof, res_, off, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0), decode_all=True)
    st = compare_decode(prof, res_, off, g, _check_selection(res, g, True), "two domains")
    assert st["regions"] >= 10
    announce(f"decode two domains: {st}")


def test_decode_selection_capacity_and_empty():
    import torch
    prof = gen.make_profile(50, 2)
    P = hg.Profile(prof, 0.0, 0.0, 0.0)
    # empty database
    D0 = hg.Database(np.zeros(0, np.uint8), np.zeros(1, np.int64))
    out0 = hg.decode(P, D0, flags=None)
    torch.cuda.synchronize()
    assert int(out0["n_dom"].cpu()[0]) == 0
    D0.close()
    # a selection that holds nothing, then a capacity smaller than the regions found
    res_, off = _ragged_db(prof, 9, lengths=[300] * 8, homolog_every=1)
    D = hg.Database(res_, off)
    flags = torch.zeros(D.n, dtype=torch.uint8, device="cuda")
    o1 = hg.decode(P, D, flags=flags, mask=hg.HMM_FWD_PASS)
    o2 = hg.decode(P, D, flags=None, max_dom=3)
    o3 = hg.decode(P, D, flags=None)
    torch.cuda.synchronize()
    assert int(o1["n_dom"].cpu()[0]) == 0 and torch.isnan(o1["exp_dom"]).all()
    n_all = int(o3["n_dom"].cpu()[0])
    assert n_all >= 6 and int(o2["n_dom"].cpu()[0]) == n_all
    t2 = {tuple(r) for r in o2["dom"].cpu().numpy().tolist()}
    t3 = {tuple(r) for r in o3["dom"][:n_all].cpu().numpy().tolist()}
    assert len(t2) == 3 and t2 <= t3
    D.close()
    P.close()


@pytest.mark.parametrize("ci", range(3))
def test_search_and_decode_match_frozen_oracle_fixtures(ci):
    """The GPU against the oracle outputs frozen in tests/golden (written by
    tests/golden/make_golden.py from the oracle alone)."""
    from test_golden import case_database, case_profile, load_cases
    c = load_cases()[ci]
    prof = case_profile(c)
    res_, off = case_database(c)
    res, g = run(prof, res_, off, tuple(c["calib"]), tuple(c["cutoffs"]), decode_all=True)
    op = oracle.OracleProfile(prof)
    by_t = {}
    for d in g["doms"]:
        by_t.setdefault(d["target"], []).append(d)
    for t, want in enumerate(c["targets"]):
        L = len(want["residues"])
        assert int(res["msv"][t]) == want["msv"] and int(res["vit"][t]) == want["vit"]
        assert int(res["flags"][t]) == want["flags"]
        assert abs(float(res["fwd"][t]) - want["fwd"]) <= 1e-3 + 1e-5 * abs(want["fwd"])
        pp = g["pp"][off[t]:off[t + 1]].astype(np.float64)
        assert np.max(np.abs(pp - np.array(want["core"]))) <= tol_pp(L)
        gd = by_t.get(t, [])
        core = np.array(want["core"])
        amb = np.any(np.abs(core - oracle.RT1) <= tol_pp(L)) or np.any(np.abs(core - oracle.RT2) <= tol_pp(L))
        if not amb:
            assert [(d["s"], d["e"]) for d in gd] == [(d["s"], d["e"]) for d in want["domains"]]
            x = res_[off[t]:off[t + 1]]
            dec = oracle.decode(op, x)
            for d, w in zip(gd, want["domains"]):
                code = g["aln"][off[t] + d["s"] - 1:off[t] + d["e"]].astype(np.int16)
                sc, ok = oracle.oa_path_score(op, dec, d["s"], d["e"], code)
                R = d["e"] - d["s"] + 1
                assert ok and sc >= w["score"] - tol_pp(L) * R - 8 * U * R
                assert abs(d["score"] - w["score"]) <= tol_pp(L) * R + 8 * U * R
    announce(f"golden case {ci} M={c['M']}: {len(c['targets'])} targets ok")


def _oracle_counts(M, residues, offsets, g):
    tot = dict(match=np.zeros((M, 20), np.int64), insert=np.zeros((max(M - 1, 0), 20), np.int64),
               trans=np.zeros((max(M - 1, 0), 7), np.int64))
    for d in g["doms"]:
        t = d["target"]
        x = residues[offsets[t]:offsets[t + 1]]
        code = g["aln"][offsets[t] + d["s"] - 1:offsets[t] + d["e"]]
        c = oracle.count_alignment(M, x, d["s"], code)
        for k in tot:
            tot[k] += c[k]
    return np.concatenate([tot["match"].ravel(), tot["insert"].ravel(), tot["trans"].ravel()])


@pytest.mark.parametrize("M,n", [(1, 50), (90, 400), (734, 300), (2500, 40)])
def test_counts_of_the_decoded_alignments(M, n):
    """hmm_count on the GPU's own alignments equals the oracle's counting
    of those alignments, exactly (integer counts)."""
    import torch
    prof = gen.make_profile(M, 40 + M)
    db = gen.make_database(n, 77 + M, prof, 0.3, len_hi=3000 if M > 1000 else 1000)
    P = hg.Profile(prof, 0.0, 0.0, 0.0)
    D = hg.Database(db.residues, db.offsets)
    dec = hg.decode(P, D, flags=None, aln=True)
    counts = torch.zeros(hg.count_size(M), dtype=torch.int32, device="cuda")
    hg.hmm_count(P.handle, D.handle, dec, counts)
    hg.hmm_count(P.handle, D.handle, dec, counts)       # accumulates: twice the counts
    torch.cuda.synchronize()
    g = dict(doms=hg.domains_table(dec), aln=dec["aln"].cpu().numpy())
    want = _oracle_counts(M, db.residues, db.offsets, g)
    got = counts.cpu().numpy().astype(np.int64)
    assert np.array_equal(got, 2 * want)
    announce(f"counts M={M}: {len(g['doms'])} domains, {int(want.sum())} events ok")
    P.close()
    D.close()


def test_one_search_iteration_end_to_end():
    """search -> decode -> count -> rebuild -> search with the new profile:
    the rebuilt profile equals the oracle's estimate from the same counts,
    and the second search matches the oracle searching with it."""
    import torch
    from paper_2111_06340_amd.calibrate import calibrate
    w = gen.WORKLOADS["C2"]
    prof = gen.workload_profile(w)
    db = gen.workload_database(w, n=4000, prof=prof)
    calib = oracle.calibrate(oracle.OracleProfile(prof), nthreads=NTHREADS)
    F = (0.02, 1e-3, 1.0)
    P = hg.Profile(prof, *calib)
    D = hg.Database(db.residues, db.offsets)
    out = hg.search(P, D, F)
    dec = hg.decode(P, D, flags=out["flags"], mask=hg.HMM_FWD_PASS, aln=True)
    counts = torch.zeros(hg.count_size(prof.M), dtype=torch.int32, device="cuda")
    hg.hmm_count(P.handle, D.handle, dec, counts)
    torch.cuda.synchronize()
    c = counts.cpu().numpy().astype(np.uint32)
    g = dict(doms=hg.domains_table(dec), aln=dec["aln"].cpu().numpy())
    assert np.array_equal(c.astype(np.int64), _oracle_counts(prof.M, db.residues, db.offsets, g))
    new = hg.hmm_rebuild(prof, c, 20.0, 10.0)
    M = prof.M
    cd = dict(match=c[:M * 20].reshape(M, 20), insert=c[M * 20:M * 40 - 20].reshape(M - 1, 20),
              trans=c[M * 40 - 20:].reshape(M - 1, 7))
    ref = oracle.rebuild_profile(prof, cd, 20.0, 10.0)
    np.testing.assert_allclose(new.match, ref.match, atol=1e-15)
    np.testing.assert_allclose(new.trans, ref.trans, atol=1e-15)
    calib2 = calibrate(new)
    P2 = hg.Profile(new, *calib2)
    out2 = hg.search(P2, D, F)
    torch.cuda.synchronize()
    g2 = {k: v.cpu().numpy() for k, v in out2.items()}
    o2 = oracle.search(oracle.OracleProfile(ref), db.residues, db.offsets, calib2, F, nthreads=NTHREADS)
    from test_gpu_parity import compare
    st = compare(g2, o2, what="iteration 2")
    announce(f"iteration: {len(g['doms'])} domains counted; second search ok {st}")
    P.close()
    P2.close()
    D.close()
