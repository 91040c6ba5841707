"""Pins of the oracle's posterior decoding, domain regions and
optimal-accuracy alignment.

Posteriors are pinned against brute-force enumeration of every Plan7 path
(each path weighted by exp(score)): the probability that each state emits
each residue, and that B / E are visited at each row.  The alignment is
pinned against enumeration of every alignment of a region, scored with the
brute-force posteriors.  Invariants (Forward total = Backward total,
emission posteriors of a residue sum to one, expected begins = expected
ends) hold at larger sizes."""
import math

import numpy as np
import pytest

import brute
import oracle
from conftest import random_profile
from test_oracle_brute import CASES, _prof, _seq, delete_favoring_case

_TN = ("MM", "MI", "MD", "IM", "II", "DM", "DD")


def _allowed(prof):
    return lambda k, n: prof.trans[k - 1, _TN.index(n)] > 0


@pytest.mark.parametrize("M,L,seed,alpha", CASES)
def test_posteriors_equal_brute_force(M, L, seed, alpha):
    prof = _prof(M, seed, alpha)
    op = oracle.OracleProfile(prof)
    x = _seq(L, seed, prof, alpha)
    d = oracle.decode(op, x)
    b = brute.posteriors(brute.float_scores(prof, L), x)
    assert d["tot"][0] == pytest.approx(b["tot"], abs=1e-10)
    assert d["tot"][1] == pytest.approx(b["tot"], abs=1e-10)
    for key in ("core", "njc", "beg", "end", "pM", "pI"):
        np.testing.assert_allclose(d[key], np.array(b[key]), rtol=0, atol=1e-11, err_msg=key)


def _zero_transition_profile(M, seed):
    """Random profile with some transitions of probability zero (a missing
    delete chain, a forbidden insert), so alignments must respect them."""
    prof = random_profile(M, seed, alpha=0.2, talpha=0.5)
    rng = np.random.default_rng(seed)
    for k in range(M - 1):
        r = rng.integers(0, 4)
        if r == 0:      # no M->D
            prof.trans[k, 2] = 0.0
        elif r == 1:    # no D->D
            prof.trans[k, 6] = 0.0
        elif r == 2:    # no M->I
            prof.trans[k, 1] = 0.0
        if r in (0, 2):
            prof.trans[k, 0:3] /= prof.trans[k, 0:3].sum()
        else:
            prof.trans[k, 5:7] = [1.0, 0.0]
    return prof


OA_CASES = [(M, L, seed, zero) for M in (1, 2, 3) for L in (1, 2, 3, 4) for seed in range(3)
            for zero in (False, True)] + [(3, 5, s, z) for s in range(3) for z in (False, True)]


@pytest.mark.parametrize("M,L,seed,zero", OA_CASES)
def test_optimal_accuracy_alignment_equals_enumeration(M, L, seed, zero):
    prof = _zero_transition_profile(M, seed) if zero else _prof(M, seed, 0.1)
    op = oracle.OracleProfile(prof)
    x = _seq(L, seed + 1, prof, 0.1)
    d = oracle.decode(op, x)
    bp = brute.posteriors(brute.float_scores(prof, L), x)
    for s in range(1, L + 1):
        for e in range(s, L + 1):
            r = oracle.oa_align(op, d, s, e)
            want = brute.oa_best(M, _allowed(prof), bp["core"], bp["pM"], bp["pI"], s, e)
            assert r["score"] == pytest.approx(want, abs=1e-10), (s, e)
            sc, ok = oracle.oa_path_score(op, d, s, e, r["code"])
            assert ok and sc == pytest.approx(r["score"], abs=1e-12)
            code = r["code"]
            nz = np.nonzero(code)[0]
            assert r["a"] == s + nz[0] and r["b"] == s + nz[-1]
            assert r["k1"] == code[nz[0]] and r["k2"] == code[nz[-1]]


def forbidden_skip_case():
    """M = 4 profile with peaked emissions whose node 2 has no D->D: for
    x = (c1, c4) the posterior puts x1 on M1 and x2 on M4 (through two hits
    joined by J), but one alignment may not hold both, since
    M1 -> D2 -> D3 -> M4 is forbidden."""
    from synth import BACKGROUND, Profile
    c = [18, 4, 1, 12]
    match = np.full((4, 20), 0.1 / 19)
    for k in range(4):
        match[k, c[k]] = 0.9
    insert = np.tile(BACKGROUND, (3, 1))
    tr = np.array([[0.1, 0.1, 0.8, 0.5, 0.5, 0.5, 0.5],
                   [0.1, 0.1, 0.8, 0.5, 0.5, 1.0, 0.0],
                   [0.8, 0.1, 0.1, 0.5, 0.5, 0.9, 0.1]])
    return Profile(4, BACKGROUND.copy(), match, insert, tr), np.array([c[0], c[3]], np.uint8)


def test_alignment_may_not_cross_a_forbidden_delete():
    prof, x = forbidden_skip_case()
    op = oracle.OracleProfile(prof)
    d = oracle.decode(op, x)
    bp = brute.posteriors(brute.float_scores(prof, 2), x)
    r = oracle.oa_align(op, d, 1, 2)
    assert r["score"] == pytest.approx(brute.oa_best(4, _allowed(prof), bp["core"], bp["pM"], bp["pI"], 1, 2),
                                       abs=1e-12)
    assert d["pM"][0, 0] > 0.3 and d["pM"][1, 3] > 0.3
    assert not oracle.oa_path_score(op, d, 1, 2, np.array([1, 4], np.int16))[1]
    assert np.count_nonzero(r["code"]) == 1


def test_alignment_follows_a_delete_path():
    # M1 -> D2 -> M3 is the only strong explanation of (c1, c3)
    prof, x = delete_favoring_case()
    op = oracle.OracleProfile(prof)
    d = oracle.decode(op, x)
    r = oracle.oa_align(op, d, 1, 2)
    assert list(r["code"]) == [1, 3]
    assert oracle.oa_path_score(op, d, 1, 2, np.array([1, 3], np.int16))[1]
    assert not oracle.oa_path_score(op, d, 1, 2, np.array([3, 1], np.int16))[1]
    assert not oracle.oa_path_score(op, d, 1, 2, np.array([-1, 3], np.int16))[1]   # starts in I
    assert not oracle.oa_path_score(op, d, 1, 2, np.array([1, -1], np.int16))[1]   # ends in I


def test_path_validity_respects_zero_transitions():
    prof = random_profile(4, 3)
    prof.trans[1, :3] = [0.5, 0.5, 0.0]      # node 2: no M->D
    prof.trans[1, 5:7] = [1.0, 0.0]          # node 2: no D->D
    op = oracle.OracleProfile(prof)
    x = np.array([1, 2, 3], np.uint8)
    d = oracle.decode(op, x)
    ok = lambda o, dd, code: oracle.oa_path_score(o, dd, 1, 3, np.array(code, np.int16))[1]
    assert ok(op, d, [1, 2, 3]) and ok(op, d, [1, -1, 2]) and ok(op, d, [1, 3, 4])  # M1->D2->M3
    assert not ok(op, d, [2, 4, 0])          # M2->D3 needs MD_2 = 0
    assert not ok(op, d, [1, 4, 0])          # M1->D2->D3->M4 needs DD_2 = 0
    assert not ok(op, d, [1, 0, 2])          # the aligned range must be contiguous
    assert not ok(op, d, [0, 0, 0])
    prof.trans[1, 5:7] = [0.5, 0.5]
    op2 = oracle.OracleProfile(prof)
    d2 = oracle.decode(op2, x)
    assert ok(op2, d2, [1, 4, 0]) and ok(op2, d2, [0, 1, 0])


def test_regions_rule_on_written_out_posteriors():
    rt1, rt2 = oracle.RT1, oracle.RT2
    core = np.array([0.05, 0.10, 0.2, 0.25, 0.099, 0.3, 0.24, 0.11, 0.09, 0.12, 0.2, 0.1, 0.5, 0.1])
    # runs >= 0.10: [2..4] (has 0.25), [6..8] (has 0.3), [10..14] (has 0.5)
    assert oracle.regions(core, rt1, rt2) == [(2, 4), (6, 8), (10, 14)]
    # a run that never reaches rt1 is dropped
    assert oracle.regions(np.array([0.2, 0.24, 0.05, 0.3]), rt1, rt2) == [(4, 4)]
    assert oracle.regions(np.zeros(5), rt1, rt2) == []
    assert oracle.regions(np.ones(3), rt1, rt2) == [(1, 3)]


@pytest.mark.parametrize("M,L,seed", [(40, 120, 0), (90, 300, 1), (150, 260, 2)])
def test_sum_rules_at_larger_sizes(M, L, seed):
    prof = random_profile(M, seed, alpha=0.5)
    op = oracle.OracleProfile(prof)
    from synth import sample_homologs
    rng = np.random.default_rng(seed)
    x = rng.integers(0, 20, L).astype(np.uint8)
    h = sample_homologs(rng, prof, 1)[0][: L // 2]
    x[10:10 + h.size] = h
    d = oracle.decode(op, x)
    assert d["tot"][1] == pytest.approx(d["tot"][0], abs=1e-9 * abs(d["tot"][0]) + 1e-9)
    assert d["tot"][0] == pytest.approx(oracle.fwd_f64(op, x), abs=1e-9)
    np.testing.assert_allclose(d["core"] + d["njc"].sum(axis=1), 1.0, atol=1e-10)
    np.testing.assert_allclose(d["core"], d["pM"].sum(1) + d["pI"].sum(1), atol=1e-12)
    assert d["beg"].sum() == pytest.approx(d["end"].sum(), abs=1e-9)
    assert np.all(d["pI"][:, M - 1] == 0.0)
    assert d["beg"][0] >= 0 and np.all(d["end"] <= 1 + 1e-12)


def test_planted_homolog_is_found_and_aligned():
    # background flanks drawn from the background composition, as in the
    # workloads; a homolog sampled from the profile in the middle
    from synth import gen, make_profile, sample_homologs
    M = 120
    prof = make_profile(M, 11)
    op = oracle.OracleProfile(prof)
    rng = np.random.default_rng(3)
    h = sample_homologs(rng, prof, 1)[0]
    x = np.concatenate([gen.background_residues(rng, 150), h, gen.background_residues(rng, 100)])
    dec, doms = oracle.domains(op, x)
    assert len(doms) == 1
    big = doms[0]
    lo, hi = 151, 150 + h.size
    assert big["s"] <= lo + 10 and big["e"] >= hi - 10
    assert big["a"] <= lo + 10 and big["b"] >= hi - 10
    assert big["k1"] <= 10 and big["k2"] >= M - 10
    assert 0.5 < big["nexp"] < 1.5
    # the alignment's match states are strictly increasing along the residues
    ks = [abs(int(c)) for c in big["code"] if c != 0]
    assert all(b >= a for a, b in zip(ks, ks[1:]))
    assert math.isfinite(big["score"])
