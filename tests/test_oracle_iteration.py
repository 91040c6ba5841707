"""Pins of the oracle's profile re-estimation (one search iteration): the
counts of an alignment written out by hand, and the properties the
estimate must have."""
import numpy as np
import pytest

import oracle
from conftest import random_profile
from synth import gen

MM, MI, MD, IM, II, DM, DD = range(7)


def test_counts_of_a_written_out_alignment():
    # residues 3..9 of x aligned as M1 M2 I2 I2 M3 (M6 via D4 D5) M7, one flank residue
    M = 8
    x = np.array([5, 6, 0, 1, 2, 3, 4, 7, 8, 9], np.uint8)
    code = [1, 2, -2, -2, 3, 6, 7, 0]            # residues 3..10
    c = oracle.count_alignment(M, x, 3, code)
    want_match = np.zeros((M, 20), int)
    for k, a in ((1, 0), (2, 1), (3, 4), (6, 7), (7, 8)):
        want_match[k - 1, a] += 1
    want_insert = np.zeros((M - 1, 20), int)
    want_insert[1, 2] += 1
    want_insert[1, 3] += 1
    want_trans = np.zeros((M - 1, 7), int)
    want_trans[0, MM] = 1                         # M1 -> M2
    want_trans[1, MI] = 1                         # M2 -> I2
    want_trans[1, II] = 1                         # I2 -> I2
    want_trans[1, IM] = 1                         # I2 -> M3
    want_trans[2, MD] = 1                         # M3 -> D4
    want_trans[3, DD] = 1                         # D4 -> D5
    want_trans[4, DM] = 1                         # D5 -> M6
    want_trans[5, MM] = 1                         # M6 -> M7
    assert np.array_equal(c["match"], want_match)
    assert np.array_equal(c["insert"], want_insert)
    assert np.array_equal(c["trans"], want_trans)


def test_counts_conserve_residues_and_path_steps():
    prof = gen.make_profile(60, 3)
    op = oracle.OracleProfile(prof)
    rng = np.random.default_rng(2)
    h = gen.sample_homologs(rng, prof, 1)[0]
    x = np.concatenate([gen.background_residues(rng, 40), h, gen.background_residues(rng, 30)])
    dec, doms = oracle.domains(op, x)
    assert doms
    for d in doms:
        c = oracle.count_alignment(prof.M, x, d["s"], d["code"])
        aligned = int(np.count_nonzero(d["code"]))
        assert c["match"].sum() + c["insert"].sum() == aligned
        # transitions leaving M states = match residues except the last one of the path
        t = c["trans"]
        assert t[:, MM].sum() + t[:, MI].sum() + t[:, MD].sum() == c["match"].sum() - 1
        assert t[:, IM].sum() + t[:, II].sum() == c["insert"].sum()
        # every delete run entered is left: MD + DD = DD + DM summed over nodes
        assert t[:, MD].sum() == t[:, DM].sum()


def test_rebuild_is_a_profile_and_weights_its_prior():
    prof = random_profile(30, 5)
    rng = np.random.default_rng(1)
    counts = dict(match=rng.integers(0, 9, (30, 20)), insert=rng.integers(0, 3, (29, 20)),
                  trans=rng.integers(0, 40, (29, 7)))
    new = oracle.rebuild_profile(prof, counts, 20.0, 10.0)
    np.testing.assert_allclose(new.match.sum(1), 1.0, atol=1e-14)
    np.testing.assert_allclose(new.insert.sum(1), 1.0, atol=1e-14)
    for g in ((0, 3), (3, 5), (5, 7)):
        np.testing.assert_allclose(new.trans[:, g[0]:g[1]].sum(1), 1.0, atol=1e-14)
    # no counts: the prior comes back unchanged; counts proportional to the
    # prior: a fixed point; huge counts: the empirical frequencies
    zero = {k: np.zeros_like(v) for k, v in counts.items()}
    same = oracle.rebuild_profile(prof, zero, 20.0, 10.0)
    np.testing.assert_allclose(same.match, prof.match, atol=1e-15)
    np.testing.assert_allclose(same.trans, prof.trans, atol=1e-15)
    prop = dict(match=prof.match * 1000.0, insert=prof.insert * 50.0, trans=np.zeros((29, 7)))
    fix = oracle.rebuild_profile(prof, prop, 20.0, 10.0)
    np.testing.assert_allclose(fix.match, prof.match, atol=1e-14)
    big = dict(match=counts["match"] * 10**9 + 1, insert=counts["insert"] * 10**9 + 1, trans=counts["trans"] * 10**9 + 1)
    emp = oracle.rebuild_profile(prof, big, 20.0, 10.0)
    np.testing.assert_allclose(emp.match, big["match"] / big["match"].sum(1, keepdims=True), rtol=0, atol=1e-9)


def test_one_iteration_sharpens_toward_the_homologs():
    """Re-estimated from alignments of homologs sampled from a peaked
    'true' profile, a flat starting profile moves toward the true one."""
    M = 40
    true = gen.make_profile(M, 11)
    flat = gen.make_profile(M, 11)
    flat.match[:] = np.tile(gen.BACKGROUND, (M, 1)) * 0.5 + true.match * 0.5
    op = oracle.OracleProfile(flat)
    rng = np.random.default_rng(3)
    tot = dict(match=np.zeros((M, 20), int), insert=np.zeros((M - 1, 20), int), trans=np.zeros((M - 1, 7), int))
    for h in gen.sample_homologs(rng, true, 60):
        x = np.concatenate([gen.background_residues(rng, 30), h, gen.background_residues(rng, 30)])
        _, doms = oracle.domains(op, x)
        for d in doms:
            c = oracle.count_alignment(M, x, d["s"], d["code"])
            for k in tot:
                tot[k] += c[k]
    new = oracle.rebuild_profile(flat, tot, 20.0, 10.0)
    dist = lambda p: float(np.abs(p.match - true.match).sum())
    assert dist(new) < 0.7 * dist(flat)
