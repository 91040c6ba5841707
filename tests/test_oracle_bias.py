"""Pins of the oracle's composition-bias filter: the bias score against
enumeration of every state path of its two-state null model, its closed
form at L = 1, its value when the profile's composition is the
background's, and the filter rule inside the search."""
import itertools
import math

import numpy as np
import pytest

import oracle
from conftest import random_profile
from synth import gen

W = oracle.BIAS_SWITCH


def _odds(prof):
    m = prof.match.mean(axis=0)
    return m / prof.bg


def _brute(prof, x):
    r = _odds(prof)
    tot = 0.0
    for path in itertools.product((0, 1), repeat=len(x)):
        p = (1 - W) if path[0] == 0 else W
        for i in range(1, len(x)):
            p *= (1 - W) if path[i] == path[i - 1] else W
        for s, a in zip(path, x):
            p *= 1.0 if s == 0 else r[a]
        tot += p
    return math.log(tot)


@pytest.mark.parametrize("L,seed", [(L, s) for L in (1, 2, 3, 5, 8, 10) for s in range(3)])
def test_bias_equals_enumeration_of_state_paths(L, seed):
    prof = random_profile(7, seed, alpha=0.3)
    op = oracle.OracleProfile(prof)
    x = np.random.default_rng(seed + 10).integers(0, 20, L).astype(np.uint8)
    assert oracle.bias(op, x) == pytest.approx(_brute(prof, x), abs=1e-12)


def test_bias_closed_form_and_background_composition():
    prof = random_profile(5, 4)
    op = oracle.OracleProfile(prof)
    r = _odds(prof)
    for a in range(20):
        assert oracle.bias(op, np.array([a], np.uint8)) == pytest.approx(math.log((1 - W) + W * r[a]), abs=1e-14)
    # a profile whose mean match composition is the background: no bias at all
    flat = gen.make_profile(6, 1)
    flat.match[:] = np.tile(flat.bg, (6, 1))
    opf = oracle.OracleProfile(flat)
    x = np.random.default_rng(0).integers(0, 20, 500).astype(np.uint8)
    assert abs(oracle.bias(opf, x)) < 1e-12


def test_low_complexity_target_gets_a_large_bias():
    prof = gen.make_profile(120, 5)
    op = oracle.OracleProfile(prof)
    a = int(np.argmax(_odds(prof)))
    run = np.full(200, a, np.uint8)
    bg = gen.background_residues(np.random.default_rng(1), 200)
    assert oracle.bias(op, run) > 20.0
    assert oracle.bias(op, bg) < 3.0


def test_filter_rule_inside_the_search():
    prof = gen.make_profile(80, 6)
    op = oracle.OracleProfile(prof)
    db = gen.make_database(300, 9, prof, 0.1)
    # low-complexity targets that the raw MSV lets through
    a = int(np.argmax(_odds(prof)))
    seqs = [db.seq(i) for i in range(db.n)] + [np.full(L, a, np.uint8) for L in (40, 150, 400)]
    off = np.zeros(len(seqs) + 1, np.int64)
    off[1:] = np.cumsum([s.size for s in seqs])
    res = np.concatenate(seqs)
    calib = oracle.calibrate(op, nthreads=4)
    F = (0.2, 0.05, 1.0)
    plain = oracle.search(op, res, off, calib, F, nthreads=4)
    bf = oracle.search(op, res, off, calib, F, nthreads=4, bias_filter=True)
    assert np.array_equal(plain["msv"], bf["msv"])
    assert np.all((plain["flags"] & oracle.F_BIAS_PASS) == 0)
    dropped = 0
    for t in range(len(seqs)):
        x = res[off[t]:off[t + 1]]
        msv_pass = (plain["flags"][t] & oracle.F_MSV_PASS) != 0
        assert ((bf["flags"][t] & oracle.F_MSV_PASS) != 0) == msv_pass
        if not msv_pass:
            assert np.isnan(bf["beta"][t]) and bf["flags"][t] == plain["flags"][t]
            continue
        b = oracle.bias(op, x)
        assert bf["beta"][t] == pytest.approx(b, abs=1e-12)
        thr8, _, _ = oracle.thresholds(calib, F, x.size)
        ovf = (plain["flags"][t] & oracle.F_MSV_OVF) != 0
        keep = ovf or int(plain["msv"][t]) - oracle.S8 * max(b, 0.0) >= thr8
        assert ((bf["flags"][t] & oracle.F_BIAS_PASS) != 0) == keep
        assert ((bf["flags"][t] & oracle.F_VIT_RAN) != 0) == keep
        if keep:
            assert bf["vit"][t] == plain["vit"][t]
        else:
            dropped += 1
    assert dropped >= 3          # at least the low-complexity targets
