"""Pins of the CPU oracle against brute-force path enumeration.

Every Plan7 path is enumerated for tiny profiles (M <= 3) and sequences
(L <= 4) with random emissions and random per-node transitions; Viterbi
must equal the best path score and Forward the log-sum over all paths.
The integer filters are pinned the same way on their own integer score
systems.  A dropped term, wrong index, swapped transition or wrong sign in
the oracle changes at least one of these values.
"""
import itertools

import numpy as np
import pytest

import brute
import oracle
from conftest import random_profile

# (M, L, seed, alpha): alpha = 1 gives diffuse random profiles, alpha = 0.1
# peaked emissions and transitions, under which insert runs, delete runs
# and multi-hit paths win often enough to be exercised.
CASES = [(M, L, seed, alpha) for M in (1, 2, 3) for L in (1, 2, 3, 4) for seed in range(6)
         for alpha in (1.0, 0.1)] + [(3, 5, seed, 0.1) for seed in range(4)]


def _prof(M, seed, alpha):
    return random_profile(M, seed, alpha=alpha, talpha=alpha * 3)


def model_sequence(prof, L, seed):
    """Length-L sequence made of homologs sampled from the profile itself
    (so consensus runs, insert runs and second hits occur), cut to L."""
    from synth import sample_homologs
    rng = np.random.default_rng(seed)
    parts = []
    while sum(p.size for p in parts) < L:
        parts.append(sample_homologs(rng, prof, 1)[0])
    return np.concatenate(parts)[:L].astype(np.uint8)


def _seq(L, seed, prof=None, alpha=1.0):
    if alpha < 1.0 and seed % 2 == 1:
        return model_sequence(prof, L, 2000 + seed)
    return np.random.default_rng(1000 + seed).integers(0, 20, size=L).astype(np.uint8)


@pytest.mark.parametrize("M,L,seed,alpha", CASES)
def test_float_viterbi_forward_equal_brute_force(M, L, seed, alpha):
    prof = _prof(M, seed, alpha)
    op = oracle.OracleProfile(prof)
    x = _seq(L, seed, prof, alpha)
    S = brute.float_scores(prof, L)
    assert oracle.vit_f64(op, x) == pytest.approx(brute.viterbi(S, x), abs=1e-10)
    assert oracle.fwd_f64(op, x) == pytest.approx(brute.forward(S, x), abs=1e-10)
    assert oracle.fwd_f64_scaled(op, x) == pytest.approx(brute.forward(S, x), abs=1e-10)


@pytest.mark.parametrize("M,L,seed,alpha", CASES)
def test_integer_viterbi_equals_brute_force(M, L, seed, alpha):
    prof = _prof(M, seed, alpha)
    op = oracle.OracleProfile(prof)
    x = _seq(L, seed, prof, alpha)
    sc = op.scalars()
    lp = oracle.length_params(L)
    S = brute.int_scores(op.tables(), M, sc["entry16"], lp["move16"], sc["ej16"])
    best = brute.viterbi(S, x)
    assert oracle.vit32(op, x) == best
    raw16, ovf = oracle.vit16(op, x)
    assert ovf == 0
    assert raw16 == best


@pytest.mark.parametrize("M,L,seed,alpha", CASES)
def test_msv_equals_best_segment_parse(M, L, seed, alpha):
    prof = _prof(M, seed, alpha)
    op = oracle.OracleProfile(prof)
    x = _seq(L, seed, prof, alpha)
    sc = op.scalars()
    cost8 = op.tables()["cost8"]
    lp = oracle.length_params(L)
    best = brute.msv_parses(lambda k, a: sc["bias8"] - int(cost8[k - 1, a]), x, M,
                            oracle.BASE8, lp["move8"], sc["entry8"], sc["exit8"])
    raw, ovf = oracle.msv(op, x)
    assert ovf == 0
    assert raw == best


def delete_favoring_case():
    """M = 3 profile whose best path for x = (c1, c3) is M1 -> D2 -> M3:
    peaked emissions (c_k at 0.9), M1->D2 = 0.8 and D2->M3 = 0.9 are much
    cheaper than ending the hit and re-entering through J."""
    from synth import BACKGROUND, Profile
    c = [18, 4, 1]                      # W, F, C
    match = np.full((3, 20), 0.1 / 19)
    for k in range(3):
        match[k, c[k]] = 0.9
    insert = np.tile(BACKGROUND, (2, 1))
    tr = np.array([[0.1, 0.1, 0.8, 0.5, 0.5, 0.5, 0.5],
                   [0.8, 0.1, 0.1, 0.5, 0.5, 0.9, 0.1]])
    return Profile(3, BACKGROUND.copy(), match, insert, tr), np.array([c[0], c[2]], np.uint8)


def test_delete_path_case_integer_and_float():
    prof, x = delete_favoring_case()
    op = oracle.OracleProfile(prof)
    S = brute.float_scores(prof, x.size)
    assert oracle.vit_f64(op, x) == pytest.approx(brute.viterbi(S, x), abs=1e-10)
    assert oracle.fwd_f64(op, x) == pytest.approx(brute.forward(S, x), abs=1e-10)
    sc = op.scalars()
    lp = oracle.length_params(x.size)
    t = op.tables()
    best = brute.viterbi(brute.int_scores(t, 3, sc["entry16"], lp["move16"], sc["ej16"]), x)
    # the best integer path is M1 -> D2 -> M3 (written out)
    path = lp["move16"] + sc["entry16"] + int(t["msc16"][0, x[0]]) + int(t["t16"][0, 2]) \
        + int(t["t16"][1, 5]) + int(t["msc16"][2, x[1]]) + sc["ej16"] + lp["move16"]
    assert best == path
    assert oracle.vit32(op, x) == best
    assert oracle.vit16(op, x) == (best, 0)


def test_brute_force_path_count_m1_l2():
    # M = 1, L = 2 has exactly three paths (N-emit then M; M then C-emit;
    # M, J, M); the enumerator must find exactly those.
    prof = random_profile(1, 0)
    S = brute.float_scores(prof, 2)
    assert len(brute.all_path_scores(S, np.array([3, 7], np.uint8))) == 3


def test_brute_force_counts_grow_with_insert_and_delete_states():
    # M = 2, L = 2, counted by hand.  One hit covering one residue (the other
    # emitted by N or C): 2 residue choices x 3 core walks (M1->E,
    # M1->D2->E, M2->E) = 6.  One hit covering both residues: only M1->M2->E
    # (I_1 would need a third residue to reach M_2) = 1.  Two hits joined by
    # J: 3 x 3 core walks = 9.
    prof = random_profile(2, 1)
    S = brute.float_scores(prof, 2)
    n = len(brute.all_path_scores(S, np.array([0, 1], np.uint8)))
    assert n == 6 + 1 + 9
