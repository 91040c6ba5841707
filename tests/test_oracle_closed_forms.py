"""Closed-form pins of the CPU oracle: cases small or structured enough that
the score is written out by hand from the model definition."""
import math

import numpy as np
import pytest

import oracle
from synth import Profile

S8 = 3.0 / math.log(2.0)
S16 = 500.0 / math.log(2.0)


def _exact_odds_profile(M):
    """Uniform background; at every node residues 0-3 have odds 2, residues
    4-11 odds 1/2 and residues 12-19 odds 1 (probabilities sum to 1), so
    every emission score is exactly +-ln 2 or 0: +-3 / 0 in MSV units and
    +-500 / 0 in Viterbi units."""
    bg = np.full(20, 1.0 / 20)
    row = np.concatenate([np.full(4, 2.0 / 20), np.full(8, 0.5 / 20), np.full(8, 1.0 / 20)])
    match = np.tile(row, (M, 1))
    insert = np.tile(bg, (max(M - 1, 0), 1))
    trans = np.tile([0.5, 0.25, 0.25, 0.5, 0.5, 0.5, 0.5], (max(M - 1, 0), 1))
    return Profile(M, bg, match, insert, trans)


def test_quantised_emission_scores_are_exact_for_power_of_two_odds():
    op = oracle.OracleProfile(_exact_odds_profile(3))
    t = op.tables()
    sc = op.scalars()
    assert sc["bias8"] == 3                      # -min sc8 = -(-3)
    assert list(t["cost8"][0, :4]) == [0] * 4     # 3 - 3
    assert list(t["cost8"][0, 4:12]) == [6] * 8   # 3 + 3
    assert list(t["cost8"][0, 12:]) == [3] * 8
    assert list(t["msc16"][1, :4]) == [500] * 4
    assert list(t["msc16"][1, 4:12]) == [-500] * 8
    assert list(t["msc16"][1, 12:]) == [0] * 8
    assert np.all(t["isc16"] == 0)
    # transitions 1/2 and 1/4 are exactly -500 and -1000
    assert list(t["t16"][0]) == [-500, -1000, -1000, -500, -500, -500, -500]
    assert sc["exit8"] == 3 and sc["ej16"] == -500


@pytest.mark.parametrize("M,entry8,entry16", [(77, 35, -5776), (256, 45, -7503),
                                              (734, 54, -9021), (2500, 65, -10788)])
def test_entry_costs_at_workload_sizes(M, entry8, entry16):
    # ENTRY = ln(2/(M(M+1))); e.g. M = 77: ln(2/6006) = -8.0073 nats,
    # x 3/ln2 = -34.66 -> 35;  x 500/ln2 = -5776.0 -> -5776.
    from synth import make_profile
    op = oracle.OracleProfile(make_profile(M, 7))
    sc = op.scalars()
    assert sc["entry8"] == entry8
    assert sc["entry16"] == entry16


@pytest.mark.parametrize("L,move8,move16", [(1, 1, -208), (30, 10, -1730), (300, 20, -3329),
                                            (1000, 25, -4193), (5000, 32, -5352)])
def test_length_model_costs(L, move8, move16):
    # MOVE = ln(3/(L+3)); L = 1: ln 0.75 = -0.28768 -> 1.245 -> 1 and -207.5 -> -208.
    lp = oracle.length_params(L)
    assert lp["move8"] == move8
    assert lp["move16"] == move16
    assert lp["null"] == pytest.approx(L * math.log(L / (L + 1)) - math.log(L + 1), abs=1e-12)


def test_single_node_single_residue_all_scores():
    # M = 1, L = 1: one path S->N->B->M1->E->C->T.
    prof = _exact_odds_profile(1)
    op = oracle.OracleProfile(prof)
    for a, lo in ((0, math.log(2)), (5, -math.log(2)), (15, 0.0)):
        x = np.array([a], np.uint8)
        expect = 2 * math.log(0.75) + 0.0 + lo + math.log(0.5)
        assert oracle.vit_f64(op, x) == pytest.approx(expect, abs=1e-12)
        assert oracle.fwd_f64(op, x) == pytest.approx(expect, abs=1e-12)
        # MSV: xB = 190 - MOVE8(1) = 189, ENTRY8 = 0, + sc8, - EXIT8 3, - MOVE8 1
        sc8 = {0: 3, 5: -3, 15: 0}[a]
        assert oracle.msv(op, x) == (189 + sc8 - 3 - 1, 0)
        # Viterbi: MOVE16 + ENTRY16(=0) + msc16 + EJ16 + MOVE16
        sc16 = {0: 500, 5: -500, 15: 0}[a]
        assert oracle.vit16(op, x) == (-208 + sc16 - 500 - 208, 0)
        assert oracle.vit32(op, x) == -208 + sc16 - 500 - 208


def test_single_node_two_residues_three_paths():
    prof = _exact_odds_profile(1)
    op = oracle.OracleProfile(prof)
    LOOP, MOVE, H = math.log(2 / 5), math.log(3 / 5), math.log(0.5)
    for x1, x2 in ((0, 5), (5, 0), (0, 0), (12, 4)):
        m1 = math.log(prof.match[0, x1] / prof.bg[x1])
        m2 = math.log(prof.match[0, x2] / prof.bg[x2])
        p1 = LOOP + MOVE + m2 + H + MOVE                    # N emits x1
        p2 = MOVE + m1 + H + LOOP + MOVE                    # C emits x2
        p3 = MOVE + m1 + H + MOVE + m2 + H + MOVE           # two hits via J
        x = np.array([x1, x2], np.uint8)
        assert oracle.vit_f64(op, x) == pytest.approx(max(p1, p2, p3), abs=1e-12)
        lse = max(p1, p2, p3) + math.log(sum(math.exp(p - max(p1, p2, p3)) for p in (p1, p2, p3)))
        assert oracle.fwd_f64(op, x) == pytest.approx(lse, abs=1e-12)


def _peaked_profile(M, p_top=0.81, seed=0):
    """Uniform background; node k emits residue c_k with probability p_top
    and every other residue with (1-p_top)/19.  Returns (profile, c)."""
    rng = np.random.default_rng(seed)
    c = rng.integers(0, 19, size=M)          # residue 19 is never the consensus
    bg = np.full(20, 0.05)
    match = np.full((M, 20), (1 - p_top) / 19)
    match[np.arange(M), c] = p_top
    insert = np.tile(bg, (M - 1, 1))
    trans = np.tile([0.9, 0.05, 0.05, 0.6, 0.4, 0.5, 0.5], (M - 1, 1))
    return Profile(M, bg, match, insert, trans), c.astype(np.uint8)


def test_consensus_target_overflows_and_rescore_is_the_diagonal_path():
    # The consensus sequence of a strongly peaked profile is best explained
    # by the single full-length diagonal path, whose integer score is
    #   MOVE16 + ENTRY16 + sum_k msc16_k(c_k) + sum_{k<M} MM16_k + EJ16 + MOVE16.
    M = 40
    prof, c = _peaked_profile(M)
    op = oracle.OracleProfile(prof)
    t = op.tables()
    sc = op.scalars()
    mv = oracle.length_params(M)["move16"]
    diag = mv + sc["entry16"] + int(t["msc16"][np.arange(M), c].astype(np.int64).sum()) \
        + int(t["t16"][:, 0].astype(np.int64).sum()) + sc["ej16"] + mv
    assert diag > 32767
    raw16, ovf = oracle.vit16(op, c)
    assert (raw16, ovf) == (32767, 1)
    assert oracle.vit32(op, c) == diag
    # MSV saturates too and reports 255
    assert oracle.msv(op, c) == (255, 1)
    # float Viterbi of the same path (loops included: no N/C/J residues)
    Lf = M
    move = math.log(3 / (Lf + 3))
    path = 2 * move + math.log(2 / (M * (M + 1))) + math.log(0.5) \
        + sum(math.log(prof.match[k, c[k]] / 0.05) for k in range(M)) + (M - 1) * math.log(0.9)
    assert oracle.vit_f64(op, c) == pytest.approx(path, abs=1e-9)


def test_msv_positive_score_cap_at_bias():
    # Peaked profile: the consensus score (q(S8 ln 16.2) = 12) exceeds BIAS8
    # (= -q(S8 ln 0.2) = 7), so its cost clamps to 0 and each consensus cell
    # gains exactly BIAS8.  With L = M = 40: MOVE8 = 12, ENTRY8 = 29,
    # so the diagonal starts at 190-12-29+7 = 156 and grows by 7 per row;
    # it reaches the overflow line 255-7 = 248 at row 15.
    M = 40
    prof, c = _peaked_profile(M)
    op = oracle.OracleProfile(prof)
    sc = op.scalars()
    assert sc["bias8"] == 7 and sc["entry8"] == 29
    assert oracle.length_params(40)["move8"] == 12
    assert np.all(op.tables()["cost8"][np.arange(M), c] == 0)
    # 14 consensus residues, then 26 copies of residue 19 (cost 7+7 = 14 at
    # every node, so no later cell gets near the diagonal's value): the
    # row-14 cell is 156 + 13*7 = 247 < 248, no overflow; xJ = 247-3 = 244,
    # msv_raw = 244 - 12 = 232.
    x = np.concatenate([c[:14], np.full(26, 19, np.uint8)])
    raw, ovf = oracle.msv(op, x)
    assert ovf == 0
    assert raw == 232


def test_degenerate_bias_overflows_every_target():
    # A near-zero emission probability puts -min sc8 above 255: BIAS8 clamps
    # to 255, the overflow line 255 - BIAS8 is 0, and every target reports
    # msv_raw = 255 with the overflow flag.
    bg = np.full(20, 0.05)
    match = np.full((3, 20), 1.0 / 20)
    match[1, 0] = 1e-300
    match[1, 1] += 1.0 / 20 - 1e-300
    prof = Profile(3, bg, match, np.tile(bg, (2, 1)), np.tile([0.9, 0.05, 0.05, 0.6, 0.4, 0.5, 0.5], (2, 1)))
    op = oracle.OracleProfile(prof)
    assert op.scalars()["bias8"] == 255
    assert oracle.msv(op, np.array([3, 4, 5], np.uint8)) == (255, 1)


@pytest.mark.parametrize("L,expect", [(33, (249 - 3 - 11, 0)), (34, (255, 1))])
def test_msv_overflow_line_is_inclusive(L, expect):
    # Exact-odds profile, M = 40 (ENTRY8 = 29), target of residue 0 only
    # (score +3 at every node, BIAS8 = 3, overflow line 255-3 = 252); for
    # L = 33 and 34, MOVE8 = 11.  The best cell after n rows is the
    # diagonal 190 - 11 - 29 + 3n: 249 at n = 33 (no overflow; xJ = 246,
    # msv_raw = 246 - 11 = 235) and exactly 252 at n = 34 (overflow).
    op = oracle.OracleProfile(_exact_odds_profile(40))
    assert op.scalars()["entry8"] == 29 and oracle.length_params(L)["move8"] == 11
    assert oracle.msv(op, np.zeros(L, np.uint8)) == expect
