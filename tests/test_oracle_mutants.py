"""Mutation check of the oracle's pins.

Each case plants one plausible mistake into a copy of the oracle source
(on the CPU), builds it, and runs a compact battery of the brute-force and
closed-form pins; every mutant must fail at least one of them.  This shows
that the pins constrain the oracle, not just that the oracle agrees with
itself."""
import math
import os

import numpy as np
import pytest

import brute
from test_oracle_brute import delete_favoring_case, model_sequence
import oracle
from conftest import random_profile
from test_oracle_closed_forms import _exact_odds_profile, _peaked_profile
from test_oracle_decode import _allowed, _zero_transition_profile, forbidden_skip_case

MUTANTS = {
    "im_uses_mm_transition": ("m = imax(m, ADD(Ip[k - 1], t[3]));", "m = imax(m, ADD(Ip[k - 1], t[0]));"),
    "d_chain_from_previous_row": ("Dc[k] = imax(ADD(Mc[k - 1], t[2])", "Dc[k] = imax(ADD(Mp[k - 1], t[2])"),
    "float_drops_d_to_m": ("m = op(m, Dp[k - 1] + t[5]);", "m = m;"),
    "float_e_ignores_d": ("E = op(op(E, Mc[k]), Dc[k]);", "E = op(E, Mc[k]);"),
    "float_j_loop_dropped": ("J = op(J + loop, E + half);", "J = E + half;"),
    "entry_off_by_one": ("p->entry = log(2.0 / ((double)M * ((double)M + 1.0)));",
                         "p->entry = log(2.0 / ((double)M * ((double)M + 2.0)));"),
    "insert_emits_match_score": ("Ic[k] = p->isc[(k - 1) * KA + a] + op(", "Ic[k] = p->msc[(k - 1) * KA + a] + op("),
    "move8_truncates": ("int orc_move8(int L) { return (int)clampl(qround(-ORC_S8 * orc_move(L)), 0, 255); }",
                        "int orc_move8(int L) { return (int)clampl((long)(-ORC_S8 * orc_move(L)), 0, 255); }"),
    "msv_jb_uses_exit": ("int jb = ssub8(xJ, mv);", "int jb = ssub8(xJ, p->exit8);"),
    "vit_ej_sign": ("xJ = imax(xJ, ADD(xE, p->ej16));", "xJ = imax(xJ, ADD(xE, -p->ej16));"),
    "scaled_fwd_forgets_shift": ("shift += ex;", "(void)ex;"),
    "msv_overflow_line_exclusive": ("if (xE >= 255 - p->bias8)", "if (xE > 255 - p->bias8)"),
    "vit16_reports_raw_on_overflow": ("if (!wide && ovf) return 32767;", ""),
    "vit_transposed_mi_ii": ("int v = imax(ADD(Mp[k], t[1]), ADD(Ip[k], t[4]));",
                             "int v = imax(ADD(Mp[k], t[4]), ADD(Ip[k], t[1]));"),
    "msv_cost_wrong_node": ("p->cost8[(k - 1) * KA + a]", "p->cost8[(k > 1 ? k - 2 : 0) * KA + a]"),
    # posterior decoding, regions and alignment
    "bwd_match_drops_exit": ("bMc[k] = lse(lse(bE, t[0] + mn), lse(t[1] + in, t[2] + bDc[k + 1]));",
                             "bMc[k] = lse(t[0] + mn, lse(t[1] + in, t[2] + bDc[k + 1]));"),
    "bwd_insert_scores_match_emission": ("const double in = p->isc[(k - 1) * KA + a] + bIn[k];",
                                         "const double in = p->msc[(k - 1) * KA + a] + bIn[k];"),
    "bwd_delete_chain_skips_dd": ("bDc[k] = lse(bE, lse(t[5] + mn, t[6] + bDc[k + 1]));",
                                  "bDc[k] = lse(bE, t[5] + mn);"),
    "bwd_begin_without_emission": ("nB = lse(nB, p->entry + p->msc[(k - 1) * KA + a] + bMn[k]);",
                                   "nB = lse(nB, p->entry + bMn[k]);"),
    "post_j_emission_without_loop": ("pnjc[3 * (i - 1) + 1] = exp(FJ(i - 1) + loop + bJ - Z);",
                                     "pnjc[3 * (i - 1) + 1] = exp(FJ(i) + bJ - Z);"),
    "oa_flank_earns_core": ("G[r + 1] = G[r] + (1.0 - pcore[s - 1 + r]);", "G[r + 1] = G[r] + pcore[s - 1 + r];"),
    "oa_ignores_zero_dd": ("if (tr[6] > -INFINITY && ODc[k - 1] > u)", "if (ODc[k - 1] > u)"),
    "bias_mean_not_divided": ("p->bias_lr[a] = log(m / (double)M / bg[a]);", "p->bias_lr[a] = log(m / bg[a]);"),
    "bias_switch_swapped": ("const double q = lse(aR + ls, aS + lt) + p->bias_lr[x[i]];",
                            "const double q = lse(aR + lt, aS + ls) + p->bias_lr[x[i]];"),
    # Forward cutoff (P-value of the exponential tail below F3)
    "fwd_cutoff_sign_of_ln_f3": ("*fwd_thr = (calib[2] - log(F[2]) / M_LN2) * M_LN2 + nul;",
                                 "*fwd_thr = (calib[2] + log(F[2]) / M_LN2) * M_LN2 + nul;"),
    "fwd_cutoff_without_null": ("*fwd_thr = (calib[2] - log(F[2]) / M_LN2) * M_LN2 + nul;",
                                "*fwd_thr = (calib[2] - log(F[2]) / M_LN2) * M_LN2;"),
    "fwd_cutoff_in_bits": ("*fwd_thr = (calib[2] - log(F[2]) / M_LN2) * M_LN2 + nul;",
                           "*fwd_thr = (calib[2] - log(F[2]) / M_LN2) + nul;"),
    "regions_strict_rt2": ("if (!(pcore[i] >= rt2)) { i++; continue; }\n    int j = i, hit = 0;\n"
                           "    while (j < L && pcore[j] >= rt2)",
                           "if (!(pcore[i] > rt2)) { i++; continue; }\n    int j = i, hit = 0;\n"
                           "    while (j < L && pcore[j] > rt2)"),
}


def _battery(lib) -> list:
    fails = []

    def check(name, ok):
        if not ok:
            fails.append(name)

    for M, L, seed in [(M, L, s) for M in (1, 2, 3) for L in (1, 2, 3, 4) for s in range(4)]:
        prof = random_profile(M, seed, alpha=0.1, talpha=0.3)
        op = oracle.OracleProfile(prof, lib)
        x = model_sequence(prof, L, 2000 + seed) if seed % 2 else \
            np.random.default_rng(1000 + seed).integers(0, 20, size=L).astype(np.uint8)
        S = brute.float_scores(prof, L)
        check("vit_f64", math.isclose(oracle.vit_f64(op, x), brute.viterbi(S, x), abs_tol=1e-9))
        check("fwd_f64", math.isclose(oracle.fwd_f64(op, x), brute.forward(S, x), abs_tol=1e-9))
        check("fwd_scaled", math.isclose(oracle.fwd_f64_scaled(op, x), brute.forward(S, x), abs_tol=1e-9))
        sc = op.scalars()
        lp = oracle.length_params(L, lib)
        tab = op.tables()
        best = brute.viterbi(brute.int_scores(tab, M, sc["entry16"], lp["move16"], sc["ej16"]), x)
        check("vit32", oracle.vit32(op, x) == best)
        check("vit16", oracle.vit16(op, x) == (best, 0))
        mb = brute.msv_parses(lambda k, a: sc["bias8"] - int(tab["cost8"][k - 1, a]), x, M,
                              oracle.BASE8, lp["move8"], sc["entry8"], sc["exit8"])
        check("msv", oracle.msv(op, x) == (mb, 0))
    for L, mv8, mv16 in ((1, 1, -208), (30, 10, -1730), (300, 20, -3329), (5000, 32, -5352)):
        lp = oracle.length_params(L, lib)
        check("move", lp["move8"] == mv8 and lp["move16"] == mv16)
    from synth import make_profile
    from synth.gen import SEED_CALIB_FWD, random_sequences
    for M, e8, e16 in ((77, 35, -5776), (734, 54, -9021)):
        s = oracle.OracleProfile(make_profile(M, 7), lib).scalars()
        check("entry", s["entry8"] == e8 and s["entry16"] == e16)
    op = oracle.OracleProfile(_exact_odds_profile(40), lib)
    check("msv_ovf_line", oracle.msv(op, np.zeros(34, np.uint8)) == (255, 1))
    prof, c = _peaked_profile(40)
    op = oracle.OracleProfile(prof, lib)
    check("vit16_ovf", oracle.vit16(op, c) == (32767, 1))
    prof, x = delete_favoring_case()
    op = oracle.OracleProfile(prof, lib)
    sc = op.scalars()
    lp = oracle.length_params(2, lib)
    best = brute.viterbi(brute.int_scores(op.tables(), 3, sc["entry16"], lp["move16"], sc["ej16"]), x)
    check("vit_delete_path", oracle.vit32(op, x) == best and oracle.vit16(op, x) == (best, 0))
    # posterior decoding and optimal-accuracy alignment against enumeration
    for M, L, seed, zero in [(2, 3, 0, False), (3, 3, 1, False), (3, 4, 2, False), (3, 4, 0, True),
                             (3, 3, 1, True), (3, 4, 2, True), (2, 4, 3, True)]:
        prof = _zero_transition_profile(M, seed) if zero else random_profile(M, seed, alpha=0.1, talpha=0.3)
        op = oracle.OracleProfile(prof, lib)
        x = model_sequence(prof, L, 3000 + seed) if seed % 2 else \
            np.random.default_rng(1000 + seed).integers(0, 20, size=L).astype(np.uint8)
        d = oracle.decode(op, x)
        bp = brute.posteriors(brute.float_scores(prof, L), x)
        for key in ("core", "njc", "beg", "end", "pM", "pI"):
            check("post_" + key, np.allclose(d[key], np.array(bp[key]), rtol=0, atol=1e-9))
        for s in range(1, L + 1):
            for e in range(s, L + 1):
                want = brute.oa_best(M, _allowed(prof), bp["core"], bp["pM"], bp["pI"], s, e)
                check("oa", math.isclose(oracle.oa_align(op, d, s, e)["score"], want, abs_tol=1e-9))
    prof, x = forbidden_skip_case()
    op = oracle.OracleProfile(prof, lib)
    d = oracle.decode(op, x)
    bp = brute.posteriors(brute.float_scores(prof, 2), x)
    want = brute.oa_best(4, _allowed(prof), bp["core"], bp["pM"], bp["pI"], 1, 2)
    check("oa_forbidden_skip", math.isclose(oracle.oa_align(op, d, 1, 2)["score"], want, abs_tol=1e-9))
    from test_oracle_bias import _brute as bias_brute
    for L, seed in ((1, 0), (4, 1), (7, 2)):
        prof = random_profile(7, seed, alpha=0.3)
        x = np.random.default_rng(seed + 10).integers(0, 20, L).astype(np.uint8)
        check("bias", math.isclose(oracle.bias(oracle.OracleProfile(prof, lib), x), bias_brute(prof, x), abs_tol=1e-9))
    # Forward cutoff: with tau fitted at tail mass 0.04 on 2,000 background
    # sequences, a fresh sample passes F3 = 0.05 at about that rate
    fprof = make_profile(20, 3)
    fop = oracle.OracleProfile(fprof, lib)
    fcal = oracle.calibrate(fop, nthreads=8, n=2000)
    fdb = random_sequences(SEED_CALIB_FWD + 97, 4000, 100)
    fr = oracle.search(fop, fdb.residues, fdb.offsets, fcal, (1.0, 1.0, 0.05), nthreads=8)
    frac = float(np.mean((fr["flags"] & oracle.F_FWD_PASS) != 0))
    check("fwd_cutoff", 0.025 < frac < 0.075)
    # ... and the exponential tail's survival at the cutoff is F3 itself
    for L, tau, F3 in ((100, -3.9, 0.05), (300, -7.2, 1e-3), (30, 2.5, 0.5)):
        thr = oracle.thresholds((0.0, 0.0, tau), (1.0, 1.0, F3), L, lib)[2]
        x = (thr - oracle.length_params(L, lib)["null"]) / math.log(2.0)
        check("fwd_cutoff_survival", math.isclose(math.exp(-math.log(2.0) * (x - tau)), F3, rel_tol=1e-9))
    core = np.array([0.05, 0.10, 0.2, 0.25, 0.099, 0.3, 0.24, 0.11, 0.09, 0.12, 0.2, 0.1, 0.5, 0.1])
    check("regions", oracle.regions(core, 0.25, 0.10, lib) == [(2, 4), (6, 8), (10, 14)])
    return fails


def test_unmodified_oracle_passes_the_battery():
    assert _battery(oracle.lib()) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_every_planted_mistake_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = oracle.source_text()
    assert src.count(old) >= 1, f"mutation anchor not found: {old}"
    path = oracle.build_variant(src.replace(old, new), os.path.join(str(tmp_path), f"mut_{name}.so"))
    fails = _battery(oracle.load(path))
    assert fails, f"mutant {name} passed every pin"
