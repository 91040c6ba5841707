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
