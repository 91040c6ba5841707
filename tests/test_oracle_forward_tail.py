"""Pins of the Forward stage's statistics: the cutoff FWD_PASS and the
calibrated tail location tau.

Reading (stated in the oracle): Forward bit scores of unrelated sequences
have an exponential upper tail P(S > x) = exp(-lambda (x - tau)) with
lambda = ln 2 per bit; a target passes when that P-value is below F3, i.e.
when its bit score exceeds tau - ln(F3) / lambda; tau is fitted by putting
the tail mass 0.04 at the (0.04 n)-th largest score of n background
sequences of length 100.

What pins them here, besides the definition itself:
  * the survival function at the oracle's cutoff equals F3, and the
    search's decision at the cutoff is strict;
  * the slope of the empirical tail of background Forward bit scores is
    near ln 2 (a scale or units mistake moves it by a factor 1.44 or more);
  * with tau fitted on one background sample, the fraction of a fresh
    sample passing F3 is F3 within the sampling error of both samples
    (F3 near the fitted tail mass), or the fraction the measured slope
    predicts (F3 well below it, where the ln 2 reading and the measured
    slope part ways);
  * planted mistakes in the cutoff and in the fit fail these checks.

Tolerance of the pass fractions: the test sample's count is binomial
(relative sd 1/sqrt(F3 n_test)); the fitted tau carries the sampling error
of the fit's order statistic (relative sd of the tail mass about
1/sqrt(0.04 n_cal)); both at 3.29 sd (99.9 %).
"""
import math

import numpy as np
import pytest

import oracle
from synth import gen

LN2 = math.log(2.0)
M_STAT = 77            # C1's profile size: long enough for a clean tail
N_CAL = 20000          # calibration sample (800 scores above the fitted tail)
N_TEST = 30000         # fresh background sample, length 100
Z999 = 3.29


@pytest.fixture(scope="module")
def tail_case():
    prof = gen.make_profile(M_STAT, 21)
    op = oracle.OracleProfile(prof)
    calib = oracle.calibrate(op, nthreads=8, n=N_CAL)
    db = gen.random_sequences(gen.SEED_CALIB_FWD + 99, N_TEST, 100)
    runs = {}
    for F3 in (0.05, 0.01):
        runs[F3] = oracle.search(op, db.residues, db.offsets, calib, (1.0, 1.0, F3), nthreads=8)
    return op, calib, db, runs


def pass_fraction(r) -> float:
    return float(np.mean((r["flags"] & oracle.F_FWD_PASS) != 0))


def fraction_band(F3: float, n_test: int, n_cal: int, extra: float = 0.0) -> tuple[float, float]:
    rel = math.sqrt(1.0 / (F3 * n_test) + 1.0 / (oracle.FWD_TAIL * n_cal))
    half = Z999 * rel + extra
    return F3 * (1.0 - half), F3 * (1.0 + half)


# ------------------------------------------------------------ definition

@pytest.mark.parametrize("L", [1, 30, 100, 300, 5000])
def test_forward_cutoff_is_the_exponential_tail_quantile(L):
    for tau in (-7.2, -3.9, 2.5):
        for F3 in (0.5, 0.05, 0.01, 1e-3):
            _, _, thr = oracle.thresholds((0.0, 0.0, tau), (1.0, 1.0, F3), L)
            x = oracle.fwd_bits(thr, L)          # cutoff in bits
            # survival of the exponential tail at the cutoff is F3
            assert math.exp(-LN2 * (x - tau)) == pytest.approx(F3, rel=1e-12)
            # scores just above the cutoff have P-values below F3, just below above it
            eps = 1e-9 * (1.0 + abs(thr))
            assert math.exp(-LN2 * (oracle.fwd_bits(thr + eps, L) - tau)) < F3
            assert math.exp(-LN2 * (oracle.fwd_bits(thr - eps, L) - tau)) > F3
    _, _, thr = oracle.thresholds((0.0, 0.0, -3.0), (1.0, 1.0, 1.0), L)
    assert thr == -math.inf


def test_forward_pass_is_strict_at_the_cutoff(tail_case):
    """FWD_PASS holds exactly for the targets whose Forward score lies
    above the cutoff: tau is set so that one target's score is the cutoff
    itself (to the last bit where fp64 allows), which must then fail."""
    op, calib, db, _ = tail_case
    x = db.seq(0)
    f = oracle.fwd_f64(op, x)
    F3 = 0.05
    # tau placing the cutoff at f: (tau - ln F3 / ln 2) ln 2 + NULL = f
    tau = (f - oracle.length_params(x.size)["null"]) / LN2 + math.log(F3) / LN2
    thr = oracle.thresholds((0.0, 0.0, tau), (1.0, 1.0, F3), x.size)[2]
    off = np.array([0, x.size], np.int64)
    r = oracle.search(op, x, off, (0.0, 0.0, tau), (1.0, 1.0, F3), nthreads=1)
    assert bool(r["flags"][0] & oracle.F_FWD_PASS) == (r["fwd"][0] > thr)
    assert abs(thr - f) <= 4 * math.ulp(f)
    # moved a few ulps either way, the decision follows the side
    for shift, want in ((-1e-9, True), (1e-9, False)):
        r = oracle.search(op, x, off, (0.0, 0.0, tau + shift), (1.0, 1.0, F3), nthreads=1)
        assert bool(r["flags"][0] & oracle.F_FWD_PASS) == want


# ------------------------------------------------------------ statistics

def test_forward_tail_slope_is_near_ln2_per_bit(tail_case):
    """Maximum-likelihood slope of the exponential tail above the 0.04
    quantile of background Forward bit scores (1,200 exceedances, relative
    sd about 3 %): within 25 % of ln 2.  The synthetic profiles measure
    0.70-0.80 per bit; scores in nats, or bits computed twice, would give
    about 1.0-1.1 or 0.48."""
    _, _, _, runs = tail_case
    r = runs[0.05]
    bits = (r["fwd"] - oracle.length_params(100)["null"]) / LN2
    b = np.sort(bits)[::-1]
    k = int(round(oracle.FWD_TAIL * b.size))
    lam = 1.0 / float(np.mean(b[:k] - b[k - 1]))
    assert 0.75 * LN2 < lam < 1.25 * LN2, lam


def test_forward_pass_fraction_near_the_fitted_tail_is_F3(tail_case):
    """At F3 = 0.05, a quarter of a bit from the fitted tail mass 0.04, the
    slope reading changes the expected fraction by at most 3 % (slopes up
    to 1.2 ln 2): allowed on top of the two sampling errors."""
    _, _, _, runs = tail_case
    p = pass_fraction(runs[0.05])
    lo, hi = fraction_band(0.05, N_TEST, N_CAL, extra=0.03)
    assert lo < p < hi, (p, lo, hi)


def test_forward_pass_fraction_far_in_the_tail_follows_the_slope(tail_case):
    """At F3 = 0.01, two bits beyond the fitted tail mass, the pass fraction
    is the one the tail's measured slope predicts from the fitted point:
    0.04 (F3 / 0.04)^(lambda_hat / ln 2) (= F3 at lambda_hat = ln 2), with
    the slope's own sampling error added."""
    _, _, _, runs = tail_case
    bits = (runs[0.05]["fwd"] - oracle.length_params(100)["null"]) / LN2
    b = np.sort(bits)[::-1]
    k = int(round(oracle.FWD_TAIL * b.size))
    lam = 1.0 / float(np.mean(b[:k] - b[k - 1]))
    F3 = 0.01
    pred = oracle.FWD_TAIL * (F3 / oracle.FWD_TAIL) ** (lam / LN2)
    slope_rel = abs(math.log(F3 / oracle.FWD_TAIL)) * (lam / LN2) / math.sqrt(k)
    lo, hi = fraction_band(pred, N_TEST, N_CAL, extra=Z999 * slope_rel)
    p = pass_fraction(runs[F3])
    assert lo < p < hi, (p, pred, lo, hi, lam)


# ------------------------------------------------------------ planted mistakes

def _fraction_check(op, calib, db, F3=0.05) -> bool:
    r = oracle.search(op, db.residues, db.offsets, calib, (1.0, 1.0, F3), nthreads=8)
    lo, hi = fraction_band(F3, db.n, 2000, extra=0.03)
    return lo < pass_fraction(r) < hi


@pytest.mark.parametrize("mistake", ["tail_sign", "log_dropped", "lambda_per_nat"])
def test_planted_calibration_mistakes_are_caught(mistake, monkeypatch):
    """A wrong tau fit is planted in the oracle on the CPU (the sign of
    ln(tail), ln(tail) replaced by tail, the slope taken per nat); the
    pass-fraction check must fail for each and hold for the unmodified
    fit.  (Mistakes in the cutoff formula itself are planted in the C
    source by the mutation battery.)"""
    prof = gen.make_profile(M_STAT, 21)
    op = oracle.OracleProfile(prof)
    db = gen.random_sequences(gen.SEED_CALIB_FWD + 98, 8000, 100)
    good = oracle.calibrate(op, nthreads=8, n=2000)
    fit = oracle.exp_tail_location

    def wrong(bits, tail=oracle.FWD_TAIL, lam=LN2):
        if mistake == "tail_sign":
            return fit(bits, tail, lam) - 2.0 * math.log(tail) / lam
        if mistake == "log_dropped":
            return fit(bits, tail, lam) - math.log(tail) / lam + tail / lam
        return fit(bits, tail, 1.0)

    monkeypatch.setattr(oracle, "exp_tail_location", wrong)
    bad = oracle.calibrate(op, nthreads=8, n=2000)
    monkeypatch.undo()
    assert _fraction_check(op, good, db)
    assert not _fraction_check(op, bad, db), (mistake, good, bad)
