"""Statistical pin of the score statistics: with the oracle's own
calibration, the fraction of i.i.d. background sequences that pass each
filter is close to the requested P-value cutoff."""
import numpy as np
import pytest

import oracle
from synth import gen


@pytest.mark.parametrize("M", [77, 256])
def test_background_pass_fractions_match_pvalue_cutoffs(M):
    prof = gen.make_profile(M, 21)
    op = oracle.OracleProfile(prof)
    calib = oracle.calibrate(op, nthreads=8)
    db = gen.make_database(20000, 22, None, 0.0)
    r = oracle.search(op, db.residues, db.offsets, calib, (0.02, 1e-3, 1.0), nthreads=8)
    msv = np.mean((r["flags"] & oracle.F_MSV_PASS) != 0)
    vit = np.mean((r["flags"] & oracle.F_VIT_PASS) != 0)
    # binomial sd at n = 20000 is 0.001 (MSV); the 200-sequence calibration
    # adds ~10 % relative error on the P-value scale.
    assert 0.012 < msv < 0.03
    assert 0.0002 < vit < 0.003
