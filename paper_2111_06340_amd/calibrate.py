"""Score calibration of a profile with the GPU search itself.

The P-value cutoffs of the filters need the location of each score
distribution on random sequences (slope fixed at ln 2 per bit): the MSV and
Viterbi scores of n i.i.d. background sequences of length 200 give the
Gumbel locations by maximum likelihood, and the Forward scores of n
sequences of length 100 give the exponential-tail location that puts a
tail mass of 0.04 at the (0.04 n)-th largest score.  The random sequences
come from the seeded generator; the scores from hmm_search.
"""
from __future__ import annotations

import math

import numpy as np

from . import Database, Profile, alloc_results, search

LN2 = math.log(2.0)
S8 = 3.0 / LN2
S16 = 500.0 / LN2
BASE8 = 190
TAIL = 0.04


def null_score(L: int) -> float:
    return L * math.log(L / (L + 1.0)) + math.log(1.0 / (L + 1.0))


def _gumbel_location(bits: np.ndarray) -> float:
    return float(-math.log(np.mean(np.exp(-LN2 * bits))) / LN2)


def calibrate(prof, n: int = 200, stream=None) -> tuple[float, float, float]:
    """(mu_msv, mu_vit, tau) in bits for a synth.Profile-like profile."""
    import torch
    from synth import gen
    P = Profile(prof, 0.0, 0.0, 0.0)
    out = {}
    for key, seed, L in (("filters", gen.SEED_CALIB_VIT, 200), ("forward", gen.SEED_CALIB_FWD, 100)):
        db = gen.random_sequences(seed, n, L)
        D = Database(db.residues, db.offsets)
        r = search(P, D, (1.0, 1.0, 1.0), stream=stream)
        torch.cuda.synchronize()
        out[key] = {k: v.cpu().numpy() for k, v in r.items()}
        D.close()
    P.close()
    nul200, nul100 = null_score(200), null_score(100)
    msv_bits = ((out["filters"]["msv"].astype(np.float64) - BASE8) / S8 - 3.0 - nul200) / LN2
    vit_bits = (out["filters"]["vit"].astype(np.float64) / S16 - 3.0 - nul200) / LN2
    fwd_bits = np.sort((out["forward"]["fwd"].astype(np.float64) - nul100) / LN2)[::-1]
    xc = fwd_bits[int(round(TAIL * n)) - 1]
    return _gumbel_location(msv_bits), _gumbel_location(vit_bits), float(xc + math.log(TAIL) / LN2)
