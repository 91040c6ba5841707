"""Frozen oracle outputs on small seeded cases (tests/golden/small_cases.json,
written by tests/golden/make_golden.py, which calls only the oracle).

The paper prints no worked example for this path, so the fixtures are
the oracle's own: this test turns any later change of the oracle's
arithmetic into a visible diff (such a change must name, in its commit,
the reading that justifies it).  The GPU side is checked against the same
fixtures in tests/test_gpu_decode.py."""
import json
import os

import numpy as np
import pytest

import oracle
from synth import Profile

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "small_cases.json")


def load_cases():
    with open(GOLDEN) as f:
        return json.load(f)["cases"]


def case_profile(c) -> Profile:
    M = c["M"]
    return Profile(M, np.array(c["bg"]), np.array(c["match"]), np.array(c["insert"]).reshape(max(M - 1, 0), 20),
                   np.array(c["trans"]).reshape(max(M - 1, 0), 7))


def case_database(c):
    seqs = [np.array(t["residues"], np.uint8) for t in c["targets"]]
    off = np.zeros(len(seqs) + 1, np.int64)
    off[1:] = np.cumsum([s.size for s in seqs])
    return np.concatenate(seqs), off


@pytest.mark.parametrize("ci", range(3))
def test_oracle_reproduces_its_frozen_outputs(ci):
    c = load_cases()[ci]
    op = oracle.OracleProfile(case_profile(c))
    res, off = case_database(c)
    r = oracle.search(op, res, off, c["calib"], c["cutoffs"], nthreads=1)
    for t, want in enumerate(c["targets"]):
        x = res[off[t]:off[t + 1]]
        assert int(r["msv"][t]) == want["msv"] and int(r["vit"][t]) == want["vit"]
        assert int(r["flags"][t]) == want["flags"]
        assert float(r["fwd"][t]) == pytest.approx(want["fwd"], abs=1e-12)
        assert oracle.vit_f64(op, x) == pytest.approx(want["vit_f64"], abs=1e-12)
        dec, doms = oracle.domains(op, x)
        np.testing.assert_allclose(dec["core"], want["core"], rtol=0, atol=1e-12)
        assert [(d["s"], d["e"], d["a"], d["b"], d["k1"], d["k2"]) for d in doms] == \
               [(d["s"], d["e"], d["a"], d["b"], d["k1"], d["k2"]) for d in want["domains"]]
        for d, w in zip(doms, want["domains"]):
            assert d["score"] == pytest.approx(w["score"], abs=1e-12)
            assert d["nexp"] == pytest.approx(w["nexp"], abs=1e-12)
            assert list(d["code"]) == w["code"]
            sc, ok = oracle.oa_path_score(op, dec, w["s"], w["e"], np.array(w["code"], np.int16))
            assert ok and sc == pytest.approx(w["score"], abs=1e-12)


def test_fixtures_cover_hits_and_misses():
    cases = load_cases()
    ndom = [sum(len(t["domains"]) for t in c["targets"]) for c in cases]
    assert all(n > 0 for n in ndom)
    assert any(len(t["domains"]) == 0 for c in cases for t in c["targets"])
