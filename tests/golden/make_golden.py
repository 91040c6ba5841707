"""Write tests/golden/small_cases.json: oracle outputs on small seeded cases.

The paper prints no worked example, score or bound for the search path
(its figures are not in the text either), so no fixture can quote it.
These fixtures freeze what the oracle computes, on inputs small enough to
read, so that a later change of the oracle's arithmetic shows up as a
diff; the oracle itself is pinned by brute force, closed forms and
invariants (tests/test_oracle_*.py).  This script calls only oracle/ and
the seeded input generators; run it from the repository root:

    python tests/golden/make_golden.py
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from synth import gen  # noqa: E402

CASES = [  # (M, profile seed, database size, database seed, planted fraction)
    (3, 11, 6, 21, 0.5),
    (12, 12, 8, 22, 0.5),
    (40, 13, 10, 23, 0.3),
]


def main():
    out = []
    for M, ps, n, ds, planted in CASES:
        prof = gen.make_profile(M, ps)
        db = gen.make_database(n, ds, prof, planted, len_lo=5, len_hi=90)
        op = oracle.OracleProfile(prof)
        calib = (0.0, 0.0, 0.0)
        F = (1.0, 1.0, 1.0)
        r = oracle.search(op, db.residues, db.offsets, calib, F, nthreads=1)
        targets = []
        for t in range(db.n):
            x = db.residues[db.offsets[t]:db.offsets[t + 1]]
            dec, doms = oracle.domains(op, x)
            targets.append(dict(
                residues=[int(v) for v in x],
                msv=int(r["msv"][t]), vit=int(r["vit"][t]), fwd=float(r["fwd"][t]), flags=int(r["flags"][t]),
                vit_f64=oracle.vit_f64(op, x),
                core=[float(v) for v in dec["core"]],
                domains=[dict(s=d["s"], e=d["e"], a=d["a"], b=d["b"], k1=d["k1"], k2=d["k2"],
                              score=d["score"], nexp=d["nexp"], code=[int(v) for v in d["code"]]) for d in doms]))
        out.append(dict(M=M, profile_seed=ps, bg=prof.bg.tolist(), match=prof.match.tolist(),
                        insert=prof.insert.tolist(), trans=prof.trans.tolist(), cutoffs=list(F),
                        calib=list(calib), targets=targets))
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "small_cases.json")
    with open(path, "w") as f:
        json.dump(dict(source="oracle/ (hmm_oracle.c) via tests/golden/make_golden.py", cases=out), f,
                  separators=(",", ":"))
    print(f"wrote {path}")


if __name__ == "__main__":
    main()
