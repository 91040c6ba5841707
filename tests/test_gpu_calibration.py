"""GPU parity of the score calibration that sets the benchmark's cutoffs.

paper_2111_06340_amd.calibrate scores the same seeded background
sequences as oracle.calibrate, on the GPU: the MSV and Viterbi scores are
bit-exact with the oracle's, so the Gumbel locations agree to rounding;
the Forward location tau is an order statistic of fp32 Forward scores,
each within the Forward tolerance of the oracle's fp64 score, so tau moves
by at most the largest of those tolerances (in bits)."""
import math

import numpy as np
import pytest

import oracle
from paper_2111_06340_amd.calibrate import calibrate as gpu_calibrate
from synth import gen

pytestmark = pytest.mark.gpu

FWD_ABS, FWD_REL = 1e-3, 1e-5


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    return torch


def check_calibration(prof, what):
    op = oracle.OracleProfile(prof)
    o = oracle.calibrate(op, nthreads=16)
    g = gpu_calibrate(prof)
    print(f"[gpu-calib] {what} M={prof.M}: oracle {o} gpu {g}", flush=True)
    assert g[0] == pytest.approx(o[0], abs=1e-9)
    assert g[1] == pytest.approx(o[1], abs=1e-9)
    db = gen.random_sequences(gen.SEED_CALIB_FWD, 200, 100)
    r = oracle.search(op, db.residues, db.offsets, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0), nthreads=16)
    tol_bits = float(np.max(FWD_ABS + FWD_REL * np.abs(r["fwd"]))) / math.log(2.0)
    assert abs(g[2] - o[2]) <= tol_bits, (g[2], o[2], tol_bits)


@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C5"])
def test_package_calibration_equals_the_oracle(name):
    check_calibration(gen.workload_profile(gen.WORKLOADS[name]), name)


@pytest.mark.parametrize("p", [0, 17, 40])
def test_package_calibration_of_c4_profiles(p):
    check_calibration(gen.c4_profiles()[p], f"C4 profile {p}")
