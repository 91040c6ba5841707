"""Host-side logic of bench.py (no GPU): the one-GPU contract, the roofline
arithmetic and the committed counter records it reads."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_peaks_follow_from_the_unit_counts():
    assert bench.PEAK_PK16_TOPS == pytest.approx(256 * 64 * 2 * 2.4e9 / 1e12)
    assert bench.PEAK_PK16_TOPS == pytest.approx(78.64, abs=0.01)
    assert bench.PEAK_I32_TOPS == pytest.approx(bench.PEAK_PK16_TOPS / 2)


def test_stage_roofline_arithmetic():
    # one profile of M = 100 over 1e9 residues: 4e11 MSV ops in 10 ms = 40 Tops/s
    ran = {"viterbi": 10**9, "rescore": 10**8, "forward": 10**8}
    out = bench.stage_roofline([100], 10**9, ran, [10.0, 1.0, 1.0, 2.0], chunks=1)
    assert out["msv"]["algorithmic_achieved"] == pytest.approx(40.0)
    assert out["msv"]["algorithmic_frac"] == pytest.approx(40.0 / bench.PEAK_PK16_TOPS, abs=1e-4)
    assert out["viterbi"]["algorithmic_achieved"] == pytest.approx(18.0)     # 18 ops x 1e9 cells / 1 ms
    assert out["rescore"]["algorithmic_achieved"] == pytest.approx(1.7)      # 17 ops x 1e8 cells / 1 ms
    assert out["forward"]["algorithmic_achieved"] == pytest.approx(0.9)      # 18 flops x 1e8 cells / 2 ms
    # pipelined: only MSV's fraction is meaningful
    piped = bench.stage_roofline([100], 10**9, ran, [10.0, 1.0, 1.0, 2.0], chunks=2)
    assert set(piped) == {"msv", "note"}
    # fused tail: one time for Viterbi, rescore and Forward (the Viterbi stage's)
    fused = bench.stage_roofline([100], 10**9, ran, [10.0, 3.0, 0.01, 0.02], chunks=1, fused=True)
    assert set(fused) == {"msv", "tail"} and fused["tail"]["ms"] == pytest.approx(3.0)


@pytest.mark.parametrize("name", ["msv_traffic_C3.json", "decode_traffic_C3.json"])
def test_counter_records_are_consistent(name):
    with open(os.path.join(ROOT, "profiles", name)) as f:
        tr = json.load(f)
    assert tr["workload"] == "C3"
    assert len(tr["kernel_source_sha"]) == 16 and len(tr["header_sha"]) == 16
    fetch = tr.get("fetch_bytes_per_launch", tr.get("fetch_bytes"))
    write = tr.get("write_bytes_per_launch", tr.get("write_bytes"))
    assert tr["bytes_per_launch"] == fetch + write
    assert tr["scale"]["FETCH_SIZE"] == pytest.approx(2.0, abs=0.01)
    if name.startswith("msv"):
        assert tr["launches_per_search"] >= 1
        assert tr["bytes_per_search"] == tr["launches_per_search"] * tr["bytes_per_launch"]
        # the kernel reads every residue of its chunk at least once
        assert tr["bytes_per_launch"] >= tr["algorithmic_bytes_per_launch"]
        # at least one VALU instruction per two cells of the launch's chunk
        cells = 734 * tr["algorithmic_bytes_per_launch"] * 0.9
        assert tr["valu_insts_per_launch"] * 64 * 2 >= cells


def test_valu_issue_arithmetic():
    # 1e9 wave instructions in 5 ms on a chip that sustains 128e12
    # element-ops/s (1e12 wave instructions/s): 0.2 of the issue rate
    out = bench.valu_issue(1e9, 5.0, 128e12)
    assert out["sustained_insts_per_s"] == pytest.approx(1e12)
    assert out["frac"] == pytest.approx(0.2)


def test_issue_roofline_arithmetic_and_the_committed_record():
    # 6.144e9 wave instructions in 10 ms = the datasheet rate: fraction 1
    out = bench.issue_roofline(6.144e9, 10.0)
    assert out["frac"] == pytest.approx(1.0)
    assert out["achieved"] == pytest.approx(bench.PEAK_PK16_TOPS, abs=0.01)
    # the C3 record: 5.709e9 instructions in the 10.231 ms launch of the
    # committed kernel trace is 0.91 of the datasheet issue rate
    with open(os.path.join(ROOT, "profiles", "msv_traffic_C3.json")) as f:
        tr = json.load(f)
    frac = bench.issue_roofline(tr["valu_insts_per_launch"], tr.get("ms_per_launch", 6.121))["frac"]
    assert 0.5 < frac <= 1.0


def test_cpu_baseline_threads_and_host():
    h = bench.host_cpus()
    assert h["nproc"] >= h["affinity"] >= 1
    assert 1 <= bench.oracle_threads() <= h["affinity"]


def test_kernel_source_sha_is_the_file_hash():
    import hashlib
    p = os.path.join(ROOT, "paper_2111_06340_amd", "csrc", "hmm_kernels.hip")
    with open(p, "rb") as f:
        assert bench.kernel_source_sha() == hashlib.sha256(f.read()).hexdigest()[:16]
