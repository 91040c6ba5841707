"""C-ABI checks that need no GPU: the library loads and exports every entry
point the header declares; argument validation rejects bad input on the
host before any GPU call; the host-side quantisation and per-length cutoffs
equal the oracle's, which are written independently."""
import math
import os
import re

import numpy as np
import pytest

import oracle
import paper_2111_06340_amd as hg
from conftest import ROOT, random_profile
from synth import gen

HEADER = os.path.join(ROOT, "include", "hmmgpu.h")


def _declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(hmm_[a-z_0-9]+)\s*\(", txt)))


def test_library_exports_every_declared_symbol():
    names = _declared()
    assert len(names) >= 10
    L = hg.lib()
    for n in names:
        assert hasattr(L, n), n
    assert sorted(hg.EXPORTED) == names


def test_header_constants_match_binding():
    txt = open(HEADER).read()
    floats = dict(re.findall(r"#define (HMM_[A-Z_0-9]+) ([0-9]+\.[0-9]+)f\b", txt))
    consts = dict(re.findall(r"#define (HMM_[A-Z_0-9]+) \(?(-?(?:0x)?[0-9a-fA-F]+)\)?(?:\s|$)", txt))
    assert set(floats) == {"HMM_RT1", "HMM_RT2"}
    for k, v in consts.items():
        assert getattr(hg, k) == int(v, 0), k
    for k, v in floats.items():
        assert getattr(hg, k) == float(v), k
        assert np.float32(getattr(hg, k)) == np.float32(float(v))
    # the library's region thresholds are the oracle's
    assert (hg.HMM_RT1, hg.HMM_RT2) == (oracle.RT1, oracle.RT2)


def test_strerror():
    for code in (hg.HMM_OK, hg.HMM_EINVAL, hg.HMM_ERANGE, hg.HMM_ENOMEM, hg.HMM_EDEVICE):
        assert hg.hmm_strerror(code)
    assert hg.hmm_strerror(-99) == "unknown status"


def _status(fn, *a, **k):
    try:
        fn(*a, **k)
    except hg.HmmError as e:
        return e.status
    return hg.HMM_OK


def _bad_profiles():
    good = gen.make_profile(5, 1)

    def mod(**kw):
        d = dict(M=good.M, bg=good.bg.copy(), match=good.match.copy(), insert=good.insert.copy(),
                 trans=good.trans.copy())
        d.update(kw)
        return d

    m = good.match.copy(); m[2, 3] += 0.01
    yield "row sum", mod(match=m), hg.HMM_EINVAL
    m = good.match.copy(); m[0, 0] = -m[0, 0]
    yield "negative", mod(match=m), hg.HMM_EINVAL
    m = good.match.copy(); m[1, 0] += m[1, 1]; m[1, 1] = 0.0
    yield "zero match", mod(match=m), hg.HMM_EINVAL
    b = good.bg.copy(); b[0] = np.nan
    yield "nan bg", mod(bg=b), hg.HMM_EINVAL
    t = good.trans.copy(); t[0, 0] -= 0.1
    yield "trans group", mod(trans=t), hg.HMM_EINVAL
    t = good.trans.copy(); t[1, 5] = 0.7
    yield "trans D group", mod(trans=t), hg.HMM_EINVAL
    yield "M=0", dict(M=0, bg=good.bg, match=good.match, insert=good.insert, trans=good.trans), hg.HMM_EINVAL
    big = gen.make_profile(3073, 2)
    yield "M>max", dict(M=3073, bg=big.bg, match=big.match, insert=big.insert, trans=big.trans), hg.HMM_ERANGE


@pytest.mark.parametrize("case", list(_bad_profiles()), ids=lambda c: c[0])
def test_profile_validation(case):
    _, d, code = case
    assert _status(hg.hmm_profile_upload, d["M"], d["bg"], d["match"], d["insert"], d["trans"],
                   0.0, 0.0, 0.0) == code
    assert hg.hmm_last_error()


def test_profile_calibration_must_be_finite():
    p = gen.make_profile(4, 1)
    assert _status(hg.hmm_profile_upload, 4, p.bg, p.match, p.insert, p.trans, math.nan, 0.0, 0.0) == hg.HMM_EINVAL


@pytest.mark.parametrize("residues,offsets,code", [
    (np.array([1, 2, 20], np.uint8), np.array([0, 3]), hg.HMM_EINVAL),        # bad code
    (np.array([1, 2, 3], np.uint8), np.array([0, 2, 2, 3]), hg.HMM_EINVAL),   # empty sequence
    (np.array([1, 2, 3], np.uint8), np.array([1, 3]), hg.HMM_EINVAL),         # offsets[0] != 0
    (np.array([1, 2, 3], np.uint8), np.array([0, 3, 2]), hg.HMM_EINVAL),      # decreasing
    (np.zeros(100001, np.uint8), np.array([0, 100001]), hg.HMM_ERANGE),       # too long
])
def test_db_validation(residues, offsets, code):
    assert _status(hg.hmm_db_upload, residues, offsets) == code
    assert hg.hmm_last_error()


def test_search_rejects_null_handles():
    import ctypes as C
    t = hg.hmm_thresholds(1.0, 1.0, 1.0)
    r = hg.hmm_results()
    assert hg.lib().hmm_search(None, None, C.byref(t), C.byref(r), None) == hg.HMM_EINVAL
    assert hg.lib().hmm_profile_free(None) == hg.HMM_OK
    assert hg.lib().hmm_db_free(None) == hg.HMM_OK
    cur = C.c_int32(-7)
    assert hg.lib().hmm_db_fused_tail(None, 2, C.byref(cur)) == hg.HMM_EINVAL and cur.value == -7
    assert hg.lib().hmm_db_pipeline(None, 2, C.byref(cur)) == hg.HMM_EINVAL and cur.value == -7


def _gpu_present():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


@pytest.mark.skipif(_gpu_present(), reason="checks the no-device error path")
def test_no_device_reports_edevice_without_crash():
    p = gen.make_profile(10, 3)
    assert _status(hg.hmm_profile_upload, 10, p.bg, p.match, p.insert, p.trans, 0.0, 0.0, 0.0) == hg.HMM_EDEVICE
    assert "hip" in hg.hmm_last_error().lower() or hg.hmm_last_error()


# ------------------------------------------------------------ tables

def _table_profiles():
    for w in gen.WORKLOADS.values():
        yield w.name, gen.workload_profile(w)
    for M, s in ((1, 1), (2, 2), (3, 3), (127, 4), (128, 5), (129, 6), (300, 7)):
        yield f"random{M}", random_profile(M, s, alpha=0.2, talpha=0.5)
    yield "c4_first", gen.c4_profiles(1)[0]
    # extreme probabilities: saturating scores, zero transitions and inserts
    p = gen.make_profile(20, 9)
    p.match[3, 0] = 1e-30
    p.match[3, 1] += 0.5 - 1e-30
    p.match[3] /= p.match[3].sum()
    p.insert[2, :] = 0.0
    p.insert[2, 5] = 1.0
    p.trans[4] = [1.0, 0.0, 0.0, 1.0, 0.0, 0.0, 1.0]
    yield "extreme", p


@pytest.mark.parametrize("name,prof", list(_table_profiles()), ids=lambda v: v if isinstance(v, str) else "")
def test_library_tables_equal_oracle_tables(name, prof):
    lt = hg.hmm_debug_tables(prof)
    op = oracle.OracleProfile(prof)
    ot = op.tables()
    osc = op.scalars()
    for k in ("bias8", "entry8", "exit8", "entry16", "ej16"):
        assert lt[k] == osc[k], k
    assert np.array_equal(lt["cost8"], ot["cost8"])
    assert np.array_equal(lt["msc16"], ot["msc16"])
    assert np.array_equal(lt["isc16"], ot["isc16"])
    assert np.array_equal(lt["t16"], ot["t16"])
    assert lt["Q8"] * 128 >= prof.M and lt["Q32"] * 64 >= prof.M


@pytest.mark.parametrize("F", [(1.0, 1.0, 1.0), (0.02, 1e-3, 1.0), (0.2, 0.01, 1e-3), (1e-6, 1e-9, 0.5)])
def test_length_params_equal_oracle(F):
    prof = gen.make_profile(50, 5)
    calib = (-8.6, -9.7, -4.1)
    for L in list(range(1, 40)) + [99, 100, 255, 256, 257, 1000, 4999, 5000, 99999, 100000]:
        lib = hg.hmm_debug_length_params(prof, calib, F, L)
        o = oracle.length_params(L)
        t8, t16, ft = oracle.thresholds(calib, F, L)
        assert (lib["move8"], lib["move16"]) == (o["move8"], o["move16"])
        assert (lib["thr8"], lib["thr16"]) == (t8, t16)
        assert lib["loop"] == o["loop"] and lib["move"] == o["move"] and lib["null"] == o["null"]
        assert lib["fwd_thr"] == ft or (math.isinf(ft) and math.isinf(lib["fwd_thr"]))


def test_decode_rejects_bad_arguments_on_the_host():
    import ctypes as C
    L = hg.lib()
    out = hg.hmm_decode_out(None, 0, None, None, None, None)
    # NULL profile / db / out, NULL dom or n_dom, negative max_dom: rejected before any GPU call
    assert L.hmm_decode(None, None, None, 0, C.byref(out), None) == hg.HMM_EINVAL
    assert L.hmm_decode(C.c_void_p(1), C.c_void_p(1), None, 0, None, None) == hg.HMM_EINVAL
    assert L.hmm_decode(C.c_void_p(1), C.c_void_p(1), None, 0, C.byref(out), None) == hg.HMM_EINVAL
    assert "dom" in hg.hmm_last_error()
    bad = hg.hmm_decode_out(C.c_void_p(8).value, -1, C.c_void_p(8).value, None, None, None)
    assert L.hmm_decode(C.c_void_p(1), C.c_void_p(1), None, 0, C.byref(bad), None) == hg.HMM_EINVAL
    assert "max_dom" in hg.hmm_last_error()


@pytest.mark.parametrize("M,seed", [(1, 0), (2, 1), (30, 2), (257, 3)])
def test_rebuild_equals_oracle_estimate(M, seed):
    """hmm_rebuild (library host code) against the oracle's numpy estimate,
    written independently; both fp64."""
    prof = random_profile(M, seed)
    rng = np.random.default_rng(seed)
    c = dict(match=rng.integers(0, 50, (M, 20)), insert=rng.integers(0, 5, (max(M - 1, 0), 20)),
             trans=rng.integers(0, 80, (max(M - 1, 0), 7)))
    flat = np.concatenate([c["match"].ravel(), c["insert"].ravel(), c["trans"].ravel()]).astype(np.uint32)
    got = hg.hmm_rebuild(prof, flat, 20.0, 10.0)
    want = oracle.rebuild_profile(prof, c, 20.0, 10.0)
    np.testing.assert_allclose(got.match, want.match, rtol=0, atol=1e-15)
    np.testing.assert_allclose(got.insert, want.insert, rtol=0, atol=1e-15)
    np.testing.assert_allclose(got.trans, want.trans, rtol=0, atol=1e-15)


def test_rebuild_rejects_bad_arguments():
    prof = random_profile(5, 1)
    z = np.zeros(hg.count_size(5), np.uint32)
    for A, B in ((0.0, 1.0), (1.0, -1.0), (float("nan"), 1.0)):
        with pytest.raises(hg.HmmError) as e:
            hg.hmm_rebuild(prof, z, A, B)
        assert e.value.status == hg.HMM_EINVAL
