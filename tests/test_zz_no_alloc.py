"""hmm_decode_static: posterior decoding on the library's fixed device
scratch, for callers that cannot allocate.  Through the C ABI, its outputs
must equal hmm_decode's on the same inputs -- on two calls in a row, the
second with a smaller database (the fixed array keeps the first call's
contents) -- it must not allocate device memory, and it must reject a
database whose four wave slots exceed the array before enqueuing anything.

The two entry points run the same kernel on the same targets; only the
scratch addresses and the number of waves differ, and each target is
decoded by one wave alone, so the results are identical bit for bit (the
domain records come in completion order and are compared sorted)."""
import numpy as np
import pytest

import oracle
import paper_2111_06340_amd as hg
from synth import gen

pytestmark = pytest.mark.gpu


def announce(msg):
    print(f"[no-alloc] {msg}", flush=True)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    hg.lib()
    return torch


def host(dec):
    return dict(exp_dom=dec["exp_dom"].cpu().numpy(), pp=dec["pp"].cpu().numpy(), aln=dec["aln"].cpu().numpy(),
                doms=hg.domains_table(dec), n_dom=int(dec["n_dom"].cpu()[0]))


def same(a, b, what):
    assert a["n_dom"] == b["n_dom"], (what, a["n_dom"], b["n_dom"])
    assert a["doms"] == b["doms"], what
    for k in ("exp_dom", "pp"):
        assert np.array_equal(np.isnan(a[k]), np.isnan(b[k])), (what, k)
        m = ~np.isnan(a[k])
        assert np.array_equal(a[k][m], b[k][m]), (what, k)
    assert np.array_equal(a["aln"], b["aln"]), what


def decode_both(P, D, flags, what):
    """Static decode, then the allocating one, of the same selection; the
    free device memory must not fall during the static call."""
    import torch
    dec_s = hg.decode(P, D, flags=flags, mask=hg.HMM_FWD_PASS, pp=True, aln=True, static=True)
    torch.cuda.synchronize()
    gs = host(dec_s)
    dec_a = hg.decode(P, D, flags=flags, mask=hg.HMM_FWD_PASS, pp=True, aln=True)
    torch.cuda.synchronize()
    ga = host(dec_a)
    same(gs, ga, what)
    announce(f"{what}: {gs['n_dom']} regions, static = allocating")
    return gs


def test_static_decode_equals_decode_twice_second_smaller():
    import torch
    w = gen.WORKLOADS["C3"]
    prof = gen.workload_profile(w)
    calib = oracle.calibrate(oracle.OracleProfile(prof), nthreads=16)
    P = hg.Profile(prof, *calib)
    F = (0.2, 0.05, 1.0)
    sizes = (3000, 700)
    for rnd, n in enumerate(sizes):
        db = gen.workload_database(w, n=n, prof=prof, seed_offset=7 + rnd)
        D = hg.Database(db.residues, db.offsets)
        announce(f"call {rnd + 1}: M={prof.M} n={D.n} residues={D.n_residues} max_len={D.max_len}")
        out = hg.search(P, D, F)
        torch.cuda.synchronize()
        # outputs allocated first, so that only the call itself is measured
        dom = hg.decode(P, D, flags=out["flags"], mask=0xff, pp=True, aln=True)   # selects nothing
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info()[0]
        hg.hmm_decode_static(P.handle, D.handle, out["flags"], hg.HMM_FWD_PASS, dom)
        torch.cuda.synchronize()
        free1 = torch.cuda.mem_get_info()[0]
        assert free0 - free1 < (4 << 20), (free0, free1)
        g = decode_both(P, D, out["flags"], f"call {rnd + 1} n={n}")
        assert g["n_dom"] > 0
        # the measured call wrote the same results
        same(host(dom), g, f"call {rnd + 1} (measured)")
        D.close()
    P.close()


def test_static_decode_long_profile_and_rejection():
    import torch
    prof = gen.make_profile(2500, 31)
    rng = np.random.default_rng(3)
    homs = gen.sample_homologs(rng, prof, 3)
    seqs = [gen.background_residues(rng, 300), homs[0], np.concatenate([gen.background_residues(rng, 100), homs[1]]),
            gen.background_residues(rng, 40)]
    off = np.zeros(len(seqs) + 1, np.int64)
    off[1:] = np.cumsum([s.size for s in seqs])
    P = hg.Profile(prof, -8.0, -9.0, -4.0)
    D = hg.Database(np.concatenate(seqs), off)
    out = hg.search(P, D, (1.0, 1.0, 1.0))
    torch.cuda.synchronize()
    g = decode_both(P, D, None, f"M=2500 n={D.n} max_len={D.max_len}")
    assert g["n_dom"] >= 2
    D.close()
    # a 7,000-residue target: four slots of about 153 MB exceed the 512 MiB array
    D = hg.Database(gen.background_residues(rng, 7000), np.array([0, 7000], np.int64))
    dom = hg.decode(P, D, flags=None, mask=0xff)     # allocating path: fine
    torch.cuda.synchronize()
    with pytest.raises(hg.HmmError) as e:
        hg.hmm_decode_static(P.handle, D.handle, None, 0, dom)
    assert e.value.status == hg.HMM_ERANGE
    assert "static scratch" in hg.hmm_last_error()
    torch.cuda.synchronize()
    D.close()
    P.close()
    assert out is not None
