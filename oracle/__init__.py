"""CPU oracle for Plan7 profile-HMM database search (ctypes over hmm_oracle.c).

TEST INFRASTRUCTURE.  Only the test suite, the package smoke check and the
benchmark's CPU-baseline leg may import this package.  It shares no code
with the GPU library (paper_2111_06340_amd); both consume the seeded inputs
of the `synth` package and nothing else in common.

Functions take numpy arrays and return Python scalars / numpy arrays.
Score conversions to bits and the score calibration below follow the
readings stated in hmm_oracle.c (lambda = ln 2 per bit, Gumbel law for the
MSV and Viterbi filter scores, exponential tail for Forward).
"""
from __future__ import annotations

import ctypes as C
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hmm_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

S8 = 3.0 / math.log(2.0)
S16 = 500.0 / math.log(2.0)
BASE8 = 190
LN2 = math.log(2.0)

F_MSV_PASS, F_MSV_OVF, F_VIT_RAN, F_VIT_PASS, F_VIT_OVF, F_FWD_RAN, F_FWD_PASS, F_BIAS_PASS = (
    0x01, 0x02, 0x04, 0x08, 0x10, 0x20, 0x40, 0x80)
BIAS_SWITCH = 1.0 / 64.0


def build(force: bool = True) -> str:
    """Compile the oracle (scalar on purpose: -O2 -fno-tree-vectorize)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fno-tree-vectorize", "-std=c11", "-D_GNU_SOURCE",
                               "-Wall", "-shared", "-fPIC", "-o", tmp, _SRC, "-lm", "-lpthread"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def build_variant(src_text: str, out_path: str) -> str:
    """Compile a modified copy of the oracle source (mutation tests)."""
    src = out_path + ".c"
    with open(src, "w") as f:
        f.write(src_text)
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-D_GNU_SOURCE", "-w", "-shared", "-fPIC",
                           "-o", out_path, src, "-lm", "-lpthread"])
    return out_path


def source_text() -> str:
    with open(_SRC) as f:
        return f.read()


def load(path: str):
    """Load an oracle build and declare its signatures."""
    L = C.CDLL(path)
    vp, ip, dp = C.c_void_p, C.c_int, C.c_double
    L.orc_profile_new.restype = vp
    L.orc_profile_new.argtypes = [ip, vp, vp, vp, vp]
    L.orc_profile_free.argtypes = [vp]
    L.orc_profile_scalars.argtypes = [vp, vp]
    L.orc_profile_tables.argtypes = [vp, vp, vp, vp, vp]
    for f in ("orc_loop", "orc_move", "orc_null"):
        getattr(L, f).restype = dp
        getattr(L, f).argtypes = [ip]
    for f in ("orc_move8", "orc_move16"):
        getattr(L, f).restype = ip
        getattr(L, f).argtypes = [ip]
    L.orc_thresholds.argtypes = [vp, vp, ip, vp, vp, vp]
    L.orc_msv.restype = ip
    L.orc_msv.argtypes = [vp, vp, ip, vp]
    L.orc_vit16.restype = ip
    L.orc_vit16.argtypes = [vp, vp, ip, vp]
    L.orc_vit32.restype = C.c_int32
    L.orc_vit32.argtypes = [vp, vp, ip]
    for f in ("orc_vit_f64", "orc_fwd_f64", "orc_fwd_f64_scaled"):
        getattr(L, f).restype = dp
        getattr(L, f).argtypes = [vp, vp, ip]
    L.orc_search.restype = ip
    L.orc_search.argtypes = [vp, vp, vp, C.c_int64, vp, vp, ip, ip, vp, vp, vp, vp, vp]
    if hasattr(L, "orc_search_bias"):
        L.orc_search_bias.restype = ip
        L.orc_search_bias.argtypes = [vp, vp, vp, C.c_int64, vp, vp, ip, ip, ip, vp, vp, vp, vp, vp, vp]
        L.orc_bias.restype = dp
        L.orc_bias.argtypes = [vp, vp, ip]
    if hasattr(L, "orc_decode"):
        L.orc_decode.restype = ip
        L.orc_decode.argtypes = [vp, vp, ip, vp, vp, vp, vp, vp, vp, vp]
        L.orc_regions.restype = ip
        L.orc_regions.argtypes = [vp, ip, dp, dp, vp, ip]
        L.orc_oa_align.restype = dp
        L.orc_oa_align.argtypes = [vp, ip, vp, vp, vp, ip, ip, vp, vp]
        L.orc_oa_path_score.restype = dp
        L.orc_oa_path_score.argtypes = [vp, ip, vp, vp, vp, ip, ip, vp, vp]
    return L


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        _lib = load(_LIB)
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


class OracleProfile:
    """Oracle-side scores and integer tables of one profile."""

    def __init__(self, prof, library=None):
        self.lib = lib() if library is None else library
        self.M = int(prof.M)
        self._keep = [np.ascontiguousarray(prof.bg, np.float64),
                      np.ascontiguousarray(prof.match, np.float64),
                      np.ascontiguousarray(prof.insert, np.float64).reshape(-1),
                      np.ascontiguousarray(prof.trans, np.float64).reshape(-1)]
        if self._keep[2].size == 0:
            self._keep[2] = np.zeros(1)
            self._keep[3] = np.zeros(1)
        self.h = self.lib.orc_profile_new(self.M, *[_ptr(a) for a in self._keep])
        if not self.h:
            raise ValueError("oracle rejected the profile")

    def __del__(self):
        h = getattr(self, "h", None)
        if h:
            self.lib.orc_profile_free(h)
            self.h = None

    def scalars(self) -> dict:
        out = np.zeros(5, np.int32)
        self.lib.orc_profile_scalars(self.h, _ptr(out))
        return dict(bias8=int(out[0]), entry8=int(out[1]), exit8=int(out[2]),
                    entry16=int(out[3]), ej16=int(out[4]))

    def tables(self) -> dict:
        M = self.M
        cost8 = np.zeros((M, 20), np.uint8)
        msc16 = np.zeros((M, 20), np.int16)
        isc16 = np.zeros((max(M - 1, 1), 20), np.int16)
        t16 = np.zeros((max(M - 1, 1), 7), np.int16)
        self.lib.orc_profile_tables(self.h, _ptr(cost8), _ptr(msc16), _ptr(isc16), _ptr(t16))
        return dict(cost8=cost8, msc16=msc16, isc16=isc16[:M - 1], t16=t16[:M - 1])


def _seq(x) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.uint8)
    if x.size < 1:
        raise ValueError("empty sequence")
    return x


def msv(p: OracleProfile, x) -> tuple[int, int]:
    x = _seq(x)
    ovf = C.c_int(0)
    r = p.lib.orc_msv(p.h, _ptr(x), x.size, C.byref(ovf))
    return int(r), int(ovf.value)


def vit16(p: OracleProfile, x) -> tuple[int, int]:
    x = _seq(x)
    ovf = C.c_int(0)
    r = p.lib.orc_vit16(p.h, _ptr(x), x.size, C.byref(ovf))
    return int(r), int(ovf.value)


def vit32(p: OracleProfile, x) -> int:
    x = _seq(x)
    return int(p.lib.orc_vit32(p.h, _ptr(x), x.size))


def vit_f64(p: OracleProfile, x) -> float:
    x = _seq(x)
    return float(p.lib.orc_vit_f64(p.h, _ptr(x), x.size))


def fwd_f64(p: OracleProfile, x) -> float:
    x = _seq(x)
    return float(p.lib.orc_fwd_f64(p.h, _ptr(x), x.size))


def fwd_f64_scaled(p: OracleProfile, x) -> float:
    x = _seq(x)
    return float(p.lib.orc_fwd_f64_scaled(p.h, _ptr(x), x.size))


def length_params(L: int, library=None) -> dict:
    l = lib() if library is None else library
    return dict(loop=l.orc_loop(L), move=l.orc_move(L), null=l.orc_null(L),
                move8=l.orc_move8(L), move16=l.orc_move16(L))


def thresholds(calib, F, L: int, library=None) -> tuple[int, int, float]:
    """(THR8(L), THR16(L), Forward cutoff in nats) of orc_thresholds."""
    c = np.asarray(calib, np.float64)
    f = np.asarray(F, np.float64)
    t8, t16, ft = C.c_int32(0), C.c_int32(0), C.c_double(0)
    (lib() if library is None else library).orc_thresholds(_ptr(c), _ptr(f), L, C.byref(t8), C.byref(t16),
                                                           C.byref(ft))
    return int(t8.value), int(t16.value), float(ft.value)


# ------------------------------------------------------------ bit scores

def msv_bits(raw: int, L: int) -> float:
    return ((raw - BASE8) / S8 - 3.0 - lib().orc_null(L)) / LN2


def vit_bits(v: int, L: int) -> float:
    return (v / S16 - 3.0 - lib().orc_null(L)) / LN2


def fwd_bits(f: float, L: int) -> float:
    return (f - lib().orc_null(L)) / LN2


def gumbel_mu(bits: np.ndarray, lam: float = LN2) -> float:
    """Maximum-likelihood Gumbel location with the slope fixed at lam."""
    b = np.asarray(bits, np.float64)
    return float(-math.log(np.mean(np.exp(-lam * b))) / lam)


FWD_TAIL = 0.04     # tail mass the Forward location is fitted at


def exp_tail_location(bits, tail: float = FWD_TAIL, lam: float = LN2) -> float:
    """Location tau of an exponential tail P(S > x) = exp(-lam (x - tau))
    that gives the (tail * n)-th largest of n scores the survival `tail`:
    exp(-lam (x_c - tau)) = tail, so tau = x_c + ln(tail) / lam."""
    b = np.sort(np.asarray(bits, np.float64))[::-1]
    xc = b[int(round(tail * b.size)) - 1]
    return float(xc + math.log(tail) / lam)


def calibrate(p: OracleProfile, nthreads: int = 8, n: int = 200) -> tuple[float, float, float]:
    """(mu_msv, mu_vit, tau) in bits from oracle scores of i.i.d. background
    sequences: n of length 200 for the filters, n of length 100 for Forward;
    tau puts a tail mass of 0.04 at the (0.04 n)-th largest Forward score
    (the 8th at n = 200)."""
    from synth import gen
    db = gen.random_sequences(gen.SEED_CALIB_VIT, n, 200)
    r = search(p, db.residues, db.offsets, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0), nthreads)
    mu_msv = gumbel_mu([msv_bits(int(v), 200) for v in r["msv"]])
    mu_vit = gumbel_mu([vit_bits(int(v), 200) for v in r["vit"]])
    dbf = gen.random_sequences(gen.SEED_CALIB_FWD, n, 100)
    rf = search(p, dbf.residues, dbf.offsets, (0.0, 0.0, 0.0), (1.0, 1.0, 1.0), nthreads)
    tau = exp_tail_location([fwd_bits(float(v), 100) for v in rf["fwd"]])
    return mu_msv, mu_vit, tau


def bias(p: OracleProfile, x) -> float:
    """Composition-bias score (nats) of one target (see orc_bias)."""
    x = _seq(x)
    return float(p.lib.orc_bias(p.h, _ptr(x), x.size))


def search(p: OracleProfile, residues, offsets, calib, F, nthreads: int = 8,
           fwd_scaled: bool = False, bias_filter: bool = False) -> dict:
    """Filter pipeline over a whole database, caller order (with the
    composition-bias filter between MSV and Viterbi when bias_filter)."""
    res = np.ascontiguousarray(residues, np.uint8)
    off = np.ascontiguousarray(offsets, np.int64)
    n = off.size - 1
    out = dict(msv=np.zeros(n, np.int16), vit=np.zeros(n, np.int32),
               fwd=np.zeros(n, np.float64), flags=np.zeros(n, np.uint8),
               beta=np.zeros(n, np.float64), stage_s=np.zeros(3, np.float64))
    c = np.asarray(calib, np.float64)
    f = np.asarray(F, np.float64)
    rc = p.lib.orc_search_bias(p.h, _ptr(res if res.size else np.zeros(1, np.uint8)), _ptr(off),
                               n, _ptr(c), _ptr(f), int(nthreads), int(fwd_scaled), int(bias_filter),
                               _ptr(out["msv"]), _ptr(out["vit"]), _ptr(out["fwd"]),
                               _ptr(out["flags"]), _ptr(out["beta"]), _ptr(out["stage_s"]))
    if rc != 0:
        raise ValueError("oracle search rejected its input")
    return out


# ------------------------------------------------------------ posterior decoding

RT1 = 0.25      # a region needs one residue with core posterior >= RT1 ...
RT2 = 0.10      # ... and extends over the run of residues with core posterior >= RT2


def decode(p: OracleProfile, x) -> dict:
    """Forward/Backward posterior decoding of one target (fp64 log space).

    tot = (Forward total, Backward total) in nats; per residue i (0-based
    here, residue i+1 of the model's notation): core = P(emitted by a match
    or insert state), njc[:, 0..2] = P(emitted by N, J, C), beg = P(B at row
    i) (a domain starts at residue i+1), end = P(E at row i+1) (a domain ends
    at residue i+1); pM, pI [L, M]: P(M_k / I_k emits residue i+1)."""
    x = _seq(x)
    L, M = x.size, p.M
    out = dict(tot=np.zeros(2), core=np.zeros(L), njc=np.zeros((L, 3)), beg=np.zeros(L),
               end=np.zeros(L), pM=np.zeros((L, M)), pI=np.zeros((L, M)))
    rc = p.lib.orc_decode(p.h, _ptr(x), L, _ptr(out["tot"]), _ptr(out["core"]), _ptr(out["njc"]),
                          _ptr(out["beg"]), _ptr(out["end"]), _ptr(out["pM"]), _ptr(out["pI"]))
    if rc != 0:
        raise MemoryError("oracle decode failed")
    return out


def regions(core, rt1: float = RT1, rt2: float = RT2, library=None) -> list:
    """Domain regions: 1-based inclusive residue ranges (s, e)."""
    c = np.ascontiguousarray(core, np.float64)
    cap = max(1, c.size)
    se = np.zeros(2 * cap, np.int32)
    n = (lib() if library is None else library).orc_regions(_ptr(c), c.size, rt1, rt2, _ptr(se), cap)
    return [(int(se[2 * r]), int(se[2 * r + 1])) for r in range(n)]


def oa_align(p: OracleProfile, dec: dict, s: int, e: int) -> dict:
    """Optimal-accuracy alignment of region [s, e] (1-based, inclusive)."""
    L = dec["core"].size
    code = np.zeros(e - s + 1, np.int16)
    abk = np.zeros(4, np.int32)
    sc = p.lib.orc_oa_align(p.h, L, _ptr(dec["core"]), _ptr(dec["pM"]), _ptr(dec["pI"]), s, e,
                            _ptr(code), _ptr(abk))
    return dict(score=float(sc), code=code, a=int(abk[0]), b=int(abk[1]), k1=int(abk[2]), k2=int(abk[3]))


def oa_path_score(p: OracleProfile, dec: dict, s: int, e: int, code) -> tuple[float, bool]:
    """(objective value, validity) of a given alignment of region [s, e]."""
    L = dec["core"].size
    c = np.ascontiguousarray(code, np.int16)
    assert c.size == e - s + 1
    valid = C.c_int(0)
    sc = p.lib.orc_oa_path_score(p.h, L, _ptr(dec["core"]), _ptr(dec["pM"]), _ptr(dec["pI"]), s, e,
                                 _ptr(c), C.byref(valid))
    return float(sc), bool(valid.value)


def domains(p: OracleProfile, x, rt1: float = RT1, rt2: float = RT2) -> tuple[dict, list]:
    """Posterior decoding, regions and one optimal-accuracy alignment per
    region.  Each domain: s, e (region), a, b (aligned residues), k1, k2
    (model nodes), score (objective), nexp (expected domain ends in the
    region), code (per residue of the region: +k M_k, -k I_k, 0 unaligned)."""
    dec = decode(p, x)
    out = []
    for s, e in regions(dec["core"], rt1, rt2, p.lib):
        d = oa_align(p, dec, s, e)
        d.update(s=s, e=e, nexp=float(dec["end"][s - 1:e].sum()))
        out.append(d)
    return dec, out


# ------------------------------------------------------------ iteration: profile from hits

def count_alignment(M: int, x, s: int, code) -> dict:
    """Emission and transition counts of one region's alignment (codes as
    oa_align: +k M_k, -k I_k, 0 not aligned; residue s + j has code[j]).

    match[k-1][a]: residues a on M_k; insert[k-1][a]: on I_k; trans[k-1][t]
    (MM MI MD IM II DM DD out of node k): the transitions between
    consecutive states of the path, where M_k -> M_k' with k' > k + 1 passes
    through D_{k+1} .. D_{k'-1} (MD_k, DD_{k+1} .. DD_{k'-2}, DM_{k'-1})."""
    match = np.zeros((M, 20), np.int64)
    insert = np.zeros((max(M - 1, 0), 20), np.int64)
    trans = np.zeros((max(M - 1, 0), 7), np.int64)
    code = [int(c) for c in code]
    MM, MI, MD, IM, II, DM, DD = range(7)
    prev = None
    for j, c in enumerate(code):
        if c == 0:
            continue
        a = int(x[s - 1 + j])
        if c > 0:
            match[c - 1, a] += 1
        else:
            insert[-c - 1, a] += 1
        if prev is not None:
            if prev > 0 and c > 0:           # M_k -> M_k'
                k, k2 = prev, c
                if k2 == k + 1:
                    trans[k - 1, MM] += 1
                else:
                    trans[k - 1, MD] += 1
                    for kk in range(k + 1, k2 - 1):
                        trans[kk - 1, DD] += 1
                    trans[k2 - 2, DM] += 1
            elif prev > 0:                   # M_k -> I_k
                trans[prev - 1, MI] += 1
            elif c < 0:                      # I_k -> I_k
                trans[-c - 1, II] += 1
            else:                            # I_k -> M_{k+1}
                trans[-prev - 1, IM] += 1
        prev = c
    return dict(match=match, insert=insert, trans=trans)


def rebuild_profile(prof, counts: dict, A: float, B: float):
    """The next iteration's profile: the counts of the accepted hits'
    alignments with the previous profile as a Dirichlet prior (fp64):
       e'_k(a) = (c_k(a) + A e_k(a)) / (sum_b c_k(b) + A)    (match and insert rows)
       t'_k    = (n_k + B t_k) / (sum over the group n + B)   (groups MM MI MD | IM II | DM DD)"""
    from synth import Profile
    M = prof.M

    def rows(c, p, w):
        c = np.asarray(c, np.float64)
        return (c + w * p) / (c.sum(axis=1, keepdims=True) + w)

    match = rows(counts["match"], prof.match, A)
    insert = rows(counts["insert"], prof.insert, A) if M > 1 else prof.insert.copy()
    trans = np.zeros_like(prof.trans)
    n = np.asarray(counts["trans"], np.float64)
    for g in ((0, 3), (3, 5), (5, 7)):
        trans[:, g[0]:g[1]] = rows(n[:, g[0]:g[1]], prof.trans[:, g[0]:g[1]], B)
    return Profile(M, prof.bg.copy(), match, insert, trans)
