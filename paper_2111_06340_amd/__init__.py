"""MI355X (gfx950) Plan7 profile-HMM database search: Python binding.

A thin ctypes layer over libhmmgpu.so with the same entry points as the C
ABI in include/hmmgpu.h (hmm_profile_upload, hmm_db_upload, hmm_search, ...).
It only marshals arguments: every step of the search runs in the library's
HIP kernels.  PyTorch provides device memory for the outputs and the stream.

The library is built in-tree by paper_2111_06340_amd.build; importing this
module fails loudly when it is missing.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

from .build import LIB as _LIB_PATH

HMM_OK, HMM_EINVAL, HMM_ERANGE, HMM_ENOMEM, HMM_EDEVICE = 0, -1, -2, -3, -4
HMM_K = 20
HMM_MAX_M = 3072
HMM_MAX_LEN = 100000
HMM_MSV_PASS, HMM_MSV_OVF, HMM_VIT_RAN, HMM_VIT_PASS, HMM_VIT_OVF, HMM_FWD_RAN, HMM_FWD_PASS, HMM_BIAS_PASS = (
    0x01, 0x02, 0x04, 0x08, 0x10, 0x20, 0x40, 0x80)

HMM_RT1, HMM_RT2 = 0.25, 0.10   # region thresholds on the core posterior (float32 in the library)

EXPORTED = ("hmm_db_free", "hmm_db_info", "hmm_db_stage_times", "hmm_db_stage_timing", "hmm_db_upload",
            "hmm_count", "hmm_db_fused_tail", "hmm_db_pipeline", "hmm_db_share", "hmm_debug_length_params",
            "hmm_debug_tables",
            "hmm_decode", "hmm_decode_static", "hmm_last_error", "hmm_profile_free", "hmm_rebuild",
            "hmm_probe_pk16", "hmm_profile_upload", "hmm_search", "hmm_search_group", "hmm_strerror")


class HmmError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where} failed ({status}): {detail}")
        self.status = status


class hmm_profile_desc(C.Structure):
    _fields_ = [("M", C.c_int32), ("bg", C.c_void_p), ("match", C.c_void_p), ("insert", C.c_void_p),
                ("trans", C.c_void_p), ("mu_msv", C.c_double), ("mu_vit", C.c_double), ("tau", C.c_double)]


class hmm_thresholds(C.Structure):
    _fields_ = [("F1", C.c_double), ("F2", C.c_double), ("F3", C.c_double), ("bias_filter", C.c_int32)]


class hmm_results(C.Structure):
    _fields_ = [("msv", C.c_void_p), ("vit", C.c_void_p), ("fwd", C.c_void_p), ("flags", C.c_void_p),
                ("counts", C.c_void_p), ("bias", C.c_void_p)]


class hmm_decode_out(C.Structure):
    _fields_ = [("dom", C.c_void_p), ("max_dom", C.c_int32), ("n_dom", C.c_void_p), ("exp_dom", C.c_void_p),
                ("pp", C.c_void_p), ("aln", C.c_void_p)]


# hmm_domain: 9 x 4 bytes (target, s, e, a, b, k1, k2 as int32; score, nexp as float32)
DOMAIN_FIELDS = ("target", "s", "e", "a", "b", "k1", "k2", "score", "nexp")

_lib = None


def lib():
    """Load libhmmgpu.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise ImportError(f"{_LIB_PATH} is missing: run `python -m paper_2111_06340_amd.build` "
                              "(the search has no CPU fallback)")
        L = C.CDLL(_LIB_PATH)
        vp, i32, i64 = C.c_void_p, C.c_int32, C.c_int64
        L.hmm_profile_upload.restype = C.c_int
        L.hmm_profile_upload.argtypes = [C.POINTER(hmm_profile_desc), vp, C.POINTER(vp)]
        L.hmm_profile_free.restype = C.c_int
        L.hmm_profile_free.argtypes = [vp]
        L.hmm_db_upload.restype = C.c_int
        L.hmm_db_upload.argtypes = [vp, vp, i64, vp, C.POINTER(vp)]
        L.hmm_db_free.restype = C.c_int
        L.hmm_db_free.argtypes = [vp]
        L.hmm_db_pipeline.restype = C.c_int
        L.hmm_db_pipeline.argtypes = [vp, i32, C.POINTER(i32)]
        L.hmm_db_fused_tail.restype = C.c_int
        L.hmm_db_fused_tail.argtypes = [vp, i32, C.POINTER(i32)]
        L.hmm_db_share.restype = C.c_int
        L.hmm_db_share.argtypes = [vp, C.POINTER(vp)]
        L.hmm_search.restype = C.c_int
        L.hmm_search.argtypes = [vp, vp, C.POINTER(hmm_thresholds), C.POINTER(hmm_results), vp]
        L.hmm_probe_pk16.restype = C.c_int
        L.hmm_probe_pk16.argtypes = [vp, C.POINTER(C.c_double), C.POINTER(C.c_float)]
        L.hmm_search_group.restype = C.c_int
        L.hmm_search_group.argtypes = [vp, vp, C.POINTER(hmm_thresholds), C.POINTER(hmm_results), i32, vp]
        L.hmm_count.restype = C.c_int
        L.hmm_count.argtypes = [vp, vp, vp, vp, i32, vp, vp, vp]
        L.hmm_rebuild.restype = C.c_int
        L.hmm_rebuild.argtypes = [C.POINTER(hmm_profile_desc), vp, C.c_double, C.c_double, vp, vp, vp]
        L.hmm_decode.restype = C.c_int
        L.hmm_decode.argtypes = [vp, vp, vp, C.c_uint8, C.POINTER(hmm_decode_out), vp]
        L.hmm_decode_static.restype = C.c_int
        L.hmm_decode_static.argtypes = [vp, vp, vp, C.c_uint8, C.POINTER(hmm_decode_out), vp]
        L.hmm_db_info.restype = C.c_int
        L.hmm_db_info.argtypes = [vp, C.POINTER(i64), C.POINTER(i64), C.POINTER(i32)]
        L.hmm_db_stage_timing.restype = C.c_int
        L.hmm_db_stage_timing.argtypes = [vp, i32]
        L.hmm_db_stage_times.restype = C.c_int
        L.hmm_db_stage_times.argtypes = [vp, vp, i32, C.POINTER(i32)]
        L.hmm_strerror.restype = C.c_char_p
        L.hmm_strerror.argtypes = [C.c_int]
        L.hmm_last_error.restype = C.c_char_p
        L.hmm_last_error.argtypes = []
        L.hmm_debug_tables.restype = C.c_int
        L.hmm_debug_tables.argtypes = [C.POINTER(hmm_profile_desc), vp, vp, vp, vp, vp]
        L.hmm_debug_length_params.restype = C.c_int
        L.hmm_debug_length_params.argtypes = [C.POINTER(hmm_profile_desc), C.POINTER(hmm_thresholds), i32, vp, vp]
        _lib = L
    return _lib


def _check(rc: int, where: str):
    if rc != HMM_OK:
        raise HmmError(rc, where, lib().hmm_last_error().decode())


def _ptr(a: np.ndarray) -> C.c_void_p:
    return C.c_void_p(a.ctypes.data) if a is not None and a.size else C.c_void_p(0)


def _stream_handle(stream) -> C.c_void_p:
    if stream is None:
        return C.c_void_p(0)
    if isinstance(stream, int):
        return C.c_void_p(stream)
    return C.c_void_p(stream.cuda_stream)


def hmm_strerror(status: int) -> str:
    return lib().hmm_strerror(status).decode()


def hmm_last_error() -> str:
    return lib().hmm_last_error().decode()


def hmm_profile_upload(M: int, bg, match, insert, trans, mu_msv: float, mu_vit: float, tau: float,
                       stream=None) -> int:
    """Quantise and upload a probability profile; returns the handle."""
    arrs = [np.ascontiguousarray(a, dtype=np.float64) if a is not None else None
            for a in (bg, match, insert, trans)]
    d = hmm_profile_desc(int(M), _ptr(arrs[0]).value, _ptr(arrs[1]).value,
                         _ptr(arrs[2]).value if arrs[2] is not None else None,
                         _ptr(arrs[3]).value if arrs[3] is not None else None,
                         float(mu_msv), float(mu_vit), float(tau))
    h = C.c_void_p(0)
    _check(lib().hmm_profile_upload(C.byref(d), _stream_handle(stream), C.byref(h)), "hmm_profile_upload")
    return h.value


def hmm_profile_free(handle: int) -> None:
    _check(lib().hmm_profile_free(C.c_void_p(handle)), "hmm_profile_free")


def hmm_db_upload(residues, offsets, stream=None) -> int:
    """Pack and upload a sequence database; returns the handle."""
    res = np.ascontiguousarray(residues, dtype=np.uint8)
    off = np.ascontiguousarray(offsets, dtype=np.int64)
    h = C.c_void_p(0)
    _check(lib().hmm_db_upload(_ptr(res), _ptr(off), int(off.size - 1), _stream_handle(stream), C.byref(h)),
           "hmm_db_upload")
    return h.value


def hmm_db_free(handle: int) -> None:
    _check(lib().hmm_db_free(C.c_void_p(handle)), "hmm_db_free")


def hmm_db_pipeline(handle: int, chunks: int = 0) -> int:
    """Set (chunks > 0) and return the number of pipelined chunks of a search."""
    cur = C.c_int32(0)
    _check(lib().hmm_db_pipeline(C.c_void_p(handle), int(chunks), C.byref(cur)), "hmm_db_pipeline")
    return cur.value


def hmm_db_fused_tail(handle: int, mode: int = 0) -> int:
    """Set (mode 1 staged, 2 fused, 3 fused when F2 = 1) and return how the stages after MSV run."""
    cur = C.c_int32(0)
    _check(lib().hmm_db_fused_tail(C.c_void_p(handle), int(mode), C.byref(cur)), "hmm_db_fused_tail")
    return cur.value


def hmm_db_share(handle: int) -> int:
    """A second handle on the same packed database, with its own scratch."""
    h = C.c_void_p(0)
    _check(lib().hmm_db_share(C.c_void_p(handle), C.byref(h)), "hmm_db_share")
    return h.value


def hmm_db_info(handle: int) -> tuple[int, int, int]:
    n, r, m = C.c_int64(), C.c_int64(), C.c_int32()
    _check(lib().hmm_db_info(C.c_void_p(handle), C.byref(n), C.byref(r), C.byref(m)), "hmm_db_info")
    return n.value, r.value, m.value


def hmm_db_stage_timing(handle: int, capacity: int) -> None:
    _check(lib().hmm_db_stage_timing(C.c_void_p(handle), int(capacity)), "hmm_db_stage_timing")


def hmm_db_stage_times(handle: int, cap: int) -> np.ndarray:
    """[n, 4] stage durations (ms): MSV, Viterbi, rescore, Forward."""
    out = np.zeros((max(cap, 1), 4), np.float32)
    n = C.c_int32(0)
    _check(lib().hmm_db_stage_times(C.c_void_p(handle), _ptr(out), int(cap), C.byref(n)), "hmm_db_stage_times")
    return out[:n.value]


def hmm_search(profile: int, db: int, F, out: dict, stream=None, bias_filter: bool = False) -> None:
    """Enqueue a search.  `out` maps msv/vit/fwd/flags (and optionally
    counts, bias) to device tensors of int16/int32/float32/uint8 (int64[4],
    float32)."""
    t = hmm_thresholds(*[float(v) for v in F[:3]], int(bool(bias_filter)))
    r = hmm_results(out["msv"].data_ptr(), out["vit"].data_ptr(), out["fwd"].data_ptr(),
                    out["flags"].data_ptr(), out["counts"].data_ptr() if out.get("counts") is not None else None,
                    out["bias"].data_ptr() if out.get("bias") is not None else None)
    _check(lib().hmm_search(C.c_void_p(profile), C.c_void_p(db), C.byref(t), C.byref(r), _stream_handle(stream)),
           "hmm_search")


def hmm_probe_pk16(stream=None) -> tuple[float, float]:
    """The packed 16-bit VALU rate the device sustains (element-ops/s) and
    the timed launch's milliseconds."""
    ops = C.c_double(0.0)
    ms = C.c_float(0.0)
    _check(lib().hmm_probe_pk16(_stream_handle(stream), C.byref(ops), C.byref(ms)), "hmm_probe_pk16")
    return ops.value, ms.value


def _results(out: dict) -> hmm_results:
    return hmm_results(out["msv"].data_ptr(), out["vit"].data_ptr(), out["fwd"].data_ptr(),
                       out["flags"].data_ptr(), out["counts"].data_ptr() if out.get("counts") is not None else None,
                       out["bias"].data_ptr() if out.get("bias") is not None else None)


def hmm_search_group(profiles, dbs, Fs, outs, stream=None, bias_filter=False) -> None:
    """Enqueue a group of searches: search i is profiles[i] against handle
    dbs[i] (distinct handles of one database) with cutoffs Fs[i] into
    outs[i] (dicts as in hmm_search); bias_filter: one flag or one per
    search."""
    n = len(profiles)
    bf = list(bias_filter) if isinstance(bias_filter, (list, tuple)) else [bias_filter] * n
    if not (len(dbs) == len(Fs) == len(outs) == len(bf) == n):
        raise ValueError("profiles, dbs, Fs, outs (and bias_filter) must have one entry per search")
    P = (C.c_void_p * max(n, 1))(*[C.c_void_p(h) for h in profiles])
    D = (C.c_void_p * max(n, 1))(*[C.c_void_p(h) for h in dbs])
    T = (hmm_thresholds * max(n, 1))(*[hmm_thresholds(*[float(v) for v in F[:3]], int(bool(b)))
                                       for F, b in zip(Fs, bf)])
    R = (hmm_results * max(n, 1))(*[_results(o) for o in outs])
    _check(lib().hmm_search_group(P, D, T, R, int(n), _stream_handle(stream)), "hmm_search_group")


def _decode_args(flags, out: dict):
    def ptr(k):
        v = out.get(k)
        return v.data_ptr() if v is not None else None
    o = hmm_decode_out(ptr("dom"), int(out["dom"].shape[0]), ptr("n_dom"), ptr("exp_dom"), ptr("pp"), ptr("aln"))
    fp = C.c_void_p(flags.data_ptr()) if flags is not None else C.c_void_p(0)
    return fp, o


def hmm_decode(profile: int, db: int, flags, mask: int, out: dict, stream=None) -> None:
    """Enqueue posterior decoding.  `flags`: device uint8 tensor (caller
    order) or None (decode every target); `out` maps dom (int32 [max_dom, 9])
    and n_dom (int32 [1]) and optionally exp_dom / pp / aln to device
    tensors."""
    fp, o = _decode_args(flags, out)
    _check(lib().hmm_decode(C.c_void_p(profile), C.c_void_p(db), fp, int(mask) & 0xff, C.byref(o),
                            _stream_handle(stream)), "hmm_decode")


def hmm_decode_static(profile: int, db: int, flags, mask: int, out: dict, stream=None) -> None:
    """hmm_decode on the library's fixed device scratch (allocates nothing)."""
    fp, o = _decode_args(flags, out)
    _check(lib().hmm_decode_static(C.c_void_p(profile), C.c_void_p(db), fp, int(mask) & 0xff, C.byref(o),
                                   _stream_handle(stream)), "hmm_decode_static")


def _desc(prof, mu_msv=0.0, mu_vit=0.0, tau=0.0):
    M = int(prof.M)
    keep = [np.ascontiguousarray(a, dtype=np.float64) for a in (prof.bg, prof.match, prof.insert, prof.trans)]
    d = hmm_profile_desc(M, _ptr(keep[0]).value, _ptr(keep[1]).value,
                         _ptr(keep[2]).value if M > 1 else None, _ptr(keep[3]).value if M > 1 else None,
                         float(mu_msv), float(mu_vit), float(tau))
    return d, keep


def hmm_debug_tables(prof) -> dict:
    """Host quantisation of a profile (no GPU): the library's own tables."""
    M = int(prof.M)
    d, keep = _desc(prof)
    sc = np.zeros(8, np.int32)
    cost8 = np.zeros((M, HMM_K), np.uint8)
    msc16 = np.zeros((M, HMM_K), np.int16)
    isc16 = np.zeros((max(M - 1, 1), HMM_K), np.int16)
    t16 = np.zeros((max(M - 1, 1), 7), np.int16)
    _check(lib().hmm_debug_tables(C.byref(d), _ptr(sc), _ptr(cost8), _ptr(msc16), _ptr(isc16), _ptr(t16)),
           "hmm_debug_tables")
    return dict(bias8=int(sc[0]), entry8=int(sc[1]), exit8=int(sc[2]), entry16=int(sc[3]), ej16=int(sc[4]),
                M=int(sc[5]), Q8=int(sc[6]), Q32=int(sc[7]), cost8=cost8, msc16=msc16,
                isc16=isc16[:M - 1], t16=t16[:M - 1])


def hmm_debug_length_params(prof, calib, F, L: int) -> dict:
    """Host per-length parameters (no GPU) for calibration (mu_msv, mu_vit, tau)."""
    d, keep = _desc(prof, *calib)
    i32 = np.zeros(6, np.int32)
    f64 = np.zeros(4, np.float64)
    t = hmm_thresholds(*[float(v) for v in F[:3]], 0)
    _check(lib().hmm_debug_length_params(C.byref(d), C.byref(t), int(L), _ptr(i32), _ptr(f64)),
           "hmm_debug_length_params")
    return dict(move8=int(i32[0]), thr8=int(i32[1]), move16=int(i32[2]), thr16=int(i32[3]),
                loop=float(f64[0]), move=float(f64[1]), null=float(f64[2]), fwd_thr=float(f64[3]))


# ------------------------------------------------------------------ helpers

class Profile:
    """Owning wrapper of a device profile (from a synth.Profile-like object)."""

    def __init__(self, prof, mu_msv: float, mu_vit: float, tau: float, stream=None):
        self.M = int(prof.M)
        self.handle = hmm_profile_upload(self.M, prof.bg, prof.match,
                                         prof.insert if self.M > 1 else None,
                                         prof.trans if self.M > 1 else None,
                                         mu_msv, mu_vit, tau, stream)

    def close(self):
        if getattr(self, "handle", None):
            hmm_profile_free(self.handle)
            self.handle = None

    __del__ = close


class Database:
    """Owning wrapper of a device database."""

    def __init__(self, residues, offsets, stream=None, _share_of=None):
        if _share_of is not None:
            self.handle = hmm_db_share(_share_of.handle)
            self._lengths = _share_of._lengths
        else:
            self.handle = hmm_db_upload(residues, offsets, stream)
            self._lengths = np.diff(np.asarray(offsets, dtype=np.int64))
        self.n, self.n_residues, self.max_len = hmm_db_info(self.handle)

    def share(self) -> "Database":
        """Another handle on the same device database, for concurrent searches."""
        return Database(None, None, _share_of=self)

    def lengths_caller(self):
        """Target lengths in the caller's order (host array)."""
        return self._lengths

    def close(self):
        if getattr(self, "handle", None):
            hmm_db_free(self.handle)
            self.handle = None

    __del__ = close


def alloc_results(n: int, device="cuda"):
    import torch
    return dict(msv=torch.empty(n, dtype=torch.int16, device=device),
                vit=torch.empty(n, dtype=torch.int32, device=device),
                fwd=torch.empty(n, dtype=torch.float32, device=device),
                flags=torch.empty(n, dtype=torch.uint8, device=device),
                counts=torch.zeros(4, dtype=torch.int64, device=device),
                bias=torch.full((n,), float("nan"), dtype=torch.float32, device=device))


def search(profile: Profile, db: Database, F, out: dict | None = None, stream=None,
           bias_filter: bool = False) -> dict:
    """Run one search on the current torch stream (or `stream`); returns the
    device result tensors (valid once the stream synchronises)."""
    import torch
    if out is None:
        out = alloc_results(db.n)
    if stream is None:
        stream = torch.cuda.current_stream()
    hmm_search(profile.handle, db.handle, F, out, stream, bias_filter)
    return out


def search_group(profiles, dbs, F, outs=None, stream=None, bias_filter=False) -> list:
    """Run a group of searches (profiles[i] against dbs[i], distinct
    handles of one database, e.g. a Database and its .share() handles) on
    the current torch stream (or `stream`); F: one cutoff triple or one per
    search.  Returns the device result dicts, in order."""
    import torch
    n = len(profiles)
    Fs = list(F) if F and isinstance(F[0], (list, tuple)) else [F] * n
    if outs is None:
        outs = [alloc_results(d.n) for d in dbs]
    if stream is None:
        stream = torch.cuda.current_stream()
    hmm_search_group([p.handle for p in profiles], [d.handle for d in dbs], Fs, outs, stream, bias_filter)
    return outs


def decode(profile: Profile, db: Database, flags=None, mask: int = HMM_FWD_PASS, max_dom: int | None = None,
           pp: bool = False, aln: bool = False, stream=None, static: bool = False) -> dict:
    """Posterior decoding of the targets whose flags hold `mask` (all targets
    when flags is None) on the current torch stream (or `stream`).  Returns
    device tensors: dom int32 [max_dom, 9] (fields DOMAIN_FIELDS; score and
    nexp are float32 bit patterns), n_dom int32 [1], exp_dom float32 [n]
    (NaN where not decoded), and pp float32 / aln int16 [n_residues] when
    asked for (caller residue layout).  static=True runs hmm_decode_static
    (the library's fixed device scratch; no device allocation)."""
    import torch
    if max_dom is None:
        max_dom = max(16, 4 * db.n)
    dev = "cuda"
    out = dict(dom=torch.zeros((max_dom, 9), dtype=torch.int32, device=dev),
               n_dom=torch.zeros(1, dtype=torch.int32, device=dev),
               exp_dom=torch.full((db.n,), float("nan"), dtype=torch.float32, device=dev))
    if pp:
        out["pp"] = torch.full((db.n_residues,), float("nan"), dtype=torch.float32, device=dev)
    if aln:
        out["aln"] = torch.full((db.n_residues,), -32768, dtype=torch.int16, device=dev)
    if stream is None:
        stream = torch.cuda.current_stream()
    (hmm_decode_static if static else hmm_decode)(profile.handle, db.handle, flags, mask, out, stream)
    return out


def domains_table(out: dict) -> list:
    """Host list of domain dicts from decode()'s outputs (after the stream
    synchronises), sorted by (target, s)."""
    n = int(out["n_dom"].cpu()[0])
    raw = out["dom"][:min(n, out["dom"].shape[0])].cpu().numpy()
    recs = []
    for row in raw:
        d = {k: int(v) for k, v in zip(DOMAIN_FIELDS[:7], row[:7])}
        d["score"] = float(row[7:8].view(np.float32)[0])
        d["nexp"] = float(row[8:9].view(np.float32)[0])
        recs.append(d)
    recs.sort(key=lambda d: (d["target"], d["s"]))
    return recs


def hmm_count(profile: int, db: int, dec: dict, counts, stream=None) -> None:
    """Enqueue the counts of decode()'s alignments into `counts` (device
    uint32 tensor of M*20 + (M-1)*20 + (M-1)*7 entries, added to)."""
    _check(lib().hmm_count(C.c_void_p(profile), C.c_void_p(db), C.c_void_p(dec["dom"].data_ptr()),
                           C.c_void_p(dec["n_dom"].data_ptr()), int(dec["dom"].shape[0]),
                           C.c_void_p(dec["aln"].data_ptr()), C.c_void_p(counts.data_ptr()),
                           _stream_handle(stream)), "hmm_count")


def count_size(M: int) -> int:
    return M * HMM_K + max(M - 1, 0) * HMM_K + max(M - 1, 0) * 7


def hmm_rebuild(prof, counts, A: float, B: float):
    """Host estimate of the next iteration's profile (a synth.Profile-like
    object with the prior's background) from host counts."""
    from types import SimpleNamespace
    M = int(prof.M)
    d, keep = _desc(prof)
    c = np.ascontiguousarray(counts, dtype=np.uint32)
    assert c.size == count_size(M)
    match = np.zeros((M, HMM_K))
    insert = np.zeros((max(M - 1, 1), HMM_K))
    trans = np.zeros((max(M - 1, 1), 7))
    _check(lib().hmm_rebuild(C.byref(d), _ptr(c), float(A), float(B), _ptr(match), _ptr(insert), _ptr(trans)),
           "hmm_rebuild")
    return SimpleNamespace(M=M, bg=np.array(prof.bg, np.float64), match=match, insert=insert[:M - 1],
                           trans=trans[:M - 1])
