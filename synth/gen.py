"""Seeded synthetic workloads for Plan7 profile-HMM database search.

This module draws random inputs only: profile probabilities, sequence
lengths, residues and planted homologs.  It contains none of the scoring
arithmetic (no log-odds, no quantisation, no dynamic programming), so both
the CPU oracle and the GPU library can consume its output without sharing
any of the method.

The paper (ParaFold, Background section) names jackhmmer searches of
UniRef90 and MGnify as the CPU-bound core of AlphaFold's MSA stage and the
medium protein set (Evaluation, Test Cases, Table "bench") spans 77-734
residues.  None of those databases is available here, so every workload is
synthetic, with the shapes below:

* profiles: M match states over the 20 standard amino acids; match and
  insert emission distributions are symmetric Dirichlet(0.5) draws, floored
  as e <- (e + 1e-4) / (1 + 20e-4) so that no probability is zero;
  transitions are the same at every node (M->M .9, M->I .05, M->D .05,
  I->M .6, I->I .4, D->M .5, D->D .5);
* databases: lengths log-normal with median 300 and sigma 0.55 (natural
  log), rounded and clipped; residues i.i.d. from a fixed background;
* planted homologs: a full-length core path sampled from the profile,
  optionally diverged (substitutions plus geometric indels), embedded at a
  uniform offset into background flanks.

Residue codes are 0..19 for the one-letter codes in ALPHABET order.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

ALPHABET = "ACDEFGHIKLMNPQRSTVWY"
K = 20

# Approximate Swiss-Prot composition; frozen here so that every seeded
# workload is reproducible.  Normalised to sum 1 in float64.
_BG_BY_LETTER = {
    "A": 0.0826, "R": 0.0553, "N": 0.0406, "D": 0.0546, "C": 0.0137,
    "Q": 0.0393, "E": 0.0674, "G": 0.0708, "H": 0.0227, "I": 0.0593,
    "L": 0.0965, "K": 0.0582, "M": 0.0241, "F": 0.0386, "P": 0.0472,
    "S": 0.0660, "T": 0.0535, "W": 0.0109, "Y": 0.0292, "V": 0.0687,
}
BACKGROUND = np.array([_BG_BY_LETTER[c] for c in ALPHABET], dtype=np.float64)
BACKGROUND /= BACKGROUND.sum()

# Transition order used everywhere: MM MI MD IM II DM DD.
TRANS_NAMES = ("MM", "MI", "MD", "IM", "II", "DM", "DD")
TRANS_DEFAULT = np.array([0.90, 0.05, 0.05, 0.60, 0.40, 0.50, 0.50])

EMISSION_FLOOR = 1e-4
LEN_MEDIAN = 300.0
LEN_SIGMA = 0.55

SEED_PROFILE = 2111063400
SEED_DB = 2111063500
SEED_C4_PROFILE = 2111063600
SEED_CALIB_VIT = 2111063700
SEED_CALIB_FWD = 2111063701


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


@dataclasses.dataclass
class Profile:
    """Probability-space Plan7 profile (all float64, C-contiguous).

    match[k-1]  = match emission distribution of node k (k = 1..M)
    insert[k-1] = insert emission distribution of node k (k = 1..M-1)
    trans[k-1]  = MM MI MD IM II DM DD out of node k (k = 1..M-1)
    """
    M: int
    bg: np.ndarray
    match: np.ndarray
    insert: np.ndarray
    trans: np.ndarray

    def __post_init__(self):
        self.bg = np.ascontiguousarray(self.bg, dtype=np.float64)
        self.match = np.ascontiguousarray(self.match, dtype=np.float64).reshape(self.M, K)
        self.insert = np.ascontiguousarray(self.insert, dtype=np.float64).reshape(max(self.M - 1, 0), K)
        self.trans = np.ascontiguousarray(self.trans, dtype=np.float64).reshape(max(self.M - 1, 0), 7)


def _floor_emissions(e: np.ndarray) -> np.ndarray:
    return (e + EMISSION_FLOOR) / (1.0 + K * EMISSION_FLOOR)


def make_profile(M: int, seed: int, insert_is_background: bool = False,
                 trans: np.ndarray | None = None) -> Profile:
    """Dirichlet(0.5) match/insert emissions, fixed transitions."""
    if M < 1:
        raise ValueError("M must be >= 1")
    rng = _rng(seed)
    match = _floor_emissions(rng.dirichlet(np.full(K, 0.5), size=M))
    insert = _floor_emissions(rng.dirichlet(np.full(K, 0.5), size=max(M - 1, 0)))
    if insert_is_background:
        insert = np.tile(BACKGROUND, (max(M - 1, 0), 1))
    t = TRANS_DEFAULT if trans is None else np.asarray(trans, dtype=np.float64)
    return Profile(M, BACKGROUND.copy(), match, insert, np.tile(t, (max(M - 1, 0), 1)))


# ---------------------------------------------------------------- residues

class _CategoricalU32:
    """Exact inverse-CDF sampling of a categorical on 32-bit uniforms.

    A 2^16-entry table resolves the code from the top 16 bits; the few
    buckets that straddle a CDF boundary fall back to a full search."""

    def __init__(self, p: np.ndarray):
        p = np.asarray(p, dtype=np.float64)
        cdf = np.cumsum(p / p.sum())
        cdf[-1] = 1.0
        self.edges = np.minimum(np.round(cdf * 2.0**32), 2.0**32).astype(np.uint64)
        lo = np.arange(65536, dtype=np.uint64) << np.uint64(16)
        hi = lo + np.uint64(0xFFFF)
        c_lo = np.searchsorted(self.edges, lo, side="right")
        c_hi = np.searchsorted(self.edges, hi, side="right")
        self.table = np.minimum(c_lo, len(p) - 1).astype(np.uint8)
        self.ambiguous = c_lo != c_hi
        self.n = len(p)

    def draw(self, rng: np.random.Generator, count: int) -> np.ndarray:
        u = rng.integers(0, 2**32, size=count, dtype=np.uint64)
        top = (u >> np.uint64(16)).astype(np.int64)
        out = self.table[top]
        amb = np.nonzero(self.ambiguous[top])[0]
        if amb.size:
            out[amb] = np.minimum(np.searchsorted(self.edges, u[amb], side="right"),
                                  self.n - 1).astype(np.uint8)
        return out


_BG_SAMPLER = _CategoricalU32(BACKGROUND)


def background_residues(rng: np.random.Generator, count: int,
                        chunk: int = 1 << 24) -> np.ndarray:
    out = np.empty(count, dtype=np.uint8)
    for s in range(0, count, chunk):
        e = min(count, s + chunk)
        out[s:e] = _BG_SAMPLER.draw(rng, e - s)
    return out


def sample_lengths(rng: np.random.Generator, n: int, lo: int, hi: int) -> np.ndarray:
    x = rng.lognormal(mean=math.log(LEN_MEDIAN), sigma=LEN_SIGMA, size=n)
    return np.clip(np.rint(x), lo, hi).astype(np.int64)


# ---------------------------------------------------------------- homologs

def sample_homologs(rng: np.random.Generator, prof: Profile, count: int) -> list[np.ndarray]:
    """Full-length core paths B->M_1 ... node M drawn from the profile.

    Each path starts in M_1 and walks node by node: from M_k it goes to
    M_{k+1}, to I_k (an insert run of geometric length, then M_{k+1}) or to
    D_{k+1}; from D_k it goes to M_{k+1} or D_{k+1}.  Match states emit from
    the node's match distribution, inserts from its insert distribution.
    Vectorised over homologs, sequential over nodes."""
    M = prof.M
    if count == 0:
        return []
    msamp = [_CategoricalU32(prof.match[k]) for k in range(M)]
    isamp = [_CategoricalU32(prof.insert[k]) for k in range(M - 1)]
    match_codes = np.full((count, M), 255, dtype=np.uint8)
    ins_counts = np.zeros((count, M), dtype=np.int64)
    ins_chunks = []          # per node: codes in homolog order
    in_d = np.zeros(count, dtype=bool)
    for k in range(M):
        in_m = ~in_d
        codes = msamp[k].draw(rng, count)
        match_codes[in_m, k] = codes[in_m]
        if k == M - 1:
            break
        t = prof.trans[k]
        u = rng.random(count)
        go_i = in_m & (u >= t[0]) & (u < t[0] + t[1])
        go_d_from_m = in_m & (u >= t[0] + t[1])
        go_d_from_d = in_d & (u >= t[5])
        n_ins = np.where(go_i, rng.geometric(1.0 - t[4], size=count), 0)
        ins_counts[:, k] = n_ins
        tot = int(n_ins.sum())
        ins_chunks.append(isamp[k].draw(rng, tot) if tot else np.empty(0, np.uint8))
        in_d = go_d_from_m | go_d_from_d

    present = (match_codes != 255).astype(np.int64)
    seg = (present + ins_counts).ravel()
    starts = np.cumsum(seg) - seg
    total = int(seg.sum())
    out = np.empty(total, dtype=np.uint8)
    pm = present.ravel().astype(bool)
    out[starts[pm]] = match_codes.ravel()[pm]
    if total - int(pm.sum()):
        # insert codes were drawn node-major; reorder to homolog-major
        node_major_idx = []
        for k in range(M - 1):
            h = np.nonzero(ins_counts[:, k])[0]
            node_major_idx.append(np.repeat(h * M + k, ins_counts[h, k]))
        flat_idx = np.concatenate(node_major_idx)
        codes = np.concatenate(ins_chunks)
        order = np.argsort(flat_idx, kind="stable")
        flat_idx = flat_idx[order]
        codes = codes[order]
        grp_first = np.searchsorted(flat_idx, flat_idx, side="left")
        within = np.arange(flat_idx.size) - grp_first
        pos = starts[flat_idx] + present.ravel()[flat_idx] + within
        out[pos] = codes
    per_h = (present + ins_counts).sum(axis=1)
    return np.split(out, np.cumsum(per_h)[:-1])


def diverge(rng: np.random.Generator, seq: np.ndarray, d: float) -> np.ndarray:
    """Substitute each residue with probability d by a background draw; at
    each position, with probability d/10, insert or delete (50/50) a run of
    Geometric(1/3) length."""
    seq = seq.copy()
    sub = rng.random(seq.size) < d
    nsub = int(sub.sum())
    if nsub:
        seq[sub] = background_residues(rng, nsub)
    events = np.nonzero(rng.random(seq.size) < d / 10.0)[0]
    if events.size == 0:
        return seq
    kinds = rng.random(events.size) < 0.5
    runs = rng.geometric(1.0 / 3.0, size=events.size)
    pieces = []
    last = 0
    for pos, is_ins, run in zip(events.tolist(), kinds.tolist(), runs.tolist()):
        if pos < last:
            continue
        pieces.append(seq[last:pos])
        if is_ins:
            pieces.append(background_residues(rng, run))
            last = pos
        else:
            last = pos + run
    pieces.append(seq[last:])
    out = np.concatenate(pieces)
    return out if out.size else seq[:1].copy()


# ---------------------------------------------------------------- databases

@dataclasses.dataclass
class Database:
    residues: np.ndarray   # uint8, codes 0..19, concatenated
    offsets: np.ndarray    # int64[n+1]
    planted: np.ndarray    # int64 ids of planted homologs

    @property
    def n(self) -> int:
        return self.offsets.size - 1

    @property
    def lengths(self) -> np.ndarray:
        return np.diff(self.offsets)

    def seq(self, i: int) -> np.ndarray:
        return self.residues[self.offsets[i]:self.offsets[i + 1]]


def make_database(n: int, seed: int, prof: Profile | None, planted_frac: float,
                  len_lo: int = 30, len_hi: int = 1000,
                  divergence: tuple[float, float] | None = None) -> Database:
    rng = _rng(seed)
    lengths = sample_lengths(rng, n, len_lo, len_hi)
    n_pl = int(round(planted_frac * n)) if prof is not None else 0
    planted = np.sort(rng.choice(n, size=n_pl, replace=False)) if n_pl else np.empty(0, np.int64)
    homs = sample_homologs(rng, prof, n_pl) if n_pl else []
    if divergence is not None:
        lo, hi = divergence
        ds = rng.uniform(lo, hi, size=n_pl)
        homs = [diverge(rng, h, float(d)) for h, d in zip(homs, ds)]
    place = []
    for idx, h in zip(planted.tolist(), homs):
        if h.size <= lengths[idx]:
            lf = int(lengths[idx])
            off = int(rng.integers(0, lf - h.size + 1))
        else:
            lf = min(h.size, len_hi)
            h = h[:lf]
            off = 0
        lengths[idx] = lf
        place.append((idx, off, h))
    offsets = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(lengths, out=offsets[1:])
    residues = background_residues(rng, int(offsets[-1]))
    for idx, off, h in place:
        s = offsets[idx] + off
        residues[s:s + h.size] = h
    return Database(residues, offsets, planted.astype(np.int64))


def random_sequences(seed: int, count: int, length: int) -> Database:
    """i.i.d. background sequences of one length (score calibration)."""
    rng = _rng(seed)
    offsets = np.arange(count + 1, dtype=np.int64) * length
    return Database(background_residues(rng, count * length), offsets, np.empty(0, np.int64))


# ---------------------------------------------------------------- configs

@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    M: int
    n: int
    planted: float
    len_hi: int = 1000
    divergence: tuple[float, float] | None = None
    F: tuple[float, float, float] = (0.02, 1e-3, 1.0)
    index: int = 1


WORKLOADS = {
    "C1": Workload("C1", 77, 5_000, 0.02, F=(1.0, 1.0, 1.0), index=1),
    "C2": Workload("C2", 256, 200_000, 0.01, index=2),
    "C3": Workload("C3", 734, 1_000_000, 0.005, divergence=(0.10, 0.60), index=3),
    "C5": Workload("C5", 2500, 2_000_000, 0.002, len_hi=5000, index=5),
}
C4_PROFILES = 64
C4_M_RANGE = (50, 400)


def workload_profile(w: Workload) -> Profile:
    return make_profile(w.M, SEED_PROFILE + w.index)


def workload_database(w: Workload, n: int | None = None, prof: Profile | None = None,
                      seed_offset: int = 0) -> Database:
    """The workload's DB; n < w.n draws a smaller DB with the same recipe
    (and a different stream of random numbers); seed_offset > 0 draws
    another database of the same recipe (a second database to search)."""
    prof = workload_profile(w) if prof is None else prof
    return make_database(w.n if n is None else n, SEED_DB + w.index + 1000 * seed_offset, prof, w.planted,
                         len_hi=w.len_hi, divergence=w.divergence)


def c4_profiles(count: int = C4_PROFILES) -> list[Profile]:
    out = []
    for p in range(count):
        rng = _rng(SEED_C4_PROFILE + p)
        M = int(rng.integers(C4_M_RANGE[0], C4_M_RANGE[1] + 1))
        out.append(make_profile(M, SEED_C4_PROFILE + 1000 + p))
    return out
