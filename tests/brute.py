"""Brute-force enumeration of every Plan7 state path (tiny M and L).

Written from the model's grammar, not from any dynamic-programming
recurrence: a path is S->N, N emits any prefix (N->N loops), N->B, B->M_k,
a core walk (M_k->M_{k+1} | I_k | D_{k+1} | E; I_k->I_k | M_{k+1};
D_k->M_{k+1} | D_{k+1} | E), E->J (J emits, J->B, another core walk) or
E->C (C emits the rest, C->T).  The score of a path is the sum of its
transition and emission scores.  Viterbi is the maximum over paths,
Forward the log of the sum of exp(score).

The MSV filter's parse space is enumerated separately: ordered,
row-disjoint ungapped diagonal segments.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Callable


@dataclass
class Scores:
    """Score system for the enumerator (floats or ints).

    msc(k, a), isc(k, a): emission of residue a by M_k / I_k (k 1-based);
    t(k, name): transition out of node k, name in MM MI MD IM II DM DD;
    entry: B->M_k; loop: N->N, J->J, C->C; move: N->B, J->B, C->T;
    ej, ec: E->J, E->C.  Exits M_k->E and D_k->E score 0."""
    M: int
    msc: Callable[[int, int], float]
    isc: Callable[[int, int], float]
    t: Callable[[int, str], float]
    entry: float
    loop: float
    move: float
    ej: float
    ec: float


def all_path_scores(S: Scores, x) -> list:
    L = len(x)
    M = S.M
    out = []

    def at_N(i, s):
        if i < L:
            at_N(i + 1, s + S.loop)
        at_B(i, s + S.move)

    def at_B(i, s):
        if i < L:
            for k in range(1, M + 1):
                at_M(k, i + 1, s + S.entry + S.msc(k, x[i]))

    def at_M(k, i, s):            # M_k has just emitted residue i (1-based)
        at_E(i, s)
        if k < M:
            if i < L:
                at_M(k + 1, i + 1, s + S.t(k, "MM") + S.msc(k + 1, x[i]))
                at_I(k, i + 1, s + S.t(k, "MI") + S.isc(k, x[i]))
            at_D(k + 1, i, s + S.t(k, "MD"))

    def at_I(k, i, s):
        if i < L:
            at_I(k, i + 1, s + S.t(k, "II") + S.isc(k, x[i]))
            at_M(k + 1, i + 1, s + S.t(k, "IM") + S.msc(k + 1, x[i]))

    def at_D(k, i, s):
        at_E(i, s)
        if k < M:
            if i < L:
                at_M(k + 1, i + 1, s + S.t(k, "DM") + S.msc(k + 1, x[i]))
            at_D(k + 1, i, s + S.t(k, "DD"))

    def at_E(i, s):
        at_J(i, s + S.ej)
        at_C(i, s + S.ec)

    def at_J(i, s):
        if i < L:
            at_J(i + 1, s + S.loop)
        at_B(i, s + S.move)

    def at_C(i, s):
        if i < L:
            at_C(i + 1, s + S.loop)
        else:
            out.append(s + S.move)

    at_N(0, 0)
    return out


def viterbi(S: Scores, x):
    return max(all_path_scores(S, x))


def forward(S: Scores, x) -> float:
    sc = all_path_scores(S, x)
    m = max(sc)
    return m + math.log(sum(math.exp(v - m) for v in sc))


_TNAMES = ("MM", "MI", "MD", "IM", "II", "DM", "DD")


def float_scores(prof, L: int) -> Scores:
    """Natural-log score system of a probability profile (synth.Profile)."""
    M = prof.M

    def lg(v):
        return math.log(v) if v > 0 else -math.inf

    return Scores(
        M=M,
        msc=lambda k, a: math.log(prof.match[k - 1, a] / prof.bg[a]),
        isc=lambda k, a: math.log(prof.insert[k - 1, a] / prof.bg[a]),
        t=lambda k, n: lg(prof.trans[k - 1, _TNAMES.index(n)]),
        entry=math.log(2.0 / (M * (M + 1.0))),
        loop=math.log(L / (L + 3.0)),
        move=math.log(3.0 / (L + 3.0)),
        ej=math.log(0.5), ec=math.log(0.5))


def int_scores(tab: dict, M: int, entry16: int, move16: int, ej16: int) -> Scores:
    """Integer score system of the Viterbi filter (loops score 0)."""
    msc16, isc16, t16 = tab["msc16"], tab["isc16"], tab["t16"]
    return Scores(
        M=M,
        msc=lambda k, a: int(msc16[k - 1, a]),
        isc=lambda k, a: int(isc16[k - 1, a]),
        t=lambda k, n: int(t16[k - 1, _TNAMES.index(n)]),
        entry=entry16, loop=0, move=move16, ej=ej16, ec=ej16)


def msv_parses(sc8, x, M: int, base8: int, move8: int, entry8: int, exit8: int) -> int:
    """Best MSV parse score: the max over ordered sets of row-disjoint
    ungapped segments (each a diagonal run of nodes within 1..M) of
       BASE8 - MOVE8 + sum_seg (-ENTRY8 + sum sc8 - EXIT8) - n_seg*MOVE8,
    or 0 when no parse scores above 0.  sc8(k, a) is the node's integer
    score (k 1-based).  Exponential: tiny cases only."""
    L = len(x)
    segs = []
    for i in range(L):
        for k in range(1, M + 1):
            s = 0
            for ln in range(1, min(L - i, M - k + 1) + 1):
                s += sc8(k + ln - 1, x[i + ln - 1])
                segs.append((i, i + ln, s))        # rows [i, i+ln)
    best = 0
    segs.sort()

    def extend(row_free, acc):
        nonlocal best
        for (r0, r1, s) in segs:
            if r0 < row_free:
                continue
            v = acc - entry8 + s - exit8
            best = max(best, v - move8)
            extend(r1, v - move8)
    extend(0, base8 - move8)
    return best


# ------------------------------------------------------------ annotated paths

def all_paths(S: Scores, x) -> list:
    """Every Plan7 path as (score, emit, begins, ends): emit[i] names the
    state that emitted residue i+1 (("M", k), ("I", k), ("N",), ("J",),
    ("C",)); begins / ends are the rows at which the path visits B / E.
    Written from the same grammar as all_path_scores, with bookkeeping."""
    L = len(x)
    M = S.M
    out = []

    def at_N(i, s, em, bg, en):
        if i < L:
            at_N(i + 1, s + S.loop, em + (("N",),), bg, en)
        at_B(i, s + S.move, em, bg, en)

    def at_B(i, s, em, bg, en):
        if i < L:
            for k in range(1, M + 1):
                at_M(k, i + 1, s + S.entry + S.msc(k, x[i]), em + (("M", k),), bg + (i,), en)

    def at_M(k, i, s, em, bg, en):
        at_E(i, s, em, bg, en)
        if k < M:
            if i < L:
                at_M(k + 1, i + 1, s + S.t(k, "MM") + S.msc(k + 1, x[i]), em + (("M", k + 1),), bg, en)
                at_I(k, i + 1, s + S.t(k, "MI") + S.isc(k, x[i]), em + (("I", k),), bg, en)
            at_D(k + 1, i, s + S.t(k, "MD"), em, bg, en)

    def at_I(k, i, s, em, bg, en):
        if i < L:
            at_I(k, i + 1, s + S.t(k, "II") + S.isc(k, x[i]), em + (("I", k),), bg, en)
            at_M(k + 1, i + 1, s + S.t(k, "IM") + S.msc(k + 1, x[i]), em + (("M", k + 1),), bg, en)

    def at_D(k, i, s, em, bg, en):
        at_E(i, s, em, bg, en)
        if k < M:
            if i < L:
                at_M(k + 1, i + 1, s + S.t(k, "DM") + S.msc(k + 1, x[i]), em + (("M", k + 1),), bg, en)
            at_D(k + 1, i, s + S.t(k, "DD"), em, bg, en)

    def at_E(i, s, em, bg, en):
        at_J(i, s + S.ej, em, bg, en + (i,))
        at_C(i, s + S.ec, em, bg, en + (i,))

    def at_J(i, s, em, bg, en):
        if i < L:
            at_J(i + 1, s + S.loop, em + (("J",),), bg, en)
        at_B(i, s + S.move, em, bg, en)

    def at_C(i, s, em, bg, en):
        if i < L:
            at_C(i + 1, s + S.loop, em + (("C",),), bg, en)
        else:
            out.append((s + S.move, em, bg, en))

    at_N(0, 0, (), (), ())
    return out


def posteriors(S: Scores, x) -> dict:
    """Posterior probabilities by weighting every path with exp(score):
    core / njc / pM / pI per residue, beg[i] = P(B at row i), i = 0..L-1,
    end[i] = P(E at row i+1)."""
    L, M = len(x), S.M
    paths = all_paths(S, x)
    top = max(p[0] for p in paths)
    w = [math.exp(p[0] - top) for p in paths]
    Z = sum(w)
    out = dict(core=[0.0] * L, njc=[[0.0] * 3 for _ in range(L)], beg=[0.0] * L, end=[0.0] * L,
               pM=[[0.0] * M for _ in range(L)], pI=[[0.0] * M for _ in range(L)],
               tot=top + math.log(Z))
    for (sc, em, bg, en), wi in zip(paths, w):
        f = wi / Z
        for i, st in enumerate(em):
            if st[0] == "M":
                out["pM"][i][st[1] - 1] += f
                out["core"][i] += f
            elif st[0] == "I":
                out["pI"][i][st[1] - 1] += f
                out["core"][i] += f
            else:
                out["njc"][i]["NJC".index(st[0])] += f
        for r in bg:
            out["beg"][r] += f
        for r in en:
            out["end"][r - 1] += f
    return out


def oa_best(M: int, allowed, core, pM, pI, s: int, e: int) -> float:
    """Best value of the optimal-accuracy objective over every alignment of
    region [s, e] (1-based), enumerated: a contiguous aligned range [a, b],
    a core walk that starts in M_k1 at residue a and ends in M_k2 at residue
    b, moving M->M (next node, next residue), M->I / I->I (same node, next
    residue), I->M (next node, next residue) or M->D..D->M (skipping nodes,
    next residue), using only allowed(k, name) transitions.  Residues of the
    region outside [a, b] earn 1 - core."""
    best = -math.inf
    flank = [1.0 - core[i - 1] for i in range(1, len(core) + 1)]

    def walk(state, k, i, b, acc):
        # state emitted residue i; acc includes it
        nonlocal best
        if i == b:
            if state == "M":
                best = max(best, acc + sum(flank[j - 1] for j in range(b + 1, e + 1)))
            return
        if state == "M":
            if k < M and allowed(k, "MM"):
                walk("M", k + 1, i + 1, b, acc + pM[i][k])
            if k < M and allowed(k, "MI"):
                walk("I", k, i + 1, b, acc + pI[i][k - 1])
            if k < M and allowed(k, "MD"):
                j = k + 1                      # in D_j
                while j < M:
                    if allowed(j, "DM"):
                        walk("M", j + 1, i + 1, b, acc + pM[i][j])
                    if not allowed(j, "DD"):
                        break
                    j += 1
        else:
            if allowed(k, "II"):
                walk("I", k, i + 1, b, acc + pI[i][k - 1])
            if allowed(k, "IM"):
                walk("M", k + 1, i + 1, b, acc + pM[i][k])

    for a in range(s, e + 1):
        pre = sum(flank[j - 1] for j in range(s, a))
        for b in range(a, e + 1):
            for k1 in range(1, M + 1):
                walk("M", k1, a, b, pre + pM[a - 1][k1 - 1])
    return best
