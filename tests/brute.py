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
