"""Ordered certification from revealed prefixes (oracle, stopping behaviour).

Sec. 2.2 transcribed directly.  At access depths d_i the observed items are
S_i(d_i); an Open list can still contribute at most u_i = g_i(d_i + 1) to an
item it has not returned, an Exhausted list 0.  For an observed x,
L(x) = sum over lists that returned x of g_i(r_i(x)) and U(x) = L(x) + sum of
u_i over Open lists that did not return it; every unseen item is bounded by
B = sum_i u_i.  Positions are fixed one at a time: x_dag is the remaining
observed item with the greatest L (ties by id); it is appended when
(L(x_dag), x_dag) precedes (U(y), y) for every other remaining y and
L(x_dag) > B strictly.

A list is Exhausted exactly when its whole complete list has been read.
The request is resolved when q_K = K positions are fixed, or when no unseen
item can score (B = 0) and no remaining observed item can score (U = 0).

Parity: pinned by brute force over every completion of the unread ranks on
tiny inputs, by the identical-lists and reversed-lists closed forms, and by the
controlled-stream outcomes the paper reports (Sec. 4.2).
"""
from __future__ import annotations

from fractions import Fraction
from typing import List, Sequence, Tuple

from .rrf import g


def certify_ref(lists: Sequence[Sequence[int]], weights, k, K: int,
                depths: Sequence[int]) -> Tuple[List[int], bool]:
    """Return (fixed prefix A, resolved?) for complete lists read to ``depths``."""
    ranks = []
    open_ = []
    u = []
    for lst, w, d in zip(lists, weights, depths):
        d = min(d, len(lst))
        ranks.append({int(x): r for r, x in enumerate(lst[:d], start=1)})
        is_open = d < len(lst)
        open_.append(is_open)
        u.append(g(d + 1, w, k) if is_open else Fraction(0))
    B = sum(u, Fraction(0))
    observed = set()
    for rk in ranks:
        observed.update(rk.keys())
    L = {}
    U = {}
    for x in observed:
        lx = Fraction(0)
        ux = Fraction(0)
        for i, rk in enumerate(ranks):
            if x in rk:
                lx += g(rk[x], weights[i], k)
            elif open_[i]:
                ux += u[i]
        L[x] = lx
        U[x] = lx + ux
    A: List[int] = []
    R = set(observed)
    while len(A) < K and R:
        xd = min(R, key=lambda x: (-L[x], x))
        ok = L[xd] > B
        if ok:
            for y in R:
                if y == xd:
                    continue
                if not (L[xd] > U[y] or (L[xd] == U[y] and xd < y)):
                    ok = False
                    break
        if not ok:
            break
        A.append(xd)
        R.discard(xd)
    resolved = len(A) == K or (B == 0 and all(U[y] == 0 for y in R))
    return A, resolved
