"""Complete-list weighted reciprocal rank fusion (oracle).

Sec. 2.1: F(x) = sum over retrievers i with x in U_i of g_i(r_i(x)), where
g_i(r) = 1 / (r / w_i + k - 1) for w_i > 0 and 0 for w_i = 0 (rank-scaled
weights).  U+ = {x : F(x) > 0}, q_K = min(K, |U+|); the target T*_K is the first
q_K items of U+ in (F descending, id ascending) order, never padded with
zero-score items.

F is compared in exact rational arithmetic (``fractions.Fraction``): k and the
weights are taken as the exact rationals of the values passed in.

Parity: pinned by closed forms (g(1) = 1/k; identical lists give the common
prefix; reversed lists give mirror ties broken by id; a zero weight gives the
other channel's ranking), by the no-padding case, and by brute force over all
items on small inputs (:func:`rrf_topk_exact` against :func:`rrf_topk`).
"""
from __future__ import annotations

from fractions import Fraction
from typing import Dict, List, Sequence

import numpy as np


def g(r: int, w, k) -> Fraction:
    """Contribution of rank r (1-based) of a retriever with weight w."""
    w = Fraction(w)
    k = Fraction(k)
    if w == 0:
        return Fraction(0)
    return 1 / (Fraction(r) / w + k - 1)


def fusion_scores_exact(lists: Sequence[Sequence[int]], weights, k) -> Dict[int, Fraction]:
    """F(x) for every item that appears in some list (exact)."""
    F: Dict[int, Fraction] = {}
    for lst, w in zip(lists, weights):
        for r, x in enumerate(lst, start=1):
            F[int(x)] = F.get(int(x), Fraction(0)) + g(r, w, k)
    return F


def rrf_topk_exact(lists: Sequence[Sequence[int]], weights, k, K: int) -> List[int]:
    """T*_K by scoring every item exactly (small inputs)."""
    F = fusion_scores_exact(lists, weights, k)
    pos = [(f, x) for x, f in F.items() if f > 0]
    pos.sort(key=lambda t: (-t[0], t[1]))
    return [x for _, x in pos[:K]]


def rrf_topk(lists: Sequence[np.ndarray], weights, k, K: int) -> List[int]:
    """T*_K for large complete lists.

    A float64 screen keeps every item whose float64 fusion score reaches the
    K-th largest one within a relative margin of 2^-40 (the float64 value of F
    is within 2^-50 relative of the exact one, so no Top-K item is dropped);
    that set is then ordered exactly by (F descending, id ascending)."""
    if K <= 0:
        return []
    n_items = 1 + max((int(np.max(l)) for l in lists if len(l)), default=-1)
    if n_items == 0:
        return []
    F64 = np.zeros(n_items, dtype=np.float64)
    seen = np.zeros(n_items, dtype=bool)
    kf = float(Fraction(k))
    for lst, w in zip(lists, weights):
        lst = np.asarray(lst, dtype=np.int64)
        seen[lst] = True
        if Fraction(w) == 0 or len(lst) == 0:
            continue
        wf = float(Fraction(w))
        r = np.arange(1, len(lst) + 1, dtype=np.float64)
        F64[lst] += 1.0 / (r / wf + kf - 1.0)
    cand = np.flatnonzero(seen & (F64 > 0))
    if len(cand) == 0:
        return []
    kk = min(K, len(cand))
    t = np.partition(-F64[cand], kk - 1)[kk - 1]        # -(K-th largest)
    keep = cand[-F64[cand] <= t * (1.0 - 2.0 ** -40)]
    keep_set = set(int(x) for x in keep)
    # exact scores of the kept items
    F: Dict[int, Fraction] = {x: Fraction(0) for x in keep_set}
    for lst, w in zip(lists, weights):
        if Fraction(w) == 0:
            continue
        lst = np.asarray(lst, dtype=np.int64)
        mask = np.isin(lst, keep)
        for r in np.flatnonzero(mask):
            F[int(lst[r])] += g(int(r) + 1, w, k)
    pos = [(f, x) for x, f in F.items() if f > 0]
    pos.sort(key=lambda p: (-p[0], p[1]))
    return [x for _, x in pos[:K]]
