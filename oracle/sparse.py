"""Brute-force sparse scores and ranking (oracle).

Sec. 2.3.2: S(x) = sum over query terms t of q_t * p_t(x), with p_t(x) = 0 when
x has no posting for t.  App. A.2: the implementation value is the float32
accumulation in one fixed term order; the order used here (and by the product)
is ascending term id, one float32 rounding per multiply and per add.  The
support set of the sparse retriever is {x : S(x) > 0} (Sec. 2.1).

Every document is scored directly from the postings, without block-max
metadata.  Parity: pinned against a per-document Python loop, on an order-
sensitive float32 sum with a closed-form value, and on tiny hand-built indexes.
"""
from __future__ import annotations

from typing import Optional

import numpy as np


def sparse_scores(term_ptr: np.ndarray, doc: np.ndarray, impact: np.ndarray,
                  q_terms: np.ndarray, q_weights: np.ndarray, n: int,
                  visible: Optional[np.ndarray] = None) -> np.ndarray:
    """float32 [n] scores; invisible documents score 0."""
    order = np.argsort(np.asarray(q_terms), kind="stable")
    S = np.zeros(n, dtype=np.float32)
    for i in order:
        t = int(q_terms[i])
        wq = np.float32(q_weights[i])
        a, b = int(term_ptr[t]), int(term_ptr[t + 1])
        contrib = np.zeros(n, dtype=np.float32)
        contrib[doc[a:b]] = (wq * impact[a:b]).astype(np.float32)
        S = (S + contrib).astype(np.float32)
    if visible is not None:
        S = np.where(visible, S, np.float32(0)).astype(np.float32)
    return S


def sparse_ranking(S: np.ndarray) -> np.ndarray:
    """Ids with S > 0 sorted by (S descending, id ascending)."""
    S = np.asarray(S, dtype=np.float32)
    ids = np.flatnonzero(S > 0).astype(np.int64)
    order = np.lexsort((ids, -S[ids].astype(np.float64)))
    return ids[order]
