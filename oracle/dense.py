"""Exact dense ranking (oracle).

Sec. 2.1: a retriever's scoring rule together with the total identifier order
defines one complete ranked list; Sec. 2.3.1 scores a pair by the inner product
q^T v.  Here every product of float32 inputs is exact in float64 and the float64
sum carries a relative error of about d * 2^-53, so the oracle ranks by
``s64 = sum_j double(q_j) * double(v_j)`` in (score descending, id ascending)
order.  Items outside the visible set are not ranked.

Parity: pinned against a plain Python loop (brute force), against a library
sort on the same scores, on an all-tied corpus (identifier order) and on
integer-valued vectors whose inner products are exact.
"""
from __future__ import annotations

from typing import Optional

import numpy as np


def scores64(q: np.ndarray, v: np.ndarray) -> np.ndarray:
    """float64 inner products, [B, n] (or [n] for a single query vector)."""
    q64 = np.asarray(q, dtype=np.float32).astype(np.float64)
    v64 = np.asarray(v, dtype=np.float32).astype(np.float64)
    return q64 @ v64.T


def rank_order(scores: np.ndarray, ids: Optional[np.ndarray] = None) -> np.ndarray:
    """Ids sorted by (score descending, id ascending).  -0.0 equals +0.0.

    Two stable sorts: by id, then by descending score, which keeps the id
    order among equal scores."""
    s = np.asarray(scores, dtype=np.float64) + 0.0   # maps -0.0 to +0.0
    if ids is None:
        ids = np.arange(len(s), dtype=np.int64)
    ids = np.asarray(ids)
    by_id = np.argsort(ids, kind="stable")
    by_score = np.argsort(-s[by_id], kind="stable")
    return ids[by_id[by_score]]


def dense_ranking(q: np.ndarray, v: np.ndarray, visible: Optional[np.ndarray] = None
                  ) -> np.ndarray:
    """Complete exact dense ranking of one query over the visible rows."""
    s = scores64(q, v)
    ids = np.arange(v.shape[0], dtype=np.int64)
    if visible is not None:
        ids = ids[visible]
        s = s[visible]
    return rank_order(s, ids)


def dense_prefix(q: np.ndarray, v: np.ndarray, depth: int,
                 visible: Optional[np.ndarray] = None, s64: Optional[np.ndarray] = None
                 ) -> np.ndarray:
    """First ``depth`` entries of :func:`dense_ranking`.

    Selects every row whose score reaches the depth-th largest score, then sorts
    that set exactly as the full ranking would; the result is the full
    ranking's prefix because every row outside the set scores strictly lower."""
    s = scores64(q, v) if s64 is None else np.asarray(s64, dtype=np.float64)
    s = s + 0.0
    ids = np.arange(v.shape[0] if v is not None else len(s), dtype=np.int64)
    if visible is not None:
        ids = ids[visible]
        s = s[visible]
    n = len(s)
    depth = min(depth, n)
    if depth == 0:
        return np.zeros(0, dtype=np.int64)
    if depth == n:
        return rank_order(s, ids)
    kth = np.partition(-s, depth - 1)[depth - 1]       # -(depth-th largest score)
    sel = np.flatnonzero(-s <= kth)
    return rank_order(s[sel], ids[sel])[:depth]
