"""Shared helpers of the GPU parity tests: the parity rules of the dense
channel and a CPU reference of the fused result.

Everything here works on corpora of several million rows: float64 scores and
norms are computed in row chunks (never a float64 copy of the whole corpus),
and the order checks are vectorised."""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from oracle import dense as odense
from oracle import rrf as orrf
from oracle import sparse as osparse

# float32 score tolerance and near-tie window, relative to max(|s64|, ||q|| ||v||)
SCORE_RTOL = 1e-5
TIE_RTOL = 2e-5

CHUNK = 1 << 19


def scores64(q, corpus):
    """float64 inner products of one query with every corpus row (chunked
    calls of the oracle's scoring rule)."""
    n = corpus.shape[0]
    out = np.empty(n, dtype=np.float64)
    for r in range(0, n, CHUNK):
        out[r:r + CHUNK] = odense.scores64(q, corpus[r:r + CHUNK])
    return out


def score_matrix(Q, corpus):
    """float64 inner products of every query with every corpus row, [B, n]
    (the oracle's scoring rule on row chunks)."""
    Q = np.asarray(Q, np.float32)
    n = corpus.shape[0]
    out = np.empty((Q.shape[0], n), dtype=np.float64)
    for r in range(0, n, CHUNK):
        out[:, r:r + CHUNK] = odense.scores64(Q, corpus[r:r + CHUNK])
    return out


def for_each_parallel(fn, items, workers=None):
    """fn(item) for every item on host threads (numpy's sorts and matrix
    products release the GIL); the first failure is raised."""
    workers = workers or min(16, os.cpu_count() or 1)
    with ThreadPoolExecutor(workers) as ex:
        for _ in ex.map(fn, list(items)):
            pass


def row_norms64(corpus):
    """||v||_2 of every row in float64 (chunked)."""
    n = corpus.shape[0]
    out = np.empty(n, dtype=np.float64)
    for r in range(0, n, CHUNK):
        out[r:r + CHUNK] = np.linalg.norm(corpus[r:r + CHUNK].astype(np.float64), axis=1)
    return out


def check_dense_prefix(q, corpus, got_ids, got_scores, visible=None, s64=None, vn=None):
    """Compare an emitted dense prefix with the exact fp64 ranking.

    * every emitted score is within SCORE_RTOL of the fp64 score;
    * the emitted ids are the fp64 prefix, except that two items may swap
      when their fp64 scores differ by less than TIE_RTOL (pairwise rule).
    ``s64`` / ``vn`` may pass precomputed scores and row norms.
    Returns the number of inverted adjacent pairs seen."""
    got_ids = np.asarray(got_ids, dtype=np.int64)
    D = len(got_ids)
    if s64 is None:
        s64 = scores64(q, corpus)
    if vn is None:
        vn = row_norms64(corpus)
    qn = float(np.linalg.norm(np.asarray(q, np.float32).astype(np.float64)))
    if D == 0:
        return 0
    # scores
    sg = s64[got_ids]
    scale_g = np.maximum(np.abs(sg), qn * vn[got_ids])
    err = np.abs(np.asarray(got_scores, np.float64) - sg)
    assert np.all(err <= SCORE_RTOL * scale_g), float(np.max(err / scale_g))
    assert len(np.unique(got_ids)) == D, "duplicate ids emitted"
    if visible is not None:
        assert np.all(visible[got_ids]), "invisible row emitted"
    want = odense.dense_prefix(q, None, D, visible, s64=s64)
    if np.array_equal(want, got_ids):
        return 0
    # sets may differ only at the boundary, by near-ties with the last item
    boundary = s64[want[-1]]
    diff = np.setxor1d(got_ids, want)
    if len(diff):
        tol = TIE_RTOL * np.maximum(np.maximum(np.abs(s64[diff]), abs(boundary)), qn * vn[diff])
        bad = np.abs(s64[diff] - boundary) >= tol
        assert not np.any(bad), (diff[bad][:5], s64[diff[bad][:5]], boundary)

    def pair_tol(a, b):
        return TIE_RTOL * np.maximum.reduce([np.abs(s64[a]), np.abs(s64[b]), qn * vn[a], qn * vn[b]])

    # order: every inverted adjacent pair must be a near-tie
    x, y = got_ids[:-1], got_ids[1:]
    sx, sy = s64[x] + 0.0, s64[y] + 0.0
    inv = (sx < sy) | ((sx == sy) & (x > y))
    if np.any(inv):
        gap = (sy - sx)[inv]
        tol = pair_tol(x[inv], y[inv])
        assert np.all(gap < tol), (np.flatnonzero(inv)[gap >= tol][:5],)
    # displaced items: the item at each position of the sorted order and the
    # emitted one there must be near-ties
    order = odense.rank_order(sg, got_ids)
    moved = order != got_ids
    if np.any(moved):
        a, b = order[moved], got_ids[moved]
        ok = np.abs(s64[a] - s64[b]) < pair_tol(a, b)
        assert np.all(ok), (np.flatnonzero(moved)[~ok][:5],)
    return int(np.count_nonzero(inv))


def full_order(s64, visible=None):
    """The oracle's complete dense ranking of the visible rows from their
    float64 scores."""
    ids = np.arange(len(s64), dtype=np.int64)
    if visible is not None:
        ids = ids[visible]
    return odense.rank_order(s64[ids], ids)


def hybrid_dense_list(gpu_prefix, q, corpus, visible=None, s64=None, full=None):
    """The GPU's emitted dense prefix followed by the rest of the visible rows
    in fp64 order: the complete list that the emitted prefix commits to
    (``full``: that complete order, if already computed)."""
    if s64 is None:
        s64 = scores64(q, corpus)
    if full is None:
        full = full_order(s64, visible)
    seen = np.zeros(len(s64), dtype=bool)
    prefix = np.asarray(gpu_prefix, dtype=np.int64)
    seen[prefix] = True
    return np.concatenate([prefix, full[~seen[full]]])


def fused_reference(dense_list, sparse_list, K, k=60, w=(1, 1)):
    return orrf.rrf_topk([dense_list, sparse_list], list(w), k, K)


def check_fusion_run(q, corpus, vn, post, qs, got, count, stats, dense_read, sparse_read, wts,
                     s64, full=None, visible=None, K=20, k=60):
    """One query of a fused run against the oracle, using what the run read:
    the dense ranks the fusion read equal the exact prefix (parity rules of
    check_dense_prefix) and number its dense depth; the sparse ranks it read
    equal the exact sparse ranking bit for bit; the fused Top-K equals the
    complete-list RRF of the GPU's dense prefix followed by the oracle's
    order of the rest, and of the exact sparse ranking."""
    di, ds = dense_read
    assert len(di) == stats["dense_depth"], (len(di), stats["dense_depth"])
    check_dense_prefix(q, corpus, di, ds, visible, s64=s64, vn=vn)
    n = corpus.shape[0]
    S = osparse.sparse_scores(post.term_ptr, post.doc, post.impact, qs[0], qs[1], n, visible)
    sr = osparse.sparse_ranking(S)
    si, ss = sparse_read
    assert len(si) == stats["sparse_depth"], (len(si), stats["sparse_depth"])
    assert np.array_equal(si, sr[:len(si)])
    assert np.array_equal(ss.view(np.int32), S[si].view(np.int32))
    if full is None:
        full = full_order(s64, visible)
    want = fused_reference(hybrid_dense_list(di, q, corpus, visible, s64=s64, full=full), sr, K, k, wts)
    assert list(got[:count]) == want
    assert stats["resolved"] == 1
