"""Shared helpers of the GPU parity tests: the parity rules of the dense
channel and a CPU reference of the fused result.

Everything here works on corpora of several million rows: float64 scores and
norms are computed in row chunks (never a float64 copy of the whole corpus),
and the order checks are vectorised."""
import numpy as np

from oracle import dense as odense
from oracle import rrf as orrf

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


def hybrid_dense_list(gpu_prefix, q, corpus, visible=None, s64=None):
    """The GPU's emitted dense prefix followed by the rest of the visible rows
    in fp64 order: the complete list that the emitted prefix commits to."""
    if s64 is None:
        s64 = scores64(q, corpus)
    ids = np.arange(len(s64), dtype=np.int64)
    if visible is not None:
        ids = ids[visible]
    full = odense.rank_order(s64[ids], ids)
    seen = np.zeros(len(s64), dtype=bool)
    prefix = np.asarray(gpu_prefix, dtype=np.int64)
    seen[prefix] = True
    return np.concatenate([prefix, full[~seen[full]]])


def fused_reference(dense_list, sparse_list, K, k=60, w=(1, 1)):
    return orrf.rrf_topk([dense_list, sparse_list], list(w), k, K)
