"""Shared helpers of the GPU parity tests: the parity rules of the dense
channel and a CPU reference of the fused result."""
import numpy as np

from oracle import dense as odense
from oracle import rrf as orrf

# float32 score tolerance and near-tie window, relative to max(|s64|, ||q|| ||v||)
SCORE_RTOL = 1e-5
TIE_RTOL = 2e-5


def check_dense_prefix(q, corpus, got_ids, got_scores, visible=None):
    """Compare an emitted dense prefix with the exact fp64 ranking.

    * every emitted score is within SCORE_RTOL of the fp64 score;
    * the emitted ids are the fp64 prefix, except that two items may swap
      when their fp64 scores differ by less than TIE_RTOL (pairwise rule).
    Returns the number of inverted adjacent pairs seen."""
    got_ids = np.asarray(got_ids, dtype=np.int64)
    D = len(got_ids)
    s64 = odense.scores64(q, corpus)
    qn = float(np.linalg.norm(q.astype(np.float64)))
    vn = np.linalg.norm(corpus.astype(np.float64), axis=1)
    scale = np.maximum(np.abs(s64), qn * vn)
    # scores
    err = np.abs(np.asarray(got_scores, np.float64) - s64[got_ids])
    assert np.all(err <= SCORE_RTOL * scale[got_ids]), float(np.max(err / scale[got_ids]))
    assert len(set(got_ids.tolist())) == D, "duplicate ids emitted"
    if visible is not None:
        assert np.all(visible[got_ids]), "invisible row emitted"
    want = odense.dense_prefix(q, corpus, D, visible, s64=s64)
    if np.array_equal(want, got_ids):
        return 0
    # sets may differ only at the boundary, by near-ties with the last item
    gs, ws = set(got_ids.tolist()), set(want.tolist())
    boundary = s64[want[-1]]
    for x in gs ^ ws:
        tol = TIE_RTOL * max(abs(s64[x]), abs(boundary), qn * vn[x])
        assert abs(s64[x] - boundary) < tol, (x, s64[x], boundary)
    # order: every inverted pair must be a near-tie
    pos = {int(x): i for i, x in enumerate(got_ids)}
    inv = 0
    for i in range(D - 1):
        x, y = int(got_ids[i]), int(got_ids[i + 1])
        if (s64[x], -x) < (s64[y], -y):
            tol = TIE_RTOL * max(abs(s64[x]), abs(s64[y]), qn * vn[x], qn * vn[y])
            assert s64[y] - s64[x] < tol, (i, x, y, s64[x], s64[y])
            inv += 1
    # non-adjacent inversions: compare against the sorted order window-wise
    order = sorted(got_ids.tolist(), key=lambda x: (-s64[x], x))
    for i, x in enumerate(order):
        j = pos[x]
        if j != i:
            y = int(got_ids[i])
            tol = TIE_RTOL * max(abs(s64[x]), abs(s64[y]), qn * vn[x], qn * vn[y])
            assert abs(s64[x] - s64[y]) < tol, (i, x, y)
    return inv


def hybrid_dense_list(gpu_prefix, q, corpus, visible=None):
    """The GPU's emitted dense prefix followed by the rest of the visible rows
    in fp64 order: the complete list that the emitted prefix commits to."""
    full = odense.dense_ranking(q, corpus, visible)
    seen = set(int(x) for x in gpu_prefix)
    rest = [int(x) for x in full if int(x) not in seen]
    return np.array(list(gpu_prefix) + rest, dtype=np.int64)


def fused_reference(dense_list, sparse_list, K, k=60, w=(1, 1)):
    return orrf.rrf_topk([dense_list, sparse_list], list(w), k, K)
