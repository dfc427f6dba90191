"""Parity at the mid-scale configuration (N = 1,000,000, d = 384, one batch of
256 queries through the MFMA scan), checked on sampled queries against the
exhaustive oracle (Sec. 2.1, 2.3)."""
import numpy as np
import pytest

from oracle import sparse as osparse
from paper_2608_07152_amd import datagen

from gpu_helpers import check_dense_prefix, fused_reference, hybrid_dense_list

pytestmark = pytest.mark.gpu

SAMPLED = (0, 77, 255)


@pytest.fixture(scope="module")
def mid():
    from paper_2608_07152_amd import eahr
    eahr.load()
    w = datagen.workload("mid")
    x, lab = datagen.corpus(w)
    q, qlab = datagen.queries(w)
    idx = eahr.pvs_build(x)
    return eahr, w, x, lab, q, qlab, idx


def test_mid_batch_prefixes_match_oracle(mid):
    E, w, x, lab, q, qlab, idx = mid
    st = E.pvs_open(idx, q)
    ids, scs, cnt, stt = E.pvs_next(st, 300)
    assert np.all(cnt == 300)
    for b in SAMPLED:
        check_dense_prefix(q[b], x, ids[b], scs[b])
    # second call continues every prefix
    ids2, scs2, cnt2, _ = E.pvs_next(st, 700)
    for b in SAMPLED:
        check_dense_prefix(q[b], x, np.concatenate([ids[b], ids2[b]]),
                           np.concatenate([scs[b], scs2[b]]))


def test_mid_eahr_topk_matches_complete_rrf(mid):
    E, w, x, lab, q, qlab, idx = mid
    post = datagen.bm25_impacts(w, datagen.sparse_docs(w, lab))
    qs = datagen.sparse_queries(w, qlab)
    pbm = E.pbm_build(post.term_ptr, post.doc, post.impact, w.n, 4096)
    ids, cnt, stt, stats = E.eahr_topk(idx, pbm, q, qs, K=20)
    assert np.all(stt == 0) and np.all(cnt == 20)
    for b in SAMPLED:
        st = E.pvs_open(idx, q[b:b + 1])
        D = stats[b]["dense_depth"]
        di, ds, _, _ = E.pvs_next(st, D)
        check_dense_prefix(q[b], x, di[0], ds[0])
        S = osparse.sparse_scores(post.term_ptr, post.doc, post.impact, qs[b][0], qs[b][1], w.n)
        want = fused_reference(hybrid_dense_list(di[0], q[b], x), osparse.sparse_ranking(S), 20)
        assert list(ids[b]) == want
