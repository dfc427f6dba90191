"""Parity at the passage scale, 8.8M x 768 (4,096 centres), in the launch
configurations bench.py times: the 256-query batch (Int8 MFMA scan) at
weights 1:1 and 2:1, a 64-query batch and single requests (dot4 GEMV scan).
Sampled queries are checked against the exhaustive oracle: float64 score of
every row and a full sort (Sec. 2.1, 2.3.1), brute-force sparse scores
(Sec. 2.3.2) and exact complete-list RRF (Sec. 2.1, 2.2)."""
import time

import numpy as np
import pytest

from paper_2608_07152_amd import datagen

from full_common import K, check_query, dense_read, load_library, note
from gpu_helpers import check_dense_prefix, row_norms64, scores64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def E():
    return load_library()


@pytest.fixture(scope="module")
def passage(E):
    t = time.time()
    w = datagen.workload("passage")
    x, lab = datagen.corpus(w)
    docs = datagen.sparse_docs(w, lab)
    post = datagen.bm25_impacts(w, docs)
    del docs
    sets = {}
    for name in ("single", "b64", "b256"):
        q, qlab = datagen.queries(w, name)
        sets[name] = (q, datagen.sparse_queries(w, qlab, datagen.query_set_offset(w, name)))
    idx = E.pvs_build(x)
    pbm = E.pbm_build(post.term_ptr, post.doc, post.impact, w.n, 4096)
    vn = row_norms64(x)
    note(f"passage set up in {time.time() - t:.1f}s")
    s64cache = {}
    yield w, x, vn, post, sets, idx, pbm, s64cache
    idx.free()
    pbm.free()


@pytest.mark.parametrize("wts", [(1, 1), (2, 1)])
def test_passage_b256_topk_matches_oracle(E, passage, wts):
    w, x, vn, post, sets, idx, pbm, s64cache = passage
    q, qs = sets["b256"]
    t = time.time()
    ids, cnt, stt, stats = E.eahr_topk(idx, pbm, q, qs, K=K, w_dense=wts[0], w_sparse=wts[1])
    note(f"b256 {wts}: eahr_topk {time.time() - t:.2f}s, median dense depth "
         f"{int(np.median([s['dense_depth'] for s in stats]))}")
    assert np.all(stt == 0) and np.all(cnt == K)
    for b in (0, 131, 255):
        key = ("b256", b)
        s64cache[key] = check_query(E, idx, x, vn, post, q[b], qs[b], ids[b], stats[b], wts,
                                    s64=s64cache.get(key))
    note(f"b256 {wts}: sampled queries checked")


def test_passage_b256_batch_prefixes(E, passage):
    """The 256-query MFMA scan at full size: sampled prefixes equal the
    oracle's and, bit for bit, the single-query GEMV prefixes."""
    w, x, vn, post, sets, idx, pbm, s64cache = passage
    q, _ = sets["b256"]
    st = E.pvs_open(idx, q)
    ids, scs, cnt, _ = E.pvs_next(st, 300)
    ids2, scs2, cnt2, _ = E.pvs_next(st, 700)
    st.close()
    assert np.all(cnt == 300) and np.all(cnt2 == 700)
    for b in (0, 131, 255):
        key = ("b256", b)
        if key not in s64cache:
            s64cache[key] = scores64(q[b], x)
        full_i = np.concatenate([ids[b], ids2[b]])
        full_s = np.concatenate([scs[b], scs2[b]])
        check_dense_prefix(q[b], x, full_i, full_s, s64=s64cache[key], vn=vn)
        di, ds = dense_read(E, idx, q[b], 1000)
        assert np.array_equal(di, full_i) and np.array_equal(ds, full_s)


def test_passage_single_requests_match_oracle(E, passage):
    w, x, vn, post, sets, idx, pbm, _ = passage
    q, qs = sets["single"]
    for b in (0, 101, 199):
        ids, cnt, stt, stats = E.eahr_topk(idx, pbm, q[b:b + 1], qs[b:b + 1], K=K)
        assert stt[0] == 0 and cnt[0] == K
        check_query(E, idx, x, vn, post, q[b], qs[b], ids[0], stats[0], (1, 1))


def test_passage_b64_matches_oracle(E, passage):
    w, x, vn, post, sets, idx, pbm, _ = passage
    q, qs = sets["b64"]
    ids, cnt, stt, stats = E.eahr_topk(idx, pbm, q, qs, K=K)
    assert np.all(stt == 0) and np.all(cnt == K)
    for b in (5, 63):
        check_query(E, idx, x, vn, post, q[b], qs[b], ids[b], stats[b], (1, 1))


def test_passage_alternative_generators_match_oracle(E, passage):
    # the rank-generator ablation (Sec. 4.4) at full size: scalar intervals
    # with one global scale, the exhaustive float32 scan and the complete
    # sparse ranking give the Top-20 of PVS + PBM, and that Top-20 is the
    # oracle's for sampled queries
    w, x, vn, post, sets, idx, pbm, s64cache = passage
    q, qs = sets["single"]
    t = time.time()
    gidx = E.pvs_build_quant(x, "global")
    note(f"global-scale index built in {time.time() - t:.1f}s")
    ref = E.eahr_topk(idx, pbm, q[:8], qs[:8], K=K)
    alts = {
        "scalar": E.eahr_topk(gidx, pbm, q[:8], qs[:8], K=K),
        "scan": E.eahr_topk(idx, pbm, q[:2], qs[:2], K=K, dense_generator="full_scan"),
        "sparse_complete": E.eahr_topk(idx, pbm, q[:8], qs[:8], K=K, sparse_generator="complete"),
    }
    for name, r in alts.items():
        n = r[0].shape[0]
        assert np.all(r[2] == 0), name
        assert np.array_equal(r[0], ref[0][:n]) and np.array_equal(r[1], ref[1][:n]), name
    for b in (0, 5):
        key = ("single", b)
        s64cache[key] = check_query(E, idx, x, vn, post, q[b], qs[b], ref[0][b], ref[3][b], (1, 1),
                                    s64=s64cache.get(key))
    gidx.free()
    note("alternative generators checked")
