"""Parity at the passage scale, 8.8M x 768 (4,096 centres), in the launch
configurations bench.py times: the 256-query batch (Int8 MFMA scan) at
weights 1:1 and 2:1, the 64-query batch and the 200 single requests (dot4
GEMV scan).  Every query of every set is checked against the exhaustive
oracle: float64 score of every row and a full sort (Sec. 2.1, 2.3.1),
brute-force sparse scores (Sec. 2.3.2) and exact complete-list RRF
(Sec. 2.1, 2.2).  The dense and sparse ranks each fusion actually read are
taken from the rank observer, so the prefix checked is the one the batched
run consumed."""
import time

import numpy as np
import pytest

from paper_2608_07152_amd import datagen

from full_common import K, check_query, dense_read, load_library, note
from gpu_helpers import (check_dense_prefix, check_fusion_run, for_each_parallel, full_order,
                         row_norms64, score_matrix)

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


def _fused_runs(E, idx, pbm, q, qs, settings, per_query=False):
    """eahr_topk over the set for each weight setting, with the ranks it read."""
    runs = []
    for wts in settings:
        t = time.time()
        if per_query:
            out = ([], [], [], [], {})
            for b in range(len(q)):
                with E.RankRecorder() as rec:
                    ids, cnt, stt, stats = E.eahr_topk(idx, pbm, q[b:b + 1], qs[b:b + 1], K=K,
                                                       w_dense=wts[0], w_sparse=wts[1])
                out[0].append(ids[0])
                out[1].append(cnt[0])
                out[2].append(stt[0])
                out[3].append(stats[0])
                out[4][b] = (rec.ranks(0, 0), rec.ranks(0, 1))
            ids, cnt, stt, stats, reads = np.array(out[0]), np.array(out[1]), np.array(out[2]), out[3], out[4]
        else:
            with E.RankRecorder() as rec:
                ids, cnt, stt, stats = E.eahr_topk(idx, pbm, q, qs, K=K, w_dense=wts[0], w_sparse=wts[1])
            reads = {b: (rec.ranks(b, 0), rec.ranks(b, 1)) for b in range(len(q))}
        note(f"{len(q)} queries {wts}: eahr_topk {time.time() - t:.2f}s, median dense depth "
             f"{int(np.median([s['dense_depth'] for s in stats]))}")
        assert np.all(stt == 0) and np.all(cnt == K)
        runs.append((wts, ids, cnt, stats, reads))
    return runs


def _check_every_query(x, vn, post, q, qs, runs, label):
    t = time.time()
    S = score_matrix(q, x)
    note(f"{label}: oracle scores of {len(q)} queries in {time.time() - t:.1f}s")

    def one(b):
        full = full_order(S[b])
        for wts, ids, cnt, stats, reads in runs:
            check_fusion_run(q[b], x, vn, post, qs[b], ids[b], cnt[b], stats[b], reads[b][0],
                             reads[b][1], wts, S[b], full=full, K=K)

    for_each_parallel(one, range(len(q)))
    note(f"{label}: every query checked in {time.time() - t:.1f}s")
    return S


def test_passage_b256_every_query_matches_oracle(E, passage):
    w, x, vn, post, sets, idx, pbm, s64cache = passage
    q, qs = sets["b256"]
    runs = _fused_runs(E, idx, pbm, q, qs, [(1, 1), (2, 1)])
    S = _check_every_query(x, vn, post, q, qs, runs, "b256")
    # the 256-query MFMA scan's own prefixes (1,000 ranks over two calls):
    # the oracle's for every query and, bit for bit, the single-query GEMV
    # prefixes of sampled queries
    st = E.pvs_open(idx, q)
    ids, scs, cnt, _ = E.pvs_next(st, 300)
    ids2, scs2, cnt2, _ = E.pvs_next(st, 700)
    st.close()
    assert np.all(cnt == 300) and np.all(cnt2 == 700)
    full_i = np.concatenate([ids, ids2], axis=1)
    full_s = np.concatenate([scs, scs2], axis=1)
    for_each_parallel(lambda b: check_dense_prefix(q[b], x, full_i[b], full_s[b], s64=S[b], vn=vn),
                      range(len(q)))
    for b in (0, 131, 255):
        di, ds = dense_read(E, idx, q[b], 1000)
        assert np.array_equal(di, full_i[b]) and np.array_equal(ds, full_s[b])
    for b in (0, 5):
        s64cache[("b256", b)] = S[b].copy()
    del S


def test_passage_b256_gpu_sparse_generator(E, passage):
    """The 256-query batch with Posting Block-Max's posting work on the GPU:
    the same Top-20, statuses, sparse ranks read and sparse work counters as
    the host generator, whose every query the test above checks against the
    oracle (so this run is oracle-exact too)."""
    w, x, vn, post, sets, idx, pbm, _ = passage
    q, qs = sets["b256"]
    out = []
    for gen in ("pbm", "pbm_gpu"):
        t = time.time()
        with E.RankRecorder() as rec:
            ids, cnt, stt, stats = E.eahr_topk(idx, pbm, q, qs, K=K, sparse_generator=gen)
        note(f"b256 sparse generator {gen}: eahr_topk {time.time() - t:.2f}s")
        out.append((ids, cnt, stt, stats, [rec.ranks(b, 1) for b in range(len(q))]))
    (ia, ca, sa, ta, ra), (ib, cb, sb, tb, rb) = out
    assert np.array_equal(ia, ib) and np.array_equal(ca, cb) and np.array_equal(sa, sb)
    for b in range(len(q)):
        assert np.array_equal(ra[b][0], rb[b][0]) and np.array_equal(ra[b][1], rb[b][1]), b
        for key in ("sparse_depth", "sparse_postings", "sparse_scored"):
            assert ta[b][key] == tb[b][key], (b, key)


def test_passage_single_requests_every_query(E, passage):
    w, x, vn, post, sets, idx, pbm, s64cache = passage
    q, qs = sets["single"]
    runs = _fused_runs(E, idx, pbm, q, qs, [(1, 1)], per_query=True)
    S = _check_every_query(x, vn, post, q, qs, runs, "single")
    for b in (0, 5):
        s64cache[("single", b)] = S[b].copy()
    del S


def test_passage_b64_every_query(E, passage):
    w, x, vn, post, sets, idx, pbm, _ = passage
    q, qs = sets["b64"]
    runs = _fused_runs(E, idx, pbm, q, qs, [(1, 1)])
    _check_every_query(x, vn, post, q, qs, runs, "b64")


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
