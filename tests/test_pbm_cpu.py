"""PBM sparse channel through the C ABI against the brute-force oracle
(Sec. 2.3.2, App. A.2).  Host only."""
import numpy as np
import pytest

from oracle import sparse as osparse
from paper_2608_07152_amd import datagen, eahr


@pytest.fixture(scope="module")
def tiny_sparse():
    w = datagen.workload("tiny", n=6000)
    _, lab = datagen.corpus(w)
    docs = datagen.sparse_docs(w, lab)
    post = datagen.bm25_impacts(w, docs)
    _, qlab = datagen.queries(w, count=6)
    qs = datagen.sparse_queries(w, qlab)
    return w, post, qs


def _oracle_ranking(post, n, terms, wts):
    S = osparse.sparse_scores(post.term_ptr, post.doc, post.impact, terms, wts, n)
    r = osparse.sparse_ranking(S)
    return r, S[r]


@pytest.mark.parametrize("range_size", [1, 7, 256, 4096, 10 ** 6])
def test_pbm_full_ranking_bit_exact(tiny_sparse, range_size):
    w, post, qs = tiny_sparse
    idx = eahr.pbm_build(post.term_ptr, post.doc, post.impact, w.n, range_size)
    for terms, wts in qs:
        want_ids, want_s = _oracle_ranking(post, w.n, terms, wts)
        st = eahr.pbm_open(idx, terms, wts)
        ids, sc, status = eahr.pbm_next(st, w.n + 5)
        assert status == eahr.LIST_EXHAUSTED
        assert np.array_equal(ids, want_ids)
        assert np.array_equal(sc, want_s)


def test_pbm_split_calls_equal_one_call(tiny_sparse):
    w, post, qs = tiny_sparse
    idx = eahr.pbm_build(post.term_ptr, post.doc, post.impact, w.n, 128)
    terms, wts = qs[0]
    want_ids, _ = _oracle_ranking(post, w.n, terms, wts)
    st = eahr.pbm_open(idx, terms, wts)
    got = []
    for m in (1, 2, 20, 0, 40, 3, 1000, 10 ** 6):
        ids, _, status = eahr.pbm_next(st, m)
        assert len(ids) == m or status == eahr.LIST_EXHAUSTED
        got.extend(ids)
    assert np.array_equal(np.array(got), want_ids)


def test_pbm_weights_and_ties():
    # hand index with exact ties across ranges and zero-weight terms
    term_ptr = np.array([0, 4, 8, 9])
    docs = np.array([0, 3, 5, 9, 1, 3, 5, 8, 2], dtype=np.int32)
    imp = np.array([1, 2, 2, 1, 1, 0, 0, 1, 5], dtype=np.float32)
    idx = eahr.pbm_build(term_ptr, docs, imp, 10, 3)
    for terms, wts in (([0, 1], [1.0, 1.0]), ([1, 0, 2], [2.0, 1.0, 0.0]), ([2], [0.5])):
        st = eahr.pbm_open(idx, terms, wts)
        ids, sc, status = eahr.pbm_next(st, 100)
        want, want_s = _oracle_ranking(
            eahr_post(term_ptr, docs, imp), 10, np.array(terms), np.array(wts, dtype=np.float32))
        assert np.array_equal(ids, want) and np.array_equal(sc, want_s)
        assert status == eahr.LIST_EXHAUSTED


def eahr_post(term_ptr, docs, imp):
    return datagen.Postings(len(term_ptr) - 1, term_ptr, docs, imp)


def test_pbm_empty_query_is_exhausted():
    idx = eahr.pbm_build(np.array([0, 1]), np.array([0], np.int32), np.array([1], np.float32), 1, 4)
    st = eahr.pbm_open(idx, [], [])
    ids, _, status = eahr.pbm_next(st, 5)
    assert len(ids) == 0 and status == eahr.LIST_EXHAUSTED


def test_pbm_uncovered_blockmax_fails(tiny_sparse):
    w, post, qs = tiny_sparse
    idx = eahr.pbm_build(post.term_ptr, post.doc, post.impact, w.n, 64)
    terms, wts = qs[1]
    t = int(terms[0])
    first_doc = int(post.doc[post.term_ptr[t]])
    eahr.pbm_debug_set_blockmax(idx, t, first_doc // 64, 0.0)
    st = eahr.pbm_open(idx, terms, wts)
    ids, _, status = eahr.pbm_next(st, w.n)
    assert status == eahr.LIST_FAILED


def test_pbm_rejects_bad_postings():
    with pytest.raises(eahr.EahrError):
        eahr.pbm_build(np.array([0, 2]), np.array([3, 3], np.int32), np.ones(2, np.float32), 5, 2)
    with pytest.raises(eahr.EahrError):
        eahr.pbm_build(np.array([0, 1]), np.array([0], np.int32), np.array([-1.0], np.float32), 5, 2)
    with pytest.raises(eahr.EahrError):
        eahr.pbm_build(np.array([0, 1]), np.array([0], np.int32), np.array([np.inf], np.float32), 5, 2)


def test_pbm_common_term_partial_publication():
    """A term in most documents makes every range worth expanding, so far
    more items become publishable than a request wants; they are published
    in runs of the smallest keys.  The complete ranking, read in doubling
    requests and in one request, equals the brute-force ranking."""
    rng = np.random.default_rng(11)
    n = 300_000
    common = np.sort(rng.choice(n, size=250_000, replace=False)).astype(np.int32)
    rare1 = np.sort(rng.choice(n, size=3_000, replace=False)).astype(np.int32)
    rare2 = np.sort(rng.choice(n, size=5_000, replace=False)).astype(np.int32)
    docs = np.concatenate([common, rare1, rare2])
    imp = np.concatenate([rng.uniform(0.01, 0.05, len(common)), rng.uniform(1, 9, len(rare1)),
                          rng.uniform(1, 9, len(rare2))]).astype(np.float32)
    # a few exact ties across the common term
    imp[:1000] = np.float32(0.03)
    term_ptr = np.array([0, len(common), len(common) + len(rare1), len(docs)], dtype=np.int64)
    post = datagen.Postings(3, term_ptr, docs, imp)
    terms = np.array([0, 1, 2], np.int32)
    wts = np.ones(3, np.float32)
    want_ids, want_s = _oracle_ranking(post, n, terms, wts)
    idx = eahr.pbm_build(term_ptr, docs, imp, n, 4096)
    st = eahr.pbm_open(idx, terms, wts)
    got_i, got_s, m, status = [], [], 20, eahr.LIST_OPEN
    while status != eahr.LIST_EXHAUSTED:
        ids, sc, status = eahr.pbm_next(st, m)
        got_i.append(ids)
        got_s.append(sc)
        m *= 2
    assert np.array_equal(np.concatenate(got_i), want_ids)
    assert np.array_equal(np.concatenate(got_s), want_s)
    st1 = eahr.pbm_open(idx, terms, wts)
    ids, sc, status = eahr.pbm_next(st1, n + 1)
    assert status == eahr.LIST_EXHAUSTED and np.array_equal(ids, want_ids)


# ---------------------------------------------------------------------------
# Complete exact sparse ranking (the alternative generator of Sec. 4.4)

@pytest.mark.parametrize("range_size", [7, 4096])
def test_complete_generator_equals_oracle_and_pbm(tiny_sparse, range_size):
    w, post, qs = tiny_sparse
    idx = eahr.pbm_build(post.term_ptr, post.doc, post.impact, w.n, range_size)
    for terms, wts in qs:
        want_ids, want_s = _oracle_ranking(post, w.n, terms, wts)
        got = []
        gs = []
        st = eahr.pbm_open(idx, terms, wts, generator="complete")
        for m in (1, 19, 0, 300, 10 ** 6):
            ids, sc, status = eahr.pbm_next(st, m)
            assert len(ids) == m or status == eahr.LIST_EXHAUSTED
            got.extend(ids)
            gs.extend(sc)
        assert status == eahr.LIST_EXHAUSTED
        assert np.array_equal(np.array(got), want_ids)
        assert np.array_equal(np.array(gs, np.float32), want_s)


def test_complete_generator_reports_metadata_failure(tiny_sparse):
    # the complete generator expands every range, so a block-max entry below
    # its postings fails the list at the first call (App. A.2)
    w, post, qs = tiny_sparse
    idx = eahr.pbm_build(post.term_ptr, post.doc, post.impact, w.n, 64)
    terms, wts = qs[1]          # the case of test_pbm_uncovered_blockmax_fails
    t = int(terms[0])
    r = int(post.doc[post.term_ptr[t]]) // 64
    eahr.pbm_debug_set_blockmax(idx, t, r, 0.0)
    st = eahr.pbm_open(idx, terms, wts, generator="complete")
    ids, _, status = eahr.pbm_next(st, 10)
    assert status == eahr.LIST_FAILED and len(ids) == 0


def test_sparse_only_topk_with_complete_generator():
    w = datagen.workload("tiny", n=5000)
    _, lab = datagen.corpus(w)
    post = datagen.bm25_impacts(w, datagen.sparse_docs(w, lab))
    _, qlab = datagen.queries(w, count=5)
    qs = datagen.sparse_queries(w, qlab)
    idx = eahr.pbm_build(post.term_ptr, post.doc, post.impact, w.n, 512)
    a = eahr.eahr_topk(None, idx, None, qs, K=20, w_dense=0, w_sparse=1)
    c = eahr.eahr_topk(None, idx, None, qs, K=20, w_dense=0, w_sparse=1, sparse_generator="complete")
    f = eahr.eahr_topk(None, idx, None, qs, K=20, w_dense=0, w_sparse=1, sparse_generator="complete",
                       schedule="frozen")
    assert np.array_equal(a[0], c[0]) and np.array_equal(a[1], c[1])
    assert np.array_equal(a[0], f[0])


def test_pbm_index_freed_before_its_states(tiny_sparse):
    # pbm_free waits for the last pbm_close (finalisation order must not matter)
    w, post, qs = tiny_sparse
    idx = eahr.pbm_build(post.term_ptr, post.doc, post.impact, w.n, 512)
    sts = [eahr.pbm_open(idx, t, wt) for t, wt in qs[:3]]
    first, _, _ = eahr.pbm_next(sts[0], 10)
    eahr.load().pbm_free(idx.h)
    idx.h = None
    again, _, _ = eahr.pbm_next(sts[1], 10)
    want, _ = _oracle_ranking(post, w.n, qs[1][0], qs[1][1])
    assert len(first) == 10 and list(again) == want[:len(again)].tolist()
    for s in sts:
        s.close()


@pytest.mark.parametrize("schedule", ["doubling", "frozen"])
def test_rank_observer_sees_the_ranks_read(tiny_sparse, schedule):
    # the observer reports every rank a fusion reads, in list order, and
    # does not change the result (sparse-only fusion runs on the host)
    w, post, qs = tiny_sparse
    idx = eahr.pbm_build(post.term_ptr, post.doc, post.impact, w.n, 512)
    plain = eahr.eahr_topk(None, idx, None, qs, K=20, w_dense=0, w_sparse=1, schedule=schedule)
    with eahr.RankRecorder() as rec:
        got = eahr.eahr_topk(None, idx, None, qs, K=20, w_dense=0, w_sparse=1, schedule=schedule)
    after = eahr.eahr_topk(None, idx, None, qs, K=20, w_dense=0, w_sparse=1, schedule=schedule)
    assert np.array_equal(plain[0], got[0]) and np.array_equal(plain[0], after[0])
    for b, (t, wt) in enumerate(qs):
        ids, scores = rec.ranks(b, 1)
        want, wscores = _oracle_ranking(post, w.n, t, wt)
        assert len(ids) >= got[3][b]["sparse_depth"] > 0
        assert np.array_equal(ids, want[:len(ids)])
        assert np.array_equal(scores.view(np.int32), wscores[:len(ids)].view(np.int32))
        assert len(rec.ranks(b, 0)[0]) == 0


def test_sparse_work_counters(tiny_sparse):
    # the complete generator reads every posting of the query terms once and
    # scores every document carrying one; PBM stops earlier
    w, post, qs = tiny_sparse
    idx = eahr.pbm_build(post.term_ptr, post.doc, post.impact, w.n, 256)
    _, _, _, full = eahr.eahr_topk(None, idx, None, qs, K=20, w_dense=0, w_sparse=1,
                                   sparse_generator="complete")
    _, _, _, pbm = eahr.eahr_topk(None, idx, None, qs, K=20, w_dense=0, w_sparse=1)
    for b, (t, _) in enumerate(qs):
        n_post = sum(int(post.term_ptr[x + 1] - post.term_ptr[x]) for x in t)
        docs = np.unique(np.concatenate([post.doc[post.term_ptr[x]:post.term_ptr[x + 1]] for x in t]))
        assert full[b]["sparse_postings"] == n_post and full[b]["sparse_scored"] == len(docs)
        assert 0 < pbm[b]["sparse_postings"] <= n_post and 0 < pbm[b]["sparse_scored"] <= len(docs)
        assert full[b]["dense_evals"] == 0 == pbm[b]["dense_evals"]
