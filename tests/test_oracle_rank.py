"""Pins of the dense and sparse ranking oracles (Sec. 2.1, Sec. 2.3, App. A.2)."""
import math

import numpy as np

from oracle import dense, sparse
from paper_2608_07152_amd import datagen


def test_dense_ranking_matches_python_loop():
    w = datagen.workload("tiny", n=1500)
    x, _ = datagen.corpus(w)
    q, _ = datagen.queries(w, count=2)
    for b in range(2):
        got = dense.dense_ranking(q[b], x)
        # exact (correctly rounded) inner products with a plain loop
        s = [math.fsum(float(a) * float(c) for a, c in zip(q[b], x[i])) for i in range(len(x))]
        want = sorted(range(len(x)), key=lambda i: (-s[i], i))
        mism = np.flatnonzero(got != np.array(want))
        for p in mism:   # only possible between scores equal to float64 precision
            assert abs(s[got[p]] - s[want[p]]) <= 1e-14


def test_dense_all_tied_corpus_is_identifier_order():
    v = np.tile(np.array([[0.5, -0.25, 1.0]], dtype=np.float32), (50, 1))
    q = np.array([1.0, 2.0, 3.0], dtype=np.float32)
    assert list(dense.dense_ranking(q, v)) == list(range(50))


def test_dense_integer_vectors_exact_order():
    n = 64
    v = np.zeros((n, 4), dtype=np.float32)
    v[:, 0] = (np.arange(n) * 37) % n          # a permutation of 0..n-1
    v[:, 1] = 5
    q = np.array([1.0, 0.0, 0.0, 0.0], dtype=np.float32)
    got = dense.dense_ranking(q, v)
    assert list(v[got, 0]) == list(range(n - 1, -1, -1))


def test_dense_negative_zero_equals_positive_zero():
    v = np.array([[0.0], [-0.0], [0.0]], dtype=np.float32)
    q = np.array([-1.0], dtype=np.float32)      # scores: -0, +0, -0
    assert list(dense.dense_ranking(q, v)) == [0, 1, 2]


def test_dense_prefix_equals_full_sort_prefix():
    rng = np.random.default_rng(2)
    v = rng.integers(-3, 4, size=(3000, 8)).astype(np.float32)   # many exact ties
    q = rng.integers(-2, 3, size=8).astype(np.float32)
    full = dense.dense_ranking(q, v)
    for depth in (1, 7, 100, 2999, 3000):
        assert np.array_equal(dense.dense_prefix(q, v, depth), full[:depth])
    vis = rng.random(3000) < 0.7
    fullv = dense.dense_ranking(q, v, vis)
    assert set(fullv) == set(np.flatnonzero(vis))
    assert np.array_equal(dense.dense_prefix(q, v, 50, vis), fullv[:50])


def test_dense_topk_matches_library_topk():
    import torch
    w = datagen.workload("tiny", n=5000)
    x, _ = datagen.corpus(w)
    q, _ = datagen.queries(w, count=3)
    s = dense.scores64(q, x)
    for b in range(3):
        vals, _ = torch.topk(torch.from_numpy(s[b]), 20)
        got = dense.dense_prefix(q[b], x, 20)
        assert np.array_equal(s[b][got], vals.numpy())


def _tiny_index():
    # three terms; postings (doc, impact)
    post = {0: [(0, 1.0), (2, 3.0)], 1: [(1, 2.0), (2, 0.5)], 2: [(3, 0.0)]}
    term_ptr = [0]
    doc, imp = [], []
    for t in range(3):
        for d_, p in post[t]:
            doc.append(d_)
            imp.append(p)
        term_ptr.append(len(doc))
    return (np.array(term_ptr), np.array(doc, dtype=np.int32),
            np.array(imp, dtype=np.float32))


def test_sparse_tiny_hand_index():
    tp, doc, imp = _tiny_index()
    S = sparse.sparse_scores(tp, doc, imp, np.array([2, 0, 1]), np.array([1.0, 2.0, 1.0]), 5)
    assert list(S) == [2.0, 2.0, 6.5, 0.0, 0.0]
    # doc 3 has a posting but a zero score: outside the support set
    assert list(sparse.sparse_ranking(S)) == [2, 0, 1]


def test_sparse_sum_uses_ascending_term_order():
    # impacts 2^24, 1, 1 on one document: ascending-term float32 accumulation
    # gives fl(fl(2^24 + 1) + 1) = 2^24, any order adding the 1s first 2^24 + 2
    tp = np.array([0, 1, 2, 3])
    doc = np.array([0, 0, 0], dtype=np.int32)
    imp = np.array([2.0 ** 24, 1.0, 1.0], dtype=np.float32)
    S = sparse.sparse_scores(tp, doc, imp, np.array([2, 1, 0]), np.ones(3, np.float32), 1)
    assert S[0] == np.float32(2.0 ** 24)


def test_sparse_matches_per_document_loop():
    w = datagen.workload("tiny", n=3000)
    _, lab = datagen.corpus(w)
    docs = datagen.sparse_docs(w, lab)
    post = datagen.bm25_impacts(w, docs)
    _, qlab = datagen.queries(w, count=4)
    qs = datagen.sparse_queries(w, qlab)
    per_doc = {}
    for t in range(post.vocab):
        for p in range(post.term_ptr[t], post.term_ptr[t + 1]):
            per_doc.setdefault(int(post.doc[p]), {})[t] = post.impact[p]
    for terms, wts in qs:
        S = sparse.sparse_scores(post.term_ptr, post.doc, post.impact, terms, wts, w.n)
        for x in range(0, w.n, 7):
            acc = np.float32(0)
            for t, wt in sorted(zip(terms, wts)):
                acc = np.float32(acc + np.float32(wt * per_doc.get(x, {}).get(int(t), np.float32(0))))
            assert S[x] == acc
        r = sparse.sparse_ranking(S)
        assert np.all(S[r] > 0) and np.count_nonzero(S > 0) == len(r)
        assert all((S[a] > S[b]) or (S[a] == S[b] and a < b) for a, b in zip(r[:-1], r[1:]))


def test_sparse_visibility_zeroes_hidden_docs():
    tp, doc, imp = _tiny_index()
    vis = np.array([True, True, False, True, True])
    S = sparse.sparse_scores(tp, doc, imp, np.array([0, 1]), np.ones(2, np.float32), 5, vis)
    assert list(sparse.sparse_ranking(S)) == [1, 0]
