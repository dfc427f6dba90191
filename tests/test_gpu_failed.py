"""The failure rules of the dense channel, run through the normal code path
(App. A.1: PVS fails the request when an evaluated authoritative score lies
outside its interval, or the dimension is out of the guard's range; Sec. 2.1:
a Failed list invalidates the request).

EAHR_TEST_FAIL_QUERY=b makes the rescoring kernel judge query b's scores
against a zero-width interval around c, so the containment check itself
reports the violation; nothing on the GPU faults or stops early."""
import numpy as np
import pytest

from oracle import dense as odense
from oracle import rrf as orrf
from oracle import sparse as osparse
from paper_2608_07152_amd import datagen

from gpu_helpers import check_dense_prefix

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def E():
    from paper_2608_07152_amd import eahr
    eahr.load()
    return eahr


@pytest.fixture(scope="module")
def tiny():
    w = datagen.workload("tiny", n=6000)
    x, lab = datagen.corpus(w)
    q, qlab = datagen.queries(w, count=5)
    post = datagen.bm25_impacts(w, datagen.sparse_docs(w, lab))
    qs = datagen.sparse_queries(w, qlab)
    return w, x, q, post, qs


def _open_failing(E, idx, q, b, monkeypatch, **kw):
    monkeypatch.setenv("EAHR_TEST_FAIL_QUERY", str(b))
    try:
        return E.pvs_open(idx, q, **kw)
    finally:
        monkeypatch.delenv("EAHR_TEST_FAIL_QUERY")


def test_pvs_next_reports_failed_and_stays_failed(E, tiny, monkeypatch):
    w, x, q, _, _ = tiny
    idx = E.pvs_build(x)
    st = _open_failing(E, idx, q, 2, monkeypatch)
    ids, scs, cnt, stt = E.pvs_next(st, 20)
    assert stt[2] == E.LIST_FAILED and cnt[2] == 0
    for b in (0, 1, 3, 4):
        assert stt[b] == E.LIST_OPEN and cnt[b] == 20
        check_dense_prefix(q[b], x, ids[b, :20], scs[b, :20])
    ids2, scs2, cnt2, stt2 = E.pvs_next(st, 40)
    assert stt2[2] == E.LIST_FAILED and cnt2[2] == 0          # sticky
    for b in (0, 1, 3, 4):
        assert cnt2[b] == 40
        check_dense_prefix(q[b], x, np.concatenate([ids[b, :20], ids2[b, :40]]),
                           np.concatenate([scs[b, :20], scs2[b, :40]]))
    # a state opened without the knob is unaffected
    st2 = E.pvs_open(idx, q)
    _, _, cnt3, stt3 = E.pvs_next(st2, 20)
    assert np.all(stt3 == E.LIST_OPEN) and np.all(cnt3 == 20)


def test_eahr_topk_fails_only_that_query(E, tiny, monkeypatch):
    w, x, q, post, qs = tiny
    idx = E.pvs_build(x)
    pbm = E.pbm_build(post.term_ptr, post.doc, post.impact, w.n, 1024)
    monkeypatch.setenv("EAHR_TEST_FAIL_QUERY", "1")
    with pytest.raises(E.EahrError) as ei:
        E.eahr_topk(idx, pbm, q, qs, K=20)
    assert ei.value.code == E.EAHR_E_FAILED
    ids, cnt, stt, stats = E.eahr_topk(idx, pbm, q, qs, K=20, allow_failed=True)
    monkeypatch.delenv("EAHR_TEST_FAIL_QUERY")
    assert stt[1] == E.LIST_FAILED and cnt[1] == 0 and np.all(ids[1] == -1)
    assert stats[1]["dense_status"] == E.LIST_FAILED
    for b in (0, 2, 3, 4):
        assert stt[b] == 0
        dense_list = odense.dense_ranking(q[b], x)
        S = osparse.sparse_scores(post.term_ptr, post.doc, post.impact, qs[b][0], qs[b][1], w.n)
        want = orrf.rrf_topk([dense_list, osparse.sparse_ranking(S)], [1, 1], 60, 20)
        assert list(ids[b, :cnt[b]]) == want


def test_dimension_out_of_guard_range(E):
    # a_m < 1 and 127^2 d < 2^31 hold up to d = 4096 (App. A.1); beyond, the
    # build is refused before any device work
    x = np.ones((4, 4097), np.float32)
    with pytest.raises(E.EahrError) as ei:
        E.pvs_build(x)
    assert ei.value.code == E.EAHR_E_RANGE
    idx = E.pvs_build(np.ones((4, 4096), np.float32))
    assert E.pvs_info(idx)[1] == 4096
