"""GPU parity of the global-scale scalar-quantisation generator (the
alternative to PVS in Sec. 4.4, Table 4-1) against the CPU oracle, through
the C ABI.  Both generators emit exact ranks, so their outputs must also be
identical to each other; they differ only in how many pairs are rescored."""
import numpy as np
import pytest

from oracle import dense as odense
from oracle import pvs as opvs
from oracle import sparse as osparse
from paper_2608_07152_amd import datagen

from gpu_helpers import check_dense_prefix, fused_reference, hybrid_dense_list

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def E():
    from paper_2608_07152_amd import eahr
    eahr.load()
    return eahr


@pytest.fixture(scope="module")
def tiny(E):
    w = datagen.workload("tiny")
    x, lab = datagen.corpus(w)
    q, qlab = datagen.queries(w)
    return w, x, q, lab, qlab


@pytest.fixture(scope="module")
def both(E, tiny):
    w, x, q, _, _ = tiny
    return E.pvs_build(x), E.pvs_build_quant(x, "global")


def _ulp_diff(a, b):
    a = np.asarray(a, np.float32).view(np.int32).astype(np.int64)
    b = np.asarray(b, np.float32).view(np.int32).astype(np.int64)
    return np.abs(a - b)


def _drain(E, st, schedule):
    ids = [[] for _ in range(st.B)]
    scs = [[] for _ in range(st.B)]
    for m in schedule:
        i, s, c, stt = E.pvs_next(st, m)
        for b in range(st.B):
            assert c[b] == m or stt[b] == E.LIST_EXHAUSTED
            ids[b].extend(i[b, :c[b]].tolist())
            scs[b].extend(s[b, :c[b]].tolist())
    return ids, scs


def test_global_codes_bit_exact(E, tiny, both):
    w, x, q, _, _ = tiny
    codes, meta = E.pvs_read_index(both[1], 0, w.n)
    ref = opvs.quantize_global(x)
    assert np.array_equal(codes, ref.z)
    assert np.array_equal(meta[:, 0], ref.s)
    assert np.all(_ulp_diff(meta[:, 1], ref.norm) <= 1)
    assert np.all(_ulp_diff(meta[:, 2], ref.enorm) <= 1)


def test_global_codes_bit_exact_on_hard_inputs(E):
    rng = np.random.default_rng(21)
    d = 100                                   # padded chunks
    x = (rng.standard_cauchy((500, d)) * 10.0 ** rng.integers(-3, 3, size=(500, 1))).astype(np.float32)
    x[7] = 0
    idx = E.pvs_build_quant(x, "global")
    codes, meta = E.pvs_read_index(idx, 0, 500)
    ref = opvs.quantize_global(x)
    assert np.array_equal(codes, ref.z)
    assert np.array_equal(meta[:, 0], ref.s)
    assert np.all(_ulp_diff(meta[:, 2], ref.enorm) <= 1)


def test_global_intervals_match_oracle(E, tiny, both):
    w, x, q, _, _ = tiny
    st = E.pvs_open(both[1], q[:3])
    rows = np.arange(w.n)
    ref = opvs.intervals(opvs.quantize(q[:3]), opvs.quantize_global(x), w.d)
    s64 = odense.scores64(q[:3], x)
    for b in range(3):
        lo, hi = E.pvs_intervals(st, b, rows)
        assert np.all(_ulp_diff(lo, ref.lo[b]) <= 2) and np.all(_ulp_diff(hi, ref.hi[b]) <= 2)
        assert np.all(lo <= s64[b]) and np.all(s64[b] <= hi)


@pytest.mark.parametrize("B", [8, 64])   # GEMV scan, then the Int8 MFMA scans
def test_global_prefixes_match_oracle_and_pvs(E, tiny, both, B):
    w, x, _, _, _ = tiny
    q, _ = datagen.queries(w, count=B)
    schedule = [20, 20, 40, 80, 160, 320, 640]
    got_v, sc_v = _drain(E, E.pvs_open(both[0], q), schedule)
    got_g, sc_g = _drain(E, E.pvs_open(both[1], q), schedule)
    for b in range(B):
        assert got_g[b] == got_v[b], b
        assert sc_g[b] == sc_v[b], b
    for b in range(0, B, max(1, B // 8)):
        check_dense_prefix(q[b], x, got_g[b], sc_g[b])


def test_global_rescores_more_pairs_than_pvs(E, tiny, both):
    # Sec. 4.4: per-vector scales give tighter intervals, so fewer float32
    # evaluations (compared on the same queries and depth; a ballpark, not a
    # bound, hence the generous margin)
    w, x, q, _, _ = tiny
    cands = []
    for idx in both:
        st = E.pvs_open(idx, q)
        E.pvs_next(st, 200)
        cands.append(E.pvs_stats(st)["candidates"])
    assert cands[1] >= cands[0] * 0.9


def test_global_eahr_topk_matches_complete_rrf(E, tiny, both):
    w, x, q, lab, qlab = tiny
    post = datagen.bm25_impacts(w, datagen.sparse_docs(w, lab))
    qs = datagen.sparse_queries(w, qlab)
    pbm = E.pbm_build(post.term_ptr, post.doc, post.impact, w.n, 1024)
    ids_v, cnt_v, _, _ = E.eahr_topk(both[0], pbm, q, qs, K=20)
    ids_g, cnt_g, stt, stats = E.eahr_topk(both[1], pbm, q, qs, K=20)
    assert np.all(stt == 0)
    assert np.array_equal(ids_g, ids_v) and np.array_equal(cnt_g, cnt_v)
    for b in range(len(q)):
        D = stats[b]["dense_depth"]
        di, ds, _, _ = E.pvs_next(E.pvs_open(both[1], q[b:b + 1]), max(D, 1))
        check_dense_prefix(q[b], x, di[0, :D], ds[0, :D])
        S = osparse.sparse_scores(post.term_ptr, post.doc, post.impact, qs[b][0], qs[b][1], w.n)
        want = fused_reference(hybrid_dense_list(di[0, :D], q[b], x), osparse.sparse_ranking(S), 20)
        assert list(ids_g[b, :cnt_g[b]]) == want, b


def test_global_scale_fixed_by_first_insert_and_clipping(E):
    w = datagen.workload("tiny", n=3000, d=64)
    x, _ = datagen.corpus(w)
    q, _ = datagen.queries(w, count=4)
    idx = E.pvs_build_quant(np.zeros((0, w.d), np.float32), "global")
    first = E.pvs_insert(idx, x[:2000])
    assert first == 0
    s = opvs.quantize_global(x[:2000]).s[0]
    big = (x[2000:] * np.float32(3.0)).astype(np.float32)   # beyond 127 s: codes clip
    E.pvs_insert(idx, big)
    epoch = E.pvs_snapshot(idx)
    codes, meta = E.pvs_read_index(idx, 0, 3000)
    ref_a = opvs.quantize_global(x[:2000])
    ref_b = opvs.quantize_global(big, scale=s)
    assert np.array_equal(codes[:2000], ref_a.z) and np.array_equal(codes[2000:], ref_b.z)
    assert np.all(meta[:, 0] == s)
    assert np.any(np.abs(ref_b.z.astype(np.int32)) == 127)
    corpus = np.concatenate([x[:2000], big])
    st = E.pvs_open(idx, q, epoch=epoch)
    ids, scs = _drain(E, st, [20, 40, 200])
    for b in range(len(q)):
        check_dense_prefix(q[b], corpus, ids[b], scs[b])


def test_unknown_quantisation_mode_rejected(E):
    import ctypes as C
    lib = E.load()
    h = C.c_void_p()
    x = np.ones((4, 8), np.float32)
    rc = lib.pvs_build_quant(x.ctypes.data_as(C.c_void_p), 4, 8, 0, None, 7, C.byref(h))
    assert rc == E.EAHR_E_INVALID and not h.value


# ---------------------------------------------------------------------------
# Exhaustive float32 scan generator (the other alternative of Table 4-1)

def test_full_scan_prefixes_equal_interval_generator(E, tiny, both):
    w, x, q, _, _ = tiny
    schedule = [20, 20, 40, 80, 160, 320, 640]
    got_i, sc_i = _drain(E, E.pvs_open(both[0], q), schedule)
    st = E.pvs_open(both[0], q, generator="full_scan")
    got_f, sc_f = _drain(E, st, schedule)
    for b in range(len(q)):
        assert got_f[b] == got_i[b], b
        assert sc_f[b] == sc_i[b], b
        check_dense_prefix(q[b], x, got_f[b], sc_f[b])
    c = E.pvs_stats(st)
    assert c["candidates"] == w.n * len(q) and c["scans"] == len(q)


def test_full_scan_to_exhaustion_with_deletes(E):
    w = datagen.workload("tiny", n=3000, d=64)
    x, _ = datagen.corpus(w)
    q, _ = datagen.queries(w, count=3)
    idx = E.pvs_build(x)
    gone = np.arange(5, 3000, 7)
    E.pvs_delete(idx, gone)
    epoch = E.pvs_snapshot(idx)
    vis = np.ones(3000, bool)
    vis[gone] = False
    st = E.pvs_open(idx, q, epoch=epoch, generator="full_scan")
    ids, scs = _drain(E, st, [100, 1000, 5000])
    ref, _ = _drain(E, E.pvs_open(idx, q, epoch=epoch), [100, 1000, 5000])
    for b in range(3):
        assert len(ids[b]) == int(vis.sum())
        assert ids[b] == ref[b]
        check_dense_prefix(q[b], x, ids[b], scs[b], visible=vis)
    _, _, c, stt = E.pvs_next(st, 10)
    assert np.all(c == 0) and np.all(stt == E.LIST_EXHAUSTED)


def test_full_scan_eahr_topk_equals_intervals(E, tiny, both):
    w, x, q, lab, qlab = tiny
    post = datagen.bm25_impacts(w, datagen.sparse_docs(w, lab))
    qs = datagen.sparse_queries(w, qlab)
    pbm = E.pbm_build(post.term_ptr, post.doc, post.impact, w.n, 1024)
    for wts in ((1, 1), (2, 1)):
        a = E.eahr_topk(both[0], pbm, q, qs, K=20, w_dense=wts[0], w_sparse=wts[1])
        f = E.eahr_topk(both[0], pbm, q, qs, K=20, w_dense=wts[0], w_sparse=wts[1],
                        dense_generator="full_scan")
        assert np.all(f[2] == 0)
        assert np.array_equal(a[0], f[0]) and np.array_equal(a[1], f[1])


def test_full_scan_anticorrelated_exhausts_both(E):
    w = datagen.workload("adv", n=3000, d=64)
    x, _ = datagen.corpus(w)
    q, _ = datagen.queries(w, count=2)
    post, qs = datagen.adversarial_postings(w, x, q)
    idx = E.pvs_build(x)
    pbm = E.pbm_build(post.term_ptr, post.doc, post.impact, w.n, 256)
    a = E.eahr_topk(idx, pbm, q, qs, K=20)
    f = E.eahr_topk(idx, pbm, q, qs, K=20, dense_generator="full_scan")
    assert np.array_equal(a[0], f[0])
    for b in range(2):
        assert f[3][b]["dense_depth"] == w.n and f[3][b]["sparse_depth"] == w.n
        S = osparse.sparse_scores(post.term_ptr, post.doc, post.impact, qs[b][0], qs[b][1], w.n)
        di, ds, _, _ = E.pvs_next(E.pvs_open(idx, q[b:b + 1], generator="full_scan"), w.n)
        check_dense_prefix(q[b], x, di[0], ds[0])
        want = fused_reference(hybrid_dense_list(di[0], q[b], x), osparse.sparse_ranking(S), 20)
        assert list(f[0][b, :f[1][b]]) == want


def test_unknown_generator_rejected(E, tiny, both):
    import ctypes as C
    w, x, q, _, _ = tiny
    lib = E.load()
    h = C.c_void_p()
    qq = np.ascontiguousarray(q[:1])
    rc = lib.pvs_open_gen(both[0].h, 0, qq.ctypes.data_as(C.c_void_p), 1, 0, 9, C.byref(h))
    assert rc == E.EAHR_E_INVALID and not h.value
