"""GPU parity of the PVS dense channel against the CPU oracle, through the C ABI
(Sec. 2.3.1, App. A.1)."""
import numpy as np
import pytest

from oracle import dense as odense
from oracle import pvs as opvs
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
    w = datagen.workload("tiny")
    x, lab = datagen.corpus(w)
    q, qlab = datagen.queries(w)
    return w, x, q


@pytest.fixture(scope="module")
def tiny_index(E, tiny):
    w, x, q = tiny
    return E.pvs_build(x)


def _ulp_diff(a, b):
    a = np.asarray(a, np.float32).view(np.int32).astype(np.int64)
    b = np.asarray(b, np.float32).view(np.int32).astype(np.int64)
    return np.abs(a - b)


def test_codes_and_scales_bit_exact(E, tiny, tiny_index):
    w, x, q = tiny
    codes, meta = E.pvs_read_index(tiny_index, 0, w.n)
    ref = opvs.quantize(x)
    assert np.array_equal(codes, ref.z)
    assert np.array_equal(meta[:, 0], ref.s)
    assert np.all(_ulp_diff(meta[:, 1], ref.norm) <= 1)
    assert np.all(_ulp_diff(meta[:, 2], ref.enorm) <= 1)


def test_codes_bit_exact_on_hard_inputs(E):
    rng = np.random.default_rng(12)
    d = 100                     # not a multiple of 16: padded chunks
    x = (rng.standard_cauchy((300, d)) * 10.0 ** rng.integers(-30, 30, size=(300, 1))).astype(np.float32)
    x[3] = 0
    x[4, :] = 0
    x[4, 7] = np.float32(1e-45)
    s = np.float32(2.0 ** -7)
    x[5, :8] = np.array([127, 0.5, -0.5, 2.5, -2.5, 0.49999997, -126.5, 1], np.float32) * s
    idx = E.pvs_build(x)
    codes, meta = E.pvs_read_index(idx, 0, 300)
    ref = opvs.quantize(x)
    assert np.array_equal(codes, ref.z)
    assert np.array_equal(meta[:, 0], ref.s)
    assert np.all(_ulp_diff(meta[:, 1], ref.norm) <= 1)


def test_query_encoding_bit_exact(E, tiny, tiny_index):
    w, x, q = tiny
    st = E.pvs_open(tiny_index, q)
    codes, meta = E.pvs_read_query(st)
    ref = opvs.quantize(q)
    assert np.array_equal(codes, ref.z)
    assert np.array_equal(meta[:, 0], ref.s)
    assert np.all(_ulp_diff(meta[:, 1], ref.norm) <= 1)
    assert np.all(_ulp_diff(meta[:, 2], ref.hnorm) <= 1)
    assert np.all(_ulp_diff(meta[:, 3], ref.enorm) <= 1)


def test_intervals_match_oracle_and_contain_scores(E, tiny, tiny_index):
    w, x, q = tiny
    st = E.pvs_open(tiny_index, q[:3])
    rows = np.arange(w.n)
    ref = opvs.intervals(opvs.quantize(q[:3]), opvs.quantize(x), w.d)
    s64 = odense.scores64(q[:3], x)
    for b in range(3):
        lo, hi = E.pvs_intervals(st, b, rows)
        s32 = E.pvs_scores(st, b, rows)
        assert np.all(_ulp_diff(lo, ref.lo[b]) <= 2) and np.all(_ulp_diff(hi, ref.hi[b]) <= 2)
        assert np.mean(lo == ref.lo[b]) > 0.99
        assert np.all(lo <= s64[b]) and np.all(s64[b] <= hi)
        assert np.all(lo <= s32) and np.all(s32 <= hi)


def test_rescored_scores_close_to_fp64(E, tiny, tiny_index):
    w, x, q = tiny
    st = E.pvs_open(tiny_index, q)
    s64 = odense.scores64(q, x)
    for b in range(len(q)):
        s32 = E.pvs_scores(st, b, np.arange(w.n))
        assert np.max(np.abs(s32 - s64[b])) < 1e-6


def _drain(E, st, schedule):
    B = st.B
    ids = [[] for _ in range(B)]
    scs = [[] for _ in range(B)]
    last = None
    for m in schedule:
        i, s, c, stt = E.pvs_next(st, m)
        for b in range(B):
            assert c[b] == m or stt[b] == E.LIST_EXHAUSTED
            ids[b].extend(i[b, :c[b]].tolist())
            scs[b].extend(s[b, :c[b]].tolist())
        last = stt
    return ids, scs, last


def test_pvs_next_prefix_parity_tiny(E, tiny, tiny_index):
    w, x, q = tiny
    st = E.pvs_open(tiny_index, q)
    ids, scs, stt = _drain(E, st, [20, 20, 40, 80, 160, 320, 640, 1280])
    for b in range(len(q)):
        assert len(ids[b]) == 2560
        check_dense_prefix(q[b], x, ids[b], scs[b])
    assert np.all(stt == E.LIST_OPEN)


def test_self_consistency_with_full_scan(E, tiny, tiny_index):
    """Concatenated pvs_next output equals the (s32 desc, id asc) sort of the
    authoritative score of every row, bit for bit."""
    w, x, q = tiny
    st = E.pvs_open(tiny_index, q[:4])
    ids, scs, _ = _drain(E, st, [7, 13, 100, 900, 3000])
    for b in range(4):
        s32 = E.pvs_scores(st, b, np.arange(w.n)).astype(np.float64) + 0.0
        order = np.lexsort((np.arange(w.n), -s32))[: len(ids[b])]
        assert np.array_equal(np.array(ids[b]), order)
        assert np.array_equal(np.array(scs[b], np.float32), s32[order].astype(np.float32))


def test_split_calls_equal_one_call(E, tiny, tiny_index):
    w, x, q = tiny
    a = E.pvs_open(tiny_index, q)
    b = E.pvs_open(tiny_index, q)
    ia, sa, _ = _drain(E, a, [1, 3, 37, 259])
    ib, sb, _ = _drain(E, b, [300])
    assert ia == ib and sa == sb


def test_batch_size_does_not_change_results(E, tiny, tiny_index):
    w, x, q = tiny
    batch = E.pvs_open(tiny_index, q)
    ib, sb, _ = _drain(E, batch, [50, 500])
    for j in (0, 5):
        one = E.pvs_open(tiny_index, q[j:j + 1])
        i1, s1, _ = _drain(E, one, [50, 500])
        assert i1[0] == ib[j] and s1[0] == sb[j]


def test_active_mask_leaves_others_untouched(E, tiny, tiny_index):
    w, x, q = tiny
    st = E.pvs_open(tiny_index, q[:3])
    i0, _, c0, _ = E.pvs_next(st, 10, active=[1, 0, 1])
    assert c0[1] == 0 and c0[0] == 10
    i1, _, _, _ = E.pvs_next(st, 10)
    ref = E.pvs_open(tiny_index, q[1:2])
    ir, _, _, _ = E.pvs_next(ref, 10)
    assert np.array_equal(i1[1], ir[0])


def test_exhaustion_small_corpus(E):
    w = datagen.workload("tiny", n=3001)
    x, _ = datagen.corpus(w)
    q, _ = datagen.queries(w, count=3)
    idx = E.pvs_build(x)
    st = E.pvs_open(idx, q)
    ids, scs, stt = _drain(E, st, [20, 40, 80, 160, 320, 640, 1280, 2560])
    assert np.all(stt == E.LIST_EXHAUSTED)
    for b in range(3):
        assert sorted(ids[b]) == list(range(3001))
        check_dense_prefix(q[b], x, ids[b], scs[b])
    i, s, c, stt2 = E.pvs_next(st, 5)
    assert np.all(c == 0) and np.all(stt2 == E.LIST_EXHAUSTED)


def test_all_tied_corpus_is_identifier_order(E):
    x = np.tile(np.array([[0.25, -0.5, 1.0, 0.125]], np.float32), (700, 1))
    idx = E.pvs_build(x)
    st = E.pvs_open(idx, np.array([[1.0, 2.0, 3.0, 4.0]], np.float32))
    ids, _, stt = _drain(E, st, [10, 690, 5])
    assert ids[0] == list(range(700))
    assert stt[0] == E.LIST_EXHAUSTED


def test_zero_query_and_zero_rows(E):
    rng = np.random.default_rng(0)
    x = rng.standard_normal((200, 32)).astype(np.float32)
    x[::3] = 0
    idx = E.pvs_build(x)
    st = E.pvs_open(idx, np.zeros((1, 32), np.float32))
    ids, scs, stt = _drain(E, st, [200])
    assert ids[0] == list(range(200)) and set(scs[0]) == {0.0}


def test_snapshots_and_visibility(E):
    w = datagen.workload("tiny", n=4000)
    x, _ = datagen.corpus(w)
    q, _ = datagen.queries(w, count=2)
    idx = E.pvs_build(x)
    st0 = E.pvs_open(idx, q, epoch=0)
    first0, _, _, _ = E.pvs_next(st0, 30)
    dels = np.unique(first0[:, :10].ravel())
    E.pvs_delete(idx, dels)
    extra = datagen.workload("tiny", n=500)
    xi, _ = datagen.queries(extra, count=500)     # new rows from another stream
    fid = E.pvs_insert(idx, xi)
    assert fid == 4000
    e1 = E.pvs_snapshot(idx)
    rows, d, vis = E.pvs_info(idx, e1)
    assert rows == 4500 and vis == 4500 - len(dels)
    # the old state is unchanged by later updates
    more0, _, _, _ = E.pvs_next(st0, 100)
    ref = E.pvs_open(E.pvs_build(x), q)
    r0, _, _, _ = E.pvs_next(ref, 130)
    assert np.array_equal(np.concatenate([first0, more0], axis=1), r0)
    # the new epoch hides deleted rows and ranks inserted ones
    allx = np.concatenate([x, xi])
    visible = np.ones(4500, bool)
    visible[dels] = False
    st1 = E.pvs_open(idx, q, epoch=e1)
    ids, scs, _ = _drain(E, st1, [200])
    for b in range(2):
        check_dense_prefix(q[b], allx, ids[b], scs[b], visible)
    codes, meta = E.pvs_read_index(idx, 4000, 500)
    ref_q = opvs.quantize(xi)
    assert np.array_equal(codes, ref_q.z) and np.array_equal(meta[:, 0], ref_q.s)


def test_nonfinite_inputs_rejected(E):
    x = np.ones((10, 8), np.float32)
    x[3, 2] = np.nan
    with pytest.raises(E.EahrError) as ei:
        E.pvs_build(x)
    assert ei.value.code == E.EAHR_E_NONFINITE
    idx = E.pvs_build(np.ones((10, 8), np.float32))
    qq = np.ones((2, 8), np.float32)
    qq[1, 0] = np.inf
    with pytest.raises(E.EahrError) as ei:
        E.pvs_open(idx, qq)
    assert ei.value.code == E.EAHR_E_NONFINITE


def _open_with_path(E, idx, q, path, monkeypatch):
    monkeypatch.setenv("EAHR_SCAN_PATH", path)
    st = E.pvs_open(idx, q)
    monkeypatch.delenv("EAHR_SCAN_PATH")
    return st


@pytest.mark.parametrize("B", [1, 5, 40, 100, 300])
def test_mfma_and_gemv_scans_agree(E, tiny, tiny_index, monkeypatch, B):
    """The Int8 MFMA scan (query tiles of 32, passes of 256) and the dot4 GEMV
    scan produce the same ranks, bit for bit."""
    w, x, q = tiny
    qb, _ = datagen.queries(datagen.workload("tiny"), count=B)
    a = _open_with_path(E, tiny_index, qb, "mfma", monkeypatch)
    g = _open_with_path(E, tiny_index, qb, "gemv", monkeypatch)
    ia, sa, _ = _drain(E, a, [20, 300])
    ig, sg, _ = _drain(E, g, [20, 300])
    assert ia == ig and sa == sg
    for b in range(0, B, max(1, B // 4)):
        check_dense_prefix(qb[b], x, ia[b], sa[b])


@pytest.mark.parametrize("path", ["gemv", "mfma"])
def test_overflowing_pools_are_scanned_again(E, tiny, tiny_index, monkeypatch, path):
    """Key regions and the candidate pool sized far too small on the first
    attempt (a test knob): the records past a sub-region's end are dropped,
    every query is scanned again with room, and the ranks are bit-equal to an
    unconstrained run."""
    w, x, q = tiny
    qb, _ = datagen.queries(datagen.workload("tiny"), count=70)
    ref = _open_with_path(E, tiny_index, qb, path, monkeypatch)
    ir, sr, _ = _drain(E, ref, [20, 300])
    monkeypatch.setenv("EAHR_CAP_SHRINK", "64")
    st = _open_with_path(E, tiny_index, qb, path, monkeypatch)
    monkeypatch.delenv("EAHR_CAP_SHRINK")
    ig, sg, _ = _drain(E, st, [20, 300])
    assert ig == ir and sg == sr
    assert E.pvs_stats(st)["overflows"] > 0 and E.pvs_stats(ref)["overflows"] == 0


def test_single_hip_runtime_in_process(E):
    import re
    maps = open("/proc/self/maps").read()
    assert len(set(re.findall(r"\S*libamdhip64\S*", maps))) == 1
    assert "libeahr.so" in maps


def test_device_pointer_inputs(E, tiny):
    import torch
    w, x, q = tiny
    xd = torch.from_numpy(x).cuda()
    qd = torch.from_numpy(q).cuda()
    idx = E.pvs_build(xd)
    st = E.pvs_open(idx, qd)
    i, s, c, _ = E.pvs_next(st, 50)
    ref = E.pvs_open(E.pvs_build(x), q)
    ir, sr, _, _ = E.pvs_next(ref, 50)
    assert np.array_equal(i, ir) and np.array_equal(s, sr)


def test_index_freed_before_its_states(E, tiny):
    # the library defers the release of an index until its last state is
    # closed, so finalisation order (e.g. Python's cyclic GC) does not matter
    w, x, q = tiny
    idx = E.pvs_build(x[:3000])
    st = E.pvs_open(idx, q[:2])
    ids, scs, cnt, _ = E.pvs_next(st, 10)
    h = idx.h
    E.load().pvs_free(h)
    idx.h = None
    ids2, _, cnt2, _ = E.pvs_next(st, 10)          # the state still works
    assert np.all(cnt2 == 10)
    st.close()
    mg_idx = [E.pvs_build(x[:100]), E.pvs_build(x[100:200])]
    mg = E.pvs_merge_open(mg_idx, [np.arange(100), np.arange(100, 200)], q[:2])
    for i in mg_idx:
        i.free()
    _, _, c, _ = E.pvs_merge_next(mg, 5)
    assert np.all(c == 5)
    mg.close()


@pytest.fixture(scope="module", params=[384, 768], ids=["d384", "d768"])
def wide_d(request, E):
    # dimensions with an unrolled single-pass MFMA kernel (12 and 24 K steps);
    # 230,000 rows: 7,188 half-blocks, so each of the 2,048 wavefronts of a
    # full grid takes three or four (its code ring runs on into the next
    # half-block), and a ragged last block
    w = datagen.workload("tiny", n=230_000, d=request.param, centers=64)
    x, _ = datagen.corpus(w)
    return w, x, E.pvs_build(x)


@pytest.mark.parametrize("B", [40, 130, 256, 300])
def test_single_pass_mfma_scan_agrees(E, wide_d, monkeypatch, B):
    """The single-pass MFMA scan (query fragments resident in LDS, 4 or 8
    tiles, two of them from L2 at d = 768), the older wide MFMA kernel and
    the dot4 GEMV scan produce the same ranks and scores, bit for bit, and
    the prefixes are the oracle's."""
    w, x, idx = wide_d
    qb, _ = datagen.queries(w, count=B)
    runs = {}
    for kern in ("lds", "wide"):
        if kern == "wide":
            monkeypatch.setenv("EAHR_MFMA_KERNEL", "wide")
        st = _open_with_path(E, idx, qb, "mfma", monkeypatch)
        runs[kern] = _drain(E, st, [20, 500])[:2]
        monkeypatch.delenv("EAHR_MFMA_KERNEL", raising=False)
    g = _open_with_path(E, idx, qb, "gemv", monkeypatch)
    runs["gemv"] = _drain(E, g, [20, 500])[:2]
    assert runs["lds"] == runs["wide"] == runs["gemv"]
    ia, sa = runs["lds"]
    for b in range(0, B, max(1, B // 5)):
        check_dense_prefix(qb[b], x, ia[b], sa[b])


def test_single_pass_mfma_scan_with_deletes(E, monkeypatch):
    # 200,000 rows: several half-blocks per wavefront
    w = datagen.workload("tiny", n=200_000, d=768, centers=16)
    x, _ = datagen.corpus(w)
    idx = E.pvs_build(x)
    rng = np.random.default_rng(3)
    dels = np.sort(rng.choice(w.n, 33_000, replace=False))
    E.pvs_delete(idx, dels)
    e1 = E.pvs_snapshot(idx)
    visible = np.ones(w.n, bool)
    visible[dels] = False
    qb, _ = datagen.queries(w, count=200)
    # invisible rows inside blocks and half-blocks (epoch 1)
    a = E.pvs_open(idx, qb, epoch=e1)
    ia, sa, _ = _drain(E, a, [20, 400])
    for b in range(0, 200, 37):
        check_dense_prefix(qb[b], x, ia[b], sa[b], visible)
