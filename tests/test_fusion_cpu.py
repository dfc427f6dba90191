"""Host fusion of the library (eahr_fuse_lists, sparse-only eahr_topk) against
the oracle's complete-list weighted RRF and certification reference
(Sec. 2.1, 2.2, 3.4).  Host only."""
import json
import os

import numpy as np
import pytest

from oracle import certify, rrf
from oracle import sparse as osparse
from paper_2608_07152_amd import datagen, eahr

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("seed", range(40))
def test_fuse_lists_equals_complete_rrf(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 400))
    a = rng.permutation(n)
    kind = seed % 4
    if kind == 0:
        b = rng.permutation(n)[: int(rng.integers(0, n + 1))]
    elif kind == 1:
        b = a[::-1].copy()
    elif kind == 2:   # overlapping heads
        b = np.concatenate([a[:10][::-1], rng.permutation(a[10:])])
    else:
        b = a.copy()
    wts = [int(rng.integers(0, 3)), int(rng.integers(1, 3))]
    k = int(rng.choice([1, 2, 60]))
    K = int(rng.integers(1, 30))
    got, st = eahr.eahr_fuse_lists(a, b, K=K, k_rrf=k, w_dense=wts[0], w_sparse=wts[1],
                                   step=int(rng.choice([0, 1, 16])))
    want = rrf.rrf_topk([a, b], wts, k, K)
    assert list(got) == want
    assert st["resolved"] == 1


@pytest.mark.parametrize("seed", range(12))
def test_fuse_lists_stops_where_reference_first_resolves(seed):
    rng = np.random.default_rng(500 + seed)
    n = int(rng.integers(20, 120))
    a = rng.permutation(n)
    b = np.concatenate([a[:8][rng.permutation(8)], rng.permutation(a[8:])])
    K, step = 5, 4
    got, st = eahr.eahr_fuse_lists(a, b, K=K, step=step)
    d = step
    while True:
        A, ok = certify.certify_ref([a, b], [1, 1], 60, K, [d, d])
        if ok or d >= n:
            break
        d = min(n, d + step)
    assert st["dense_depth"] == min(d, n) and st["sparse_depth"] == min(d, n)
    assert list(got) == A


@pytest.mark.parametrize("relation", list(datagen.STREAM_RELATIONS))
def test_controlled_stream_instances(relation):
    # the controlled rank streams of Sec. 3.4 (3 sizes x 3 seeds per
    # relation, both lists advancing together, a check every 16 ranks):
    # correlated and all-tied streams first resolve at depth 32 at every
    # size, anti-correlated streams exhaust both lists (Sec. 4.2, pinned in
    # tests/golden), and every fused Top-20 is the complete-list RRF
    g = json.load(open(os.path.join(GOLDEN, "e5_controlled_streams.json")))
    assert list(datagen.STREAM_SIZES) == g["sizes"] and list(datagen.STREAM_SEEDS) == g["seeds"]
    for n in datagen.STREAM_SIZES:
        for seed in datagen.STREAM_SEEDS:
            a, b = datagen.controlled_streams(relation, n, seed)
            got, st = eahr.eahr_fuse_lists(a, b, K=g["K"], step=g["check_every"])
            if relation in ("correlated", "all_tied"):
                want = g["outcomes"]["correlated_32_block_permutation"]["first_resolved_depth"]
                assert st["dense_depth"] == want and st["sparse_depth"] == want
            if relation == "anti":
                assert st["dense_status"] == eahr.LIST_EXHAUSTED and st["sparse_status"] == eahr.LIST_EXHAUSTED
                assert st["dense_depth"] == n and st["sparse_depth"] == n
            else:
                assert st["dense_status"] == eahr.LIST_OPEN and st["sparse_status"] == eahr.LIST_OPEN
            assert st["dense_depth"] == st["sparse_depth"] and st["dense_depth"] % g["check_every"] == 0 \
                or st["dense_depth"] == n
            assert list(got) == rrf.rrf_topk([a, b], [1, 1], 60, g["K"]), (relation, n, seed)


def test_controlled_stream_generator_shapes():
    n = 5000
    for rel in datagen.STREAM_RELATIONS:
        a, b = datagen.controlled_streams(rel, n, 1729)
        assert sorted(a.tolist()) == list(range(n)) == sorted(b.tolist())
    a, b = datagen.controlled_streams("correlated", n, 1729)
    assert all(set(a[i:i + 32]) == set(b[i:i + 32]) for i in range(0, n, 32))
    a, b = datagen.controlled_streams("partial", n, 1729)
    assert len(set(a[:1000]) & set(b[:1000])) == 500
    assert set(b[:1000]) - set(a[:1000]) == set(a[1000:1500])
    rest = [x for x in a if x not in set(b[:1000])]
    assert list(b[1000:]) == rest
    a, b = datagen.controlled_streams("anti", n, 1729)
    assert np.array_equal(b, a[::-1])
    a, b = datagen.controlled_streams("all_tied", n, 1729)
    assert np.array_equal(a, np.arange(n)) and np.array_equal(b, np.arange(n))


def test_fuse_lists_no_padding_and_zero_weight():
    got, st = eahr.eahr_fuse_lists(np.arange(50), np.array([42, 7, 9]), K=20, w_dense=0)
    assert list(got) == [42, 7, 9]
    got, _ = eahr.eahr_fuse_lists(np.arange(50), np.array([42, 7, 9]), K=5, w_sparse=0)
    assert list(got) == [0, 1, 2, 3, 4]
    got, _ = eahr.eahr_fuse_lists(np.zeros(0, np.int64), np.zeros(0, np.int64), K=5)
    assert list(got) == []


def test_fuse_lists_weight_two_to_one():
    rng = np.random.default_rng(77)
    for _ in range(10):
        n = 300
        a = rng.permutation(n)
        b = np.concatenate([rng.permutation(a[:40]), rng.permutation(a[40:])])
        got, _ = eahr.eahr_fuse_lists(a, b, K=20, w_dense=2, w_sparse=1)
        assert list(got) == rrf.rrf_topk([a, b], [2, 1], 60, 20)


def test_fuse_lists_rejects_a_repeated_id():
    """A list that repeats an id is not a ranking (Sec. 2.1: each retriever
    ranks a set of distinct items)."""
    with pytest.raises(eahr.EahrError) as ei:
        eahr.eahr_fuse_lists(np.array([3, 1, 3, 0]), np.array([1, 0, 2]), K=2, depth0=2)
    assert ei.value.code == eahr.EAHR_E_INVALID


@pytest.mark.parametrize("seed", range(6))
def test_fuse_lists_one_list_closed_early(seed):
    """The sparse list ends long before the dense one: later dense ranks are
    joined against the closed list by id bitmap (Sec. 2.2 exhaustion: a closed
    list contributes its complete ranking)."""
    rng = np.random.default_rng(100 + seed)
    n = 20000
    a = rng.permutation(n)
    b = rng.choice(n, size=int(rng.integers(30, 300)), replace=False)
    for wts in ((1, 1), (2, 1), (1, 2)):
        got, st = eahr.eahr_fuse_lists(a, b, K=20, w_dense=wts[0], w_sparse=wts[1])
        assert list(got) == rrf.rrf_topk([a, b], list(wts), 60, 20)
    # a repeat in the open list after the other closed is still rejected
    bad = np.concatenate([a[:5000], a[100:101], a[5000:]])
    with pytest.raises(eahr.EahrError):
        eahr.eahr_fuse_lists(bad, b[:40], K=20, depth0=20)


def test_fuse_lists_deep_reads_after_the_other_list_closed():
    """The sparse list holds ids from the tail of the dense list, so the dense
    list is read far past the point where the sparse list closed; appends of
    that size are split over several host threads.  A repeat deep in the open
    list is still rejected."""
    rng = np.random.default_rng(11)
    n = 600_000
    a = rng.permutation(n)
    b = rng.permutation(a[n - 200_000:])[:3000]
    for wts in ((1, 1), (2, 1)):
        got, st = eahr.eahr_fuse_lists(a, b, K=20, w_dense=wts[0], w_sparse=wts[1])
        assert list(got) == rrf.rrf_topk([a, b], list(wts), 60, 20)
        assert st["dense_depth"] > 300_000
    bad = np.concatenate([a[:400_000], a[350_000:350_001], a[400_000:]])
    with pytest.raises(eahr.EahrError):
        eahr.eahr_fuse_lists(bad, b, K=20)


def test_fuse_lists_deep_reads_with_both_lists_open():
    """Two long partially overlapping lists read deep while both stay open:
    appends of that size sort, join and merge over several host threads.  A
    repeat deep in one list is still rejected."""
    rng = np.random.default_rng(12)
    n = 700_000
    a = rng.permutation(n)
    b = a.copy()
    for s0 in range(0, n, 50_000):
        b[s0:s0 + 50_000] = rng.permutation(b[s0:s0 + 50_000])
    b = np.concatenate([b[300_000:], b[:300_000]])
    for wts in ((1, 1), (2, 1)):
        got, st = eahr.eahr_fuse_lists(a, b, K=20, w_dense=wts[0], w_sparse=wts[1])
        assert list(got) == rrf.rrf_topk([a, b], list(wts), 60, 20)
        assert st["dense_depth"] > 200_000 and st["sparse_status"] == eahr.LIST_OPEN
    bad = np.concatenate([a[:250_000], a[200_000:200_001], a[250_000:]])
    with pytest.raises(eahr.EahrError):
        eahr.eahr_fuse_lists(bad, b, K=20)


def test_fuse_lists_concurrent_calls():
    """Several host threads call the fusion at once, each with appends long
    enough to be split over the shared worker threads (nested and concurrent
    use of the pool); every call returns its own exact result."""
    import threading
    rng = np.random.default_rng(13)
    cases = []
    for _ in range(4):
        n = 300_000
        a = rng.permutation(n)
        b = a.copy()
        for s0 in range(0, n, 30_000):
            b[s0:s0 + 30_000] = rng.permutation(b[s0:s0 + 30_000])
        b = np.concatenate([b[100_000:], b[:100_000]])
        cases.append((a, b))
    want = [rrf.rrf_topk([a, b], [1, 1], 60, 20) for a, b in cases]
    got = [None] * len(cases)

    def run(i):
        got[i] = list(eahr.eahr_fuse_lists(*cases[i], K=20)[0])

    ts = [threading.Thread(target=run, args=(i,)) for i in range(len(cases))]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    assert got == want


def test_fuse_lists_large_prefixes_equal_complete_rrf():
    """Deep prefixes (several table growths of the id bookkeeping): partially
    overlapping permutations of 200,000 ids."""
    rng = np.random.default_rng(5)
    n = 200_000
    a = rng.permutation(n)
    b = a.copy()
    blk = 5000
    for s0 in range(0, n, blk):
        b[s0:s0 + blk] = rng.permutation(b[s0:s0 + blk])
    b = np.concatenate([b[n // 2:], b[:n // 2]])
    for wts in ((1, 1), (2, 1)):
        got, st = eahr.eahr_fuse_lists(a, b, K=20, w_dense=wts[0], w_sparse=wts[1])
        assert list(got) == rrf.rrf_topk([a, b], list(wts), 60, 20)


def test_sparse_only_topk_through_eahr_topk():
    # the dense channel is not touched when its weight is 0 (no GPU needed)
    w = datagen.workload("tiny", n=5000)
    _, lab = datagen.corpus(w)
    post = datagen.bm25_impacts(w, datagen.sparse_docs(w, lab))
    _, qlab = datagen.queries(w, count=5)
    qs = datagen.sparse_queries(w, qlab)
    idx = eahr.pbm_build(post.term_ptr, post.doc, post.impact, w.n, 512)
    ids, cnt, stt, stats = eahr.eahr_topk(None, idx, None, qs, K=20, w_dense=0, w_sparse=1)
    for b, (t, wt) in enumerate(qs):
        S = osparse.sparse_scores(post.term_ptr, post.doc, post.impact, t, wt, w.n)
        want = list(osparse.sparse_ranking(S)[:20])
        assert list(ids[b, :cnt[b]]) == want
        assert stt[b] == 0


def test_unknown_dense_generator_rejected():
    import ctypes as C
    from paper_2608_07152_amd import eahr
    lib = eahr.load()
    prm = eahr._params(20, 60, 1, 1, 20, 2)
    prm.dense_generator = 9
    a = np.arange(10, dtype=np.int64)
    out = np.zeros(20, dtype=np.int64)
    cnt = C.c_int32()
    rc = lib.eahr_fuse_lists(a.ctypes.data_as(C.POINTER(C.c_int64)), 10,
                             a.ctypes.data_as(C.POINTER(C.c_int64)), 10, C.byref(prm), 0,
                             out.ctypes.data_as(C.POINTER(C.c_int64)), C.byref(cnt), None)
    assert rc == eahr.EAHR_E_INVALID


# ---------------------------------------------------------------------------
# Frozen scheduler (Sec. 3.5): an independent simulation of its rules, with the
# oracle's certification at every check, must stop at the same depths as the
# library, and the Top-K must be the complete-list RRF Top-K.

def _frozen_reference(a, b, w, k, K):
    from fractions import Fraction
    n = [len(a), len(b)]
    use = [w[0] > 0 and n[0] > 0, w[1] > 0 and n[1] > 0]
    d, skip, checks = [0, 0], [0, 0], 0

    def g(i, r):
        return Fraction(w[i], r + w[i] * (k - 1))

    while True:
        a0 = d[0] + d[1]
        target = a0 + min(1024, max(64, a0 // 8))
        stepped = False
        while True:
            can = [use[i] and d[i] < n[i] for i in range(2)]
            if not any(can):
                break
            if all(can):
                pick = 0 if g(0, d[0] + 1) >= g(1, d[1] + 1) else 1
                if skip[1 - pick] >= 16:
                    pick = 1 - pick
            else:
                pick = 0 if can[0] else 1
            d[pick] += min(16, n[pick] - d[pick])
            skip[pick] = 0
            if can[1 - pick]:
                skip[1 - pick] += 1
            stepped = True
            if d[pick] == n[pick]:
                break
            acc = d[0] + d[1]
            if a0 < 4 * K or acc <= 4 * K or acc >= target:
                break
        checks += 1
        A, ok = certify.certify_ref([a, b], w, k, K, list(d))
        if ok:
            return d, A, checks
        assert stepped, "complete lists must resolve"


def _stream_pair(kind, n, rng):
    a = rng.permutation(n)
    if kind == "independent":
        b = rng.permutation(n)
    elif kind == "block32":
        b = np.concatenate([rng.permutation(a[i:i + 32]) for i in range(0, n, 32)])
    elif kind == "reversed":
        b = a[::-1].copy()
    else:   # partial: the second list is a shuffled subset
        b = rng.permutation(a[: n * 3 // 4])
    return a.astype(np.int64), b.astype(np.int64)


@pytest.mark.parametrize("kind", ["independent", "block32", "reversed", "partial"])
@pytest.mark.parametrize("w", [(1, 1), (2, 1), (1, 3)])
def test_frozen_schedule_matches_independent_simulation(kind, w):
    # fixed seed per case (string hashing is randomised per process)
    seed = 1000 * ["independent", "block32", "reversed", "partial"].index(kind) + 10 * w[0] + w[1]
    rng = np.random.default_rng(seed)
    a, b = _stream_pair(kind, 1500, rng)
    d, A, checks = _frozen_reference(a.tolist(), b.tolist(), list(w), 60, 20)
    top, st = eahr.eahr_fuse_lists(a, b, K=20, k_rrf=60, w_dense=w[0], w_sparse=w[1], schedule="frozen")
    assert list(top) == rrf.rrf_topk([a.tolist(), b.tolist()], list(w), 60, 20)
    assert list(top) == list(A)
    assert (st["dense_depth"], st["sparse_depth"]) == (d[0], d[1])
    assert st["rounds"] == checks


def test_frozen_schedule_hand_worked_case():
    # identical lists, K = 2, weights 1:1, k = 60.  Check 1 after the first
    # step (dense 16 ranks, the tie goes to the dense list): items 0 and 1 are
    # seen by one list only, an unseen item could still lead, unresolved.
    # The access (16) is past 4K = 8, so the next check comes after
    # max(64, 16 / 8) more ranks: sparse 16 (g(1) > g(17)), dense 32 (tie at
    # rank 17), sparse 32, dense 48 -> access 80.  Check 2 resolves.
    a = np.arange(500, dtype=np.int64)
    top, st = eahr.eahr_fuse_lists(a, a, K=2, schedule="frozen")
    assert list(top) == [0, 1]
    assert (st["dense_depth"], st["sparse_depth"], st["rounds"]) == (48, 32, 2)


@pytest.mark.parametrize("K", [1, 3, 20])
def test_fuse_lists_exhausted_with_few_kept_both_seen_items(K):
    """Nearly reversed lists of 300,000 ids are both read to the end, and
    almost every id becomes seen by both lists in the last rounds (appends
    split over host threads).  Only the best K - |A| + 1 of them can still be
    fixed, so the fusion keeps those and drops the rest as they are found
    (Sec. 2.2).  At equal weights mirrored ranks give equal F, decided by id,
    and the heads tie until both lists end."""
    rng = np.random.default_rng(21 + K)
    n = 300_000
    a = rng.permutation(n)
    b = a[::-1].copy()
    swap = np.flatnonzero(rng.random(n // 2) < 0.5) * 2
    b[swap], b[swap + 1] = b[swap + 1].copy(), b[swap].copy()
    for wts in ((1, 1), (2, 1)):
        got, st = eahr.eahr_fuse_lists(a, b, K=K, w_dense=wts[0], w_sparse=wts[1])
        assert list(got) == rrf.rrf_topk([a, b], list(wts), 60, K)
        if wts == (1, 1):   # the mirrored heads tie until both lists end
            assert st["dense_status"] == eahr.LIST_EXHAUSTED and st["sparse_status"] == eahr.LIST_EXHAUSTED


def _fusion_modes_exe(tmp_path_factory):
    import shutil
    import subprocess
    if shutil.which("g++") is None:
        pytest.skip("needs g++")
    here = os.path.dirname(os.path.abspath(__file__))
    exe = tmp_path_factory.mktemp("fusion_modes") / "fusion_modes"
    subprocess.run(["g++", "-O2", "-std=c++17", "-pthread", "-I",
                    os.path.join(here, "..", "paper_2608_07152_amd", "csrc"),
                    os.path.join(here, "native", "fusion_modes.cpp"), "-o", str(exe)], check=True)
    return exe


@pytest.fixture(scope="module")
def fusion_modes(tmp_path_factory):
    return _fusion_modes_exe(tmp_path_factory)


def _run_modes(exe, tmp_path, a, b, K, wts, threads):
    import subprocess
    pa, pb = tmp_path / "a.bin", tmp_path / "b.bin"
    np.asarray(a, dtype=np.int64).tofile(pa)
    np.asarray(b, dtype=np.int64).tofile(pb)
    r = subprocess.run([str(exe), str(pa), str(pb), str(K), "60", str(wts[0]), str(wts[1]), str(threads)],
                       capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr
    out = r.stdout.split()
    if out == ["dup"]:
        return out, None
    return [int(x) for x in out], [int(x) for x in r.stderr.split()[1:3]]


@pytest.mark.parametrize("threads", [1, 8])
@pytest.mark.parametrize("closed", ["sparse", "dense"])
def test_fusion_reads_deep_after_one_list_closed(fusion_modes, tmp_path, threads, closed):
    """Depth doubling with the id range unknown (as eahr_topk runs it): one
    short list closes early and the other is read to depth 524,288 with the
    bitmaps, in parts by position over host threads when long; the fixed
    Top-K equals complete-list RRF (Sec. 2.1, 2.2), and a repeat deep in the
    open list is reported."""
    rng = np.random.default_rng(31)
    n = 600_000
    a = rng.permutation(n)
    short = rng.permutation(np.concatenate([a[n - 250_000:n - 247_000], rng.choice(a[:1000], 40, replace=False)]))
    for K, wts in ((20, (1, 1)), (5, (2, 1))):
        lists = (a, short) if closed == "sparse" else (short, a)
        got, depth = _run_modes(fusion_modes, tmp_path, *lists, K, wts, threads)
        assert got == rrf.rrf_topk(list(lists), list(wts), 60, K), (K, wts)
        long_side = 0 if closed == "sparse" else 1
        assert depth[1 - long_side] == len(short) and depth[long_side] > 300_000, depth
    bad = np.concatenate([a[:400_000], a[300_000:300_001], a[400_000:]])
    lists = (bad, short) if closed == "sparse" else (short, bad)
    assert _run_modes(fusion_modes, tmp_path, *lists, 20, (1, 1), threads)[0] == ["dup"]


@pytest.mark.parametrize("threads", [1, 8])
def test_fusion_closed_list_shares_most_ids(fusion_modes, tmp_path, threads):
    """A short list made of the long list's last ids, reversed: it closes
    first, and nearly every later rank of the long list is found in it, so
    each one's rank in the closed list is looked up (from the closed list's
    id bitmap and id order); the Top-K equals complete-list RRF."""
    rng = np.random.default_rng(33)
    n = 300_000
    a = rng.permutation(n)
    short = a[::-1][:120_000].copy()
    for K, wts in ((20, (1, 1)), (10, (1, 2))):
        got, depth = _run_modes(fusion_modes, tmp_path, a, short, K, wts, threads)
        assert got == rrf.rrf_topk([a, short], list(wts), 60, K), (K, wts)
        assert depth[1] == len(short) and depth[0] > n - len(short), depth


@pytest.mark.parametrize("threads", [1, 8])
def test_fusion_reads_deep_with_both_lists_open(fusion_modes, tmp_path, threads):
    """Both lists stay open while read deep: the id-order merges, split over
    host threads when long; the Top-K equals complete-list RRF."""
    rng = np.random.default_rng(32)
    n = 400_000
    a = rng.permutation(n)
    b = a.copy()
    for s0 in range(0, n, 40_000):
        b[s0:s0 + 40_000] = rng.permutation(b[s0:s0 + 40_000])
    b = np.concatenate([b[150_000:], b[:150_000]])
    got, depth = _run_modes(fusion_modes, tmp_path, a, b, 20, (1, 1), threads)
    assert got == rrf.rrf_topk([a, b], [1, 1], 60, 20)
    assert min(depth) > 100_000, depth
