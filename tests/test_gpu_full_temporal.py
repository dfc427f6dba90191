"""Parity on temporal snapshots at full size: a base corpus of 4,000,000 x 768
clustered rows with sparse documents, then five snapshots, each deleting 10 %
of the visible rows and inserting 10 % new rows from drifted centres
(quantised on insert).  The same 100 queries run on every snapshot; every
query is checked against the oracle over that snapshot's visible rows,
with sparse statistics recomputed per snapshot (Sec. 2.1 visibility, Sec. 2.4
snapshots, Sec. 3.2)."""
import time

import numpy as np
import pytest

from paper_2608_07152_amd import datagen

from full_common import K, dense_read, load_library, note
from gpu_helpers import (check_dense_prefix, check_fusion_run, for_each_parallel, full_order,
                         row_norms64, score_matrix, scores64)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def E():
    return load_library()


@pytest.fixture(scope="module")
def temporal(E):
    t = time.time()
    w = datagen.workload("temporal")
    x0, lab0 = datagen.corpus(w)
    steps = list(datagen.temporal_steps(w, w.n))
    x = np.concatenate([x0] + [s.insert_rows for s in steps])
    del x0
    lab = np.concatenate([lab0] + [s.insert_labels for s in steps])
    docs = datagen.temporal_docs(w, lab, w.n)
    q, qlab = datagen.queries(w)
    qs = datagen.sparse_queries(w, qlab)
    vn = row_norms64(x)
    idx = E.pvs_build(x[:w.n])
    # visibility of every epoch over all physical rows
    vis = np.zeros(len(x), dtype=bool)
    vis[:w.n] = True
    epochs = [(0, vis.copy())]
    rows = w.n
    for s in steps:
        E.pvs_delete(idx, s.delete_ids)
        first = E.pvs_insert(idx, s.insert_rows)
        assert first == rows
        vis[s.delete_ids] = False
        vis[rows:rows + len(s.insert_rows)] = True
        rows += len(s.insert_rows)
        epochs.append((E.pvs_snapshot(idx), vis.copy()))
    note(f"temporal set up in {time.time() - t:.1f}s ({rows} physical rows)")
    yield w, x, vn, docs, q, qs, idx, epochs
    idx.free()


def test_temporal_snapshots_match_oracle(E, temporal):
    """Every query on every snapshot (S0 and the 500 runs of S1..S5)."""
    w, x, vn, docs, q, qs, idx, epochs = temporal
    t = time.time()
    S = score_matrix(q, x)          # a row's score does not depend on the snapshot
    note(f"temporal: oracle scores of {len(q)} queries over {len(x)} rows in {time.time() - t:.1f}s")
    for si, (epoch, vis) in enumerate(epochs):
        rows, _, n_vis = E.pvs_info(idx, epoch)
        assert n_vis == int(vis.sum())
        post = datagen.bm25_impacts(w, docs, vis)
        pbm = E.pbm_build(post.term_ptr, post.doc, post.impact, len(x), 4096)
        t = time.time()
        with E.RankRecorder() as rec:
            ids, cnt, stt, stats = E.eahr_topk(idx, pbm, q, qs, K=K, epoch=epoch)
        note(f"snapshot {si}: eahr_topk {time.time() - t:.2f}s")
        assert np.all(stt == 0) and np.all(cnt == K)

        def one(b):
            check_fusion_run(q[b], x, vn, post, qs[b], ids[b], cnt[b], stats[b], rec.ranks(b, 0),
                             rec.ranks(b, 1), (1, 1), S[b], full=full_order(S[b], vis), visible=vis, K=K)
            assert np.all(vis[ids[b]])

        t = time.time()
        for_each_parallel(one, range(len(q)))
        note(f"snapshot {si}: every query checked in {time.time() - t:.1f}s")
        pbm.free()


def test_temporal_state_survives_later_updates(E, temporal):
    """A state opened on an epoch keeps ranking that epoch after later
    deletes and inserts, and agrees with a state opened afterwards."""
    w, x, vn, docs, q, qs, idx, epochs = temporal
    epoch, vis = epochs[1]
    st = E.pvs_open(idx, q[:8], epoch=epoch)
    a, sa, _, _ = E.pvs_next(st, 500)
    E.pvs_delete(idx, np.flatnonzero(vis)[:1000])     # rows visible at that epoch
    E.pvs_insert(idx, x[:2000])                        # copies of old rows, new ids
    b_, sb, _, _ = E.pvs_next(st, 1500)
    st.close()
    got = np.concatenate([a, b_], axis=1)
    gsc = np.concatenate([sa, sb], axis=1)
    for j in (0, 5):
        s64 = scores64(q[j], x)
        check_dense_prefix(q[j], x, got[j], gsc[j], vis, s64=s64, vn=vn)
        di, ds = dense_read(E, idx, q[j], 2000, epoch)
        assert np.array_equal(di, got[j]) and np.array_equal(ds, gsc[j])
