"""Shared pieces of the full-size parity tests."""
import sys

import numpy as np  # noqa: F401

from oracle import sparse as osparse

from gpu_helpers import check_dense_prefix, fused_reference, hybrid_dense_list, scores64

K = 20


def note(msg):
    print(f"[full] {msg}", file=sys.stderr, flush=True)


def load_library():
    from paper_2608_07152_amd import eahr
    eahr.load()
    return eahr


def dense_read(E, idx, q, D, epoch=0):
    """The first D dense ranks of one query (a fresh single-query state)."""
    st = E.pvs_open(idx, q[None, :], epoch=epoch)
    ids, scs, cnt, _ = E.pvs_next(st, max(int(D), 1))
    st.close()
    return ids[0, :cnt[0]][:D], scs[0, :cnt[0]][:D]


def check_query(E, idx, x, vn, post, q, qs, got, stats, wts, visible=None, epoch=0, s64=None):
    """Dense prefix the fusion read, and the fused Top-K, against the oracle."""
    D = stats["dense_depth"]
    di, ds = dense_read(E, idx, q, D, epoch)
    assert len(di) == D
    if s64 is None:
        s64 = scores64(q, x)
    check_dense_prefix(q, x, di, ds, visible, s64=s64, vn=vn)
    S = osparse.sparse_scores(post.term_ptr, post.doc, post.impact, qs[0], qs[1], x.shape[0], visible)
    want = fused_reference(hybrid_dense_list(di, q, x, visible, s64=s64),
                           osparse.sparse_ranking(S), K, 60, wts)
    assert list(got) == want
    assert stats["resolved"] == 1
    return s64


