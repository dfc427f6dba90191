"""Seeded synthetic workloads for hybrid dense + sparse retrieval.

This module only *draws* inputs: clustered unit vectors, documents made of terms,
BM25-style impacts and queries.  It holds none of the retrieval method's own
arithmetic (no quantisation, no score intervals, no ranking, no fusion), so the
GPU path and the CPU oracle can both read what it produces without sharing any
of the method's code.

Every array is addressed by (workload, stream, chunk) and regenerated bit for bit
from ``numpy.random.SeedSequence(1729, spawn_key=(workload_id, stream, chunk))``,
independent of how many worker processes produce it.

Workload recipe (the paper gives the collection sizes and BM25 parameters; the
rest are readings stated here):

* dense: ``C`` centres ``~ N(0, I_d)``; each row picks a centre uniformly and is
  ``normalize_fp64(centre + std * N(0, I_d))`` cast to float32.  Queries are
  drawn the same way from their own stream.
* sparse: document length ``max(1, Poisson(L))``; each token is, with
  probability 1/2, a truncated Zipf(1.1) draw over the vocabulary (rank mapped
  to a term id through a seeded permutation) and otherwise a uniform draw from
  the 200-term topic vocabulary of the document's cluster.  Impacts are
  Lucene-form BM25 with k1 = 0.9, b = 0.4, evaluated in float64 and stored as
  float32.  A query takes ``q_terms`` distinct terms of its own cluster's topic
  vocabulary with weight 1.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ProcessPoolExecutor
from typing import Dict, List, Optional, Tuple

import numpy as np

BASE_SEED = 1729

# stream ids inside one workload
S_CENTERS = 0
S_ROWS = 1
S_QUERIES = 2
S_DOCS = 3
S_SPARSE_Q = 4
S_TOPICS = 5
S_ZIPF_PERM = 6
S_TEMPORAL = 7
S_TEMPORAL_ROWS = 8
S_TEMPORAL_DOCS = 9

CHUNK_ROWS = 131072


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    wid: int               # workload id used in every seed
    n: int                 # corpus rows
    d: int                 # dimension
    centers: int
    std: float = 0.5
    vocab: int = 30000
    doc_len: float = 60.0
    topic_size: int = 200
    q_terms: int = 4
    zipf_s: float = 1.1
    k1: float = 0.9
    b: float = 0.4
    # temporal snapshots
    snapshots: int = 0
    delete_frac: float = 0.10
    insert_frac: float = 0.10
    drift: float = 0.1
    # sparse impacts anti-correlated with the dense ranking
    adversarial: bool = False


WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", 0, n=20_000, d=128, centers=32, vocab=5_000, doc_len=40.0),
    "mid": Workload("mid", 1, n=1_000_000, d=384, centers=1024),
    "passage": Workload("passage", 2, n=8_800_000, d=768, centers=4096),
    "adv": Workload("adv", 3, n=2_000_000, d=768, centers=1024, adversarial=True),
    "temporal": Workload("temporal", 4, n=4_000_000, d=768, centers=4096, snapshots=5),
}

# named query sets: (stream offset, count)
QUERY_SETS = {
    "tiny": {"default": (0, 8)},
    "mid": {"default": (0, 256)},
    "passage": {"single": (0, 200), "b64": (1, 64), "b256": (2, 256)},
    "adv": {"default": (0, 100)},
    "temporal": {"default": (0, 100)},
}


def workload(name: str, **overrides) -> Workload:
    """Return a named workload, optionally with some fields replaced (e.g. a
    smaller ``n`` for a quick CPU test)."""
    return dataclasses.replace(WORKLOADS[name], **overrides)


def _rng(w: Workload, stream: int, chunk: int = 0) -> np.random.Generator:
    ss = np.random.SeedSequence(BASE_SEED, spawn_key=(w.wid, stream, chunk))
    return np.random.default_rng(ss)


def _workers() -> int:
    env = os.environ.get("EAHR_GEN_WORKERS")
    if env:
        return max(1, int(env))
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


# --------------------------------------------------------------------------
# dense vectors
# --------------------------------------------------------------------------
def centers(w: Workload) -> np.ndarray:
    """Cluster centres, float64 [centers, d], ~ N(0, I)."""
    return _rng(w, S_CENTERS).standard_normal((w.centers, w.d))


def _normalize_rows(x: np.ndarray) -> np.ndarray:
    nrm = np.sqrt(np.einsum("ij,ij->i", x, x))
    nrm[nrm == 0.0] = 1.0
    return (x / nrm[:, None]).astype(np.float32)


def _draw_rows(w: Workload, ctr: np.ndarray, stream: int, chunk: int, rows: int,
               shift: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray]:
    rng = _rng(w, stream, chunk)
    labels = rng.integers(0, w.centers, size=rows).astype(np.int32)
    noise = rng.standard_normal((rows, w.d), dtype=np.float32).astype(np.float64)
    base = ctr[labels]
    if shift is not None:
        base = base + shift[labels]
    return _normalize_rows(base + w.std * noise), labels


def n_chunks(n: int) -> int:
    return (n + CHUNK_ROWS - 1) // CHUNK_ROWS


def corpus_chunk(w: Workload, chunk: int, ctr: Optional[np.ndarray] = None
                 ) -> Tuple[np.ndarray, np.ndarray]:
    """Rows ``[chunk*CHUNK_ROWS, ...)`` of the base corpus: (float32 [r,d], labels)."""
    if ctr is None:
        ctr = centers(w)
    lo = chunk * CHUNK_ROWS
    rows = min(w.n, lo + CHUNK_ROWS) - lo
    return _draw_rows(w, ctr, S_ROWS, chunk, rows)


def _corpus_chunk_job(args):
    """Worker: write chunk c straight into the shared output buffer."""
    from multiprocessing import shared_memory
    w, c, shm_name = args
    shm = shared_memory.SharedMemory(name=shm_name)
    try:
        out = np.ndarray((w.n, w.d), dtype=np.float32, buffer=shm.buf)
        x, lab = corpus_chunk(w, c)
        out[c * CHUNK_ROWS: c * CHUNK_ROWS + len(x)] = x
        del out
    finally:
        shm.close()
    return lab


def corpus(w: Workload, workers: Optional[int] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Whole base corpus, float32 [n, d] and int32 labels [n].

    Large corpora are produced by worker processes writing into one shared
    buffer, which is copied once into an ordinary array and released."""
    out = np.empty((w.n, w.d), dtype=np.float32)
    labels = np.empty(w.n, dtype=np.int32)
    nc = n_chunks(w.n)
    workers = workers or _workers()
    if nc == 1 or workers == 1:
        ctr = centers(w)
        for c in range(nc):
            x, lab = corpus_chunk(w, c, ctr)
            out[c * CHUNK_ROWS: c * CHUNK_ROWS + len(x)] = x
            labels[c * CHUNK_ROWS: c * CHUNK_ROWS + len(x)] = lab
        return out, labels
    try:
        st = os.statvfs("/dev/shm")
        shm_free = st.f_bavail * st.f_frsize
    except OSError:
        shm_free = 0
    if shm_free < out.nbytes + (1 << 30):
        # not enough shared memory: threads write into `out` directly
        from concurrent.futures import ThreadPoolExecutor
        ctr = centers(w)

        def fill(c):
            x, lab = corpus_chunk(w, c, ctr)
            out[c * CHUNK_ROWS: c * CHUNK_ROWS + len(x)] = x
            labels[c * CHUNK_ROWS: c * CHUNK_ROWS + len(x)] = lab

        with ThreadPoolExecutor(max_workers=workers) as ex:
            list(ex.map(fill, range(nc)))
        return out, labels
    from multiprocessing import shared_memory
    shm = shared_memory.SharedMemory(create=True, size=max(1, out.nbytes))
    try:
        with ProcessPoolExecutor(max_workers=workers) as ex:
            jobs = [(w, c, shm.name) for c in range(nc)]
            for c, lab in enumerate(ex.map(_corpus_chunk_job, jobs)):
                labels[c * CHUNK_ROWS: c * CHUNK_ROWS + len(lab)] = lab
        view = np.ndarray((w.n, w.d), dtype=np.float32, buffer=shm.buf)
        out[...] = view
        del view
    finally:
        shm.close()
        shm.unlink()
    return out, labels


def queries(w: Workload, qset: str = "default", count: Optional[int] = None
            ) -> Tuple[np.ndarray, np.ndarray]:
    """Dense queries of a named set: float32 [B, d] and their cluster labels."""
    off, nq = QUERY_SETS[w.name][qset]
    if count is not None:
        nq = count
    return _draw_rows(w, centers(w), S_QUERIES, off, nq)


# --------------------------------------------------------------------------
# sparse documents and impacts
# --------------------------------------------------------------------------
def topic_vocab(w: Workload) -> np.ndarray:
    """int32 [centers, topic_size]: each cluster's topic terms (distinct)."""
    rng = _rng(w, S_TOPICS)
    out = np.empty((w.centers, w.topic_size), dtype=np.int32)
    for c in range(w.centers):
        out[c] = rng.choice(w.vocab, size=w.topic_size, replace=False)
    return out


def _zipf_table(w: Workload) -> Tuple[np.ndarray, np.ndarray]:
    ranks = np.arange(1, w.vocab + 1, dtype=np.float64)
    p = ranks ** (-w.zipf_s)
    cdf = np.cumsum(p)
    cdf /= cdf[-1]
    perm = _rng(w, S_ZIPF_PERM).permutation(w.vocab).astype(np.int32)
    return cdf, perm


def _draw_docs(w: Workload, labels: np.ndarray, stream: int, chunk: int,
               topics: np.ndarray, zipf: Tuple[np.ndarray, np.ndarray]):
    """Token draws for the documents of one chunk.

    Returns (doc_local int64, term int32, tf int32, doc_len int32[rows]) with one
    entry per distinct (doc, term), sorted by (term, doc)."""
    cdf, perm = zipf
    rng = _rng(w, stream, chunk)
    rows = len(labels)
    dl = np.maximum(1, rng.poisson(w.doc_len, size=rows)).astype(np.int64)
    total = int(dl.sum())
    doc = np.repeat(np.arange(rows, dtype=np.int64), dl)
    from_zipf = rng.random(total) < 0.5
    u = rng.random(total)
    zr = np.searchsorted(cdf, u, side="right")
    zr = np.minimum(zr, w.vocab - 1)
    tpos = rng.integers(0, w.topic_size, size=total)
    term = np.where(from_zipf, perm[zr], topics[labels[doc], tpos]).astype(np.int64)
    key = term * rows + doc
    ukey, tf = np.unique(key, return_counts=True)
    return (ukey % rows, (ukey // rows).astype(np.int32), tf.astype(np.int32),
            dl.astype(np.int32))


@dataclasses.dataclass
class SparseDocs:
    """Term-major postings of raw term frequencies.

    ``term_ptr[t]:term_ptr[t+1]`` slices ``doc``/``tf`` for term ``t``; doc ids
    ascend within a term.  ``doc_len[x]`` counts every token of document x."""
    vocab: int
    term_ptr: np.ndarray   # int64 [vocab+1]
    doc: np.ndarray        # int32 [P]
    tf: np.ndarray         # int32 [P]
    doc_len: np.ndarray    # int32 [n]


def _merge_chunks(vocab: int, parts, n: int, row_offsets) -> SparseDocs:
    counts = np.zeros((len(parts), vocab), dtype=np.int64)
    for i, (dloc, term, tf, dl) in enumerate(parts):
        counts[i] = np.bincount(term, minlength=vocab)
    per_term = counts.sum(axis=0)
    term_ptr = np.zeros(vocab + 1, dtype=np.int64)
    np.cumsum(per_term, out=term_ptr[1:])
    P = int(term_ptr[-1])
    doc = np.empty(P, dtype=np.int32)
    tfo = np.empty(P, dtype=np.int32)
    doc_len = np.empty(n, dtype=np.int32)
    before = np.zeros(vocab, dtype=np.int64)
    for i, (dloc, term, tf, dl) in enumerate(parts):
        r0 = row_offsets[i]
        doc_len[r0:r0 + len(dl)] = dl
        # entries of this chunk are sorted by (term, doc): the position of an
        # entry inside its term segment is its index minus the segment start
        starts = np.zeros(vocab + 1, dtype=np.int64)
        np.cumsum(counts[i], out=starts[1:])
        idx = np.arange(len(term), dtype=np.int64) - starts[term]
        pos = term_ptr[term] + before[term] + idx
        doc[pos] = (dloc + r0).astype(np.int32)
        tfo[pos] = tf
        before += counts[i]
    return SparseDocs(vocab, term_ptr, doc, tfo, doc_len)


def _docs_chunk_job(args):
    w, labels, stream, chunk, topics, zipf = args
    return _draw_docs(w, labels, stream, chunk, topics, zipf)


def sparse_docs(w: Workload, labels: np.ndarray, workers: Optional[int] = None) -> SparseDocs:
    """Documents of the base corpus (document i belongs to cluster labels[i])."""
    topics = topic_vocab(w)
    zipf = _zipf_table(w)
    nc = n_chunks(len(labels))
    jobs = [(w, labels[c * CHUNK_ROWS:(c + 1) * CHUNK_ROWS], S_DOCS, c, topics, zipf)
            for c in range(nc)]
    workers = workers or _workers()
    if nc == 1 or workers == 1:
        parts = [_docs_chunk_job(j) for j in jobs]
    else:
        with ProcessPoolExecutor(max_workers=workers) as ex:
            parts = list(ex.map(_docs_chunk_job, jobs))
    return _merge_chunks(w.vocab, parts, len(labels), [c * CHUNK_ROWS for c in range(nc)])


@dataclasses.dataclass
class Postings:
    """Term-major postings with float32 impacts (doc ids ascend per term)."""
    vocab: int
    term_ptr: np.ndarray   # int64 [vocab+1]
    doc: np.ndarray        # int32 [P]
    impact: np.ndarray     # float32 [P]


def bm25_impacts(w: Workload, docs: SparseDocs, visible: Optional[np.ndarray] = None) -> Postings:
    """Lucene-form BM25 impacts, computed in float64 and stored as float32.

    idf = ln(1 + (N - df + 0.5) / (df + 0.5));  impact = idf * tf / (tf + k1 (1 - b + b dl/avgdl)).
    Statistics (N, df, avgdl) are taken over the visible documents only, and
    postings of invisible documents are dropped."""
    doc, tf = docs.doc, docs.tf
    term_ptr = docs.term_ptr
    if visible is not None:
        keep = visible[doc]
        owner = np.repeat(np.arange(docs.vocab, dtype=np.int64), np.diff(term_ptr))
        counts = np.bincount(owner[keep], minlength=docs.vocab).astype(np.int64)
        term_ptr = np.zeros(docs.vocab + 1, dtype=np.int64)
        np.cumsum(counts, out=term_ptr[1:])
        doc, tf = doc[keep], tf[keep]
        n_vis = int(visible.sum())
        avgdl = float(docs.doc_len[visible].astype(np.float64).mean())
    else:
        n_vis = len(docs.doc_len)
        avgdl = float(docs.doc_len.astype(np.float64).mean())
    df = np.diff(term_ptr).astype(np.float64)
    idf = np.log1p((n_vis - df + 0.5) / (df + 0.5))
    term_of = np.repeat(np.arange(docs.vocab, dtype=np.int64), np.diff(term_ptr))
    dl = docs.doc_len[doc].astype(np.float64)
    tf64 = tf.astype(np.float64)
    imp = idf[term_of] * tf64 / (tf64 + w.k1 * (1.0 - w.b + w.b * dl / avgdl))
    return Postings(docs.vocab, term_ptr, doc.astype(np.int32), imp.astype(np.float32))


def sparse_queries(w: Workload, labels: np.ndarray, stream_off: int = 0
                   ) -> List[Tuple[np.ndarray, np.ndarray]]:
    """Per query: (term ids int32 ascending, weights float32 = 1)."""
    topics = topic_vocab(w)
    rng = _rng(w, S_SPARSE_Q, stream_off)
    out = []
    for lab in labels:
        t = np.sort(rng.choice(topics[lab], size=w.q_terms, replace=False)).astype(np.int32)
        out.append((t, np.ones(len(t), dtype=np.float32)))
    return out


def query_set_offset(w: Workload, qset: str) -> int:
    return QUERY_SETS[w.name][qset][0]


# --------------------------------------------------------------------------
# adversarial (anti-correlated) sparse channel
# --------------------------------------------------------------------------
def adversarial_postings(w: Workload, corpus_f32: np.ndarray, q_f32: np.ndarray) -> Tuple[
        Postings, List[Tuple[np.ndarray, np.ndarray]]]:
    """Sparse channel whose ranking is the reverse of the dense one.

    Query j owns a private term j that every document carries, with impact
    ``2 - <q_j, x>`` (inner product in float64, stored float32), so a document's
    sparse rank is about ``N + 1 -`` its dense rank.  Query j's sparse query is
    that single term with weight 1."""
    n = corpus_f32.shape[0]
    nq = q_f32.shape[0]
    term_ptr = np.arange(nq + 1, dtype=np.int64) * n
    doc = np.tile(np.arange(n, dtype=np.int32), nq)
    imp = np.empty(nq * n, dtype=np.float32)
    q64 = q_f32.astype(np.float64)
    step = 65536
    for r0 in range(0, n, step):
        blk = corpus_f32[r0:r0 + step].astype(np.float64) @ q64.T   # [rows, nq]
        for j in range(nq):
            imp[j * n + r0: j * n + r0 + blk.shape[0]] = (2.0 - blk[:, j]).astype(np.float32)
    qs = [(np.array([j], dtype=np.int32), np.ones(1, dtype=np.float32)) for j in range(nq)]
    return Postings(nq, term_ptr, doc, imp), qs


# --------------------------------------------------------------------------
# temporal snapshots
# --------------------------------------------------------------------------
@dataclasses.dataclass
class SnapshotStep:
    """One corpus update: delete some visible ids, then append new rows."""
    delete_ids: np.ndarray     # int64, ascending
    insert_rows: np.ndarray    # float32 [k, d]
    insert_labels: np.ndarray  # int32 [k]


def temporal_steps(w: Workload, base_n: int, steps: Optional[int] = None):
    """Yield ``w.snapshots`` updates.  Step s deletes ``delete_frac`` of the
    currently visible ids (uniformly) and inserts ``insert_frac`` of the visible
    count as new rows (ids continue after the last physical row), drawn from
    centres that drift cumulatively by ``drift * N(0, I)`` per step."""
    ctr = centers(w)
    shift = np.zeros_like(ctr)
    visible = np.ones(base_n, dtype=bool)
    steps = w.snapshots if steps is None else steps
    for s in range(1, steps + 1):
        rng = _rng(w, S_TEMPORAL, s)
        shift = shift + w.drift * rng.standard_normal(ctr.shape)
        vis_ids = np.flatnonzero(visible)
        n_vis = len(vis_ids)
        n_del = int(round(w.delete_frac * n_vis))
        n_ins = int(round(w.insert_frac * n_vis))
        dels = np.sort(rng.choice(vis_ids, size=n_del, replace=False)).astype(np.int64)
        visible[dels] = False
        rows = []
        labs = []
        for c in range(n_chunks(n_ins)):
            r = min(n_ins, (c + 1) * CHUNK_ROWS) - c * CHUNK_ROWS
            x, lab = _draw_rows(w, ctr, S_TEMPORAL_ROWS, s * 4096 + c, r, shift=shift)
            rows.append(x)
            labs.append(lab)
        ins = np.concatenate(rows) if rows else np.zeros((0, w.d), np.float32)
        ins_lab = np.concatenate(labs) if labs else np.zeros(0, np.int32)
        visible = np.concatenate([visible, np.ones(n_ins, dtype=bool)])
        yield SnapshotStep(dels, ins, ins_lab)


def temporal_docs(w: Workload, labels_all: np.ndarray, base_n: int) -> SparseDocs:
    """Documents of the base corpus plus every inserted row (labels_all covers
    all physical rows in id order); inserted documents use their own stream."""
    topics = topic_vocab(w)
    zipf = _zipf_table(w)
    parts = []
    offs = []
    for c in range(n_chunks(base_n)):
        lab = labels_all[c * CHUNK_ROWS:min(base_n, (c + 1) * CHUNK_ROWS)]
        parts.append(_draw_docs(w, lab, S_DOCS, c, topics, zipf))
        offs.append(c * CHUNK_ROWS)
    rest = labels_all[base_n:]
    for c in range(n_chunks(len(rest))):
        lab = rest[c * CHUNK_ROWS:(c + 1) * CHUNK_ROWS]
        parts.append(_draw_docs(w, lab, S_TEMPORAL_DOCS, c, topics, zipf))
        offs.append(base_n + c * CHUNK_ROWS)
    return _merge_chunks(w.vocab, parts, len(labels_all), offs)


# --------------------------------------------------------------------------
# controlled rank streams (Sec. 3.4)
# --------------------------------------------------------------------------
STREAM_SIZES = (100_000, 1_000_000, 5_000_000)
STREAM_SEEDS = (1729, 2027, 65537)
STREAM_RELATIONS = ("correlated", "partial", "independent", "anti", "all_tied")


def controlled_streams(relation: str, n: int, seed: int) -> Tuple[np.ndarray, np.ndarray]:
    """Two complete rankings of the ids 0..n-1 with a given relationship:
    the first list is a random permutation (except all-tied); the second
    permutes it inside contiguous blocks of 32 ("correlated"), takes 500
    random items of the first list's top 1,000 and the 500 items that follow
    that top 1,000 in the first list, shuffled, as its own top 1,000, followed
    by the other items in the first list's order ("partial"), is an
    independent permutation ("independent") or the
    reversed first list ("anti").  All-tied: every item scores the same in
    both lists, so both are identifier order."""
    rng = np.random.default_rng(seed)
    if relation == "all_tied":
        ids = np.arange(n, dtype=np.int64)
        return ids, ids.copy()
    a = rng.permutation(n).astype(np.int64)
    if relation == "correlated":
        order = np.lexsort((rng.random(n), np.arange(n) // 32))
        b = a[order]
    elif relation == "partial":
        top = min(1000, n)
        half = top // 2
        inside = rng.choice(a[:top], size=half, replace=False)
        outside = a[top:top + (top - half)]
        head = rng.permutation(np.concatenate([inside, outside]))
        used = np.zeros(n, dtype=bool)
        used[head] = True
        b = np.concatenate([head, a[~used[a]]])
    elif relation == "independent":
        b = rng.permutation(n).astype(np.int64)
    elif relation == "anti":
        b = a[::-1].copy()
    else:
        raise ValueError(f"unknown stream relation {relation!r}")
    return a, b.astype(np.int64)
