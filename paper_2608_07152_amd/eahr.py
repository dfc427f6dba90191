"""ctypes binding of ``libeahr.so`` (declared in ``include/eahr.h``).

Argument marshalling only: every step of the retrieval path runs inside the
library.  Functions carry the C names; handles are small Python objects whose
``close()``/``free()`` release the library handle (also done on garbage
collection).  Arrays may be numpy (host) or torch CUDA tensors (device).

Loading fails loudly when the library has not been built
(``python -m paper_2608_07152_amd.build``).
"""
from __future__ import annotations

import ctypes as C
import os
from typing import List, Optional, Sequence, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libeahr.so")

EAHR_OK = 0
EAHR_E_INVALID = -1
EAHR_E_NONFINITE = -2
EAHR_E_RANGE = -3
EAHR_E_OOM = -4
EAHR_E_HIP = -5
EAHR_E_FAILED = -6
LIST_OPEN, LIST_EXHAUSTED, LIST_FAILED = 0, 1, 2
PTR_HOST, PTR_DEVICE = 0, 1

_ERRNAMES = {EAHR_E_INVALID: "EAHR_E_INVALID", EAHR_E_NONFINITE: "EAHR_E_NONFINITE",
             EAHR_E_RANGE: "EAHR_E_RANGE", EAHR_E_OOM: "EAHR_E_OOM", EAHR_E_HIP: "EAHR_E_HIP",
             EAHR_E_FAILED: "EAHR_E_FAILED"}


class EahrError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{_ERRNAMES.get(code, code)}: {msg}")
        self.code = code


class eahr_sparse_query(C.Structure):
    _fields_ = [("terms", C.POINTER(C.c_int32)), ("weights", C.POINTER(C.c_float)),
                ("n_terms", C.c_int32)]


class eahr_params(C.Structure):
    _fields_ = [("K", C.c_int32), ("depth0", C.c_int32), ("growth", C.c_int32),
                ("k_rrf", C.c_int32), ("w_dense", C.c_int32), ("w_sparse", C.c_int32),
                ("dense_generator", C.c_int32), ("schedule", C.c_int32),
                ("sparse_generator", C.c_int32)]


class eahr_query_stats(C.Structure):
    _fields_ = [("dense_depth", C.c_int64), ("sparse_depth", C.c_int64),
                ("dense_len", C.c_int64), ("sparse_len", C.c_int64),
                ("dense_status", C.c_int32), ("sparse_status", C.c_int32),
                ("rounds", C.c_int32), ("resolved", C.c_int32),
                ("dense_evals", C.c_int64), ("sparse_postings", C.c_int64),
                ("sparse_scored", C.c_int64)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


class pvs_counters(C.Structure):
    _fields_ = [(n, C.c_int64) for n in ("scans", "sample_scans", "rows_scanned", "bytes_scanned",
                                          "candidates", "certified", "emitted", "rescans",
                                          "overflows")]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


class pvs_profile(C.Structure):
    _fields_ = [("scan_ms", C.c_double), ("scan_launches", C.c_int64), ("scan_bytes", C.c_int64),
                ("sample_ms", C.c_double), ("rescore_ms", C.c_double), ("rescore_rows", C.c_int64),
                ("sort_ms", C.c_double), ("scan_rounds", C.c_int64),
                ("mfma_launches", C.c_int64), ("host_dense_ms", C.c_double),
                ("host_sparse_ms", C.c_double), ("host_fuse_ms", C.c_double),
                ("variant_ms", C.c_double * 12), ("variant_launches", C.c_int64 * 12),
                ("variant_bytes", C.c_int64 * 12), ("rescore_certified", C.c_int64),
                ("rescore_row_reads", C.c_int64)]

    VARIANTS = [f"k_scan_gemv<{q}>" for q in range(1, 9)] + \
        [f"k_scan_mfma<{t}>" for t in (1, 2, 4, 8)]

    def as_dict(self):
        out = {}
        for f, _ in self._fields_:
            v = getattr(self, f)
            out[f] = list(v) if f.startswith("variant_") else v
        return out


_P = C.c_void_p
_i32, _i64, _f32p = C.c_int32, C.c_int64, C.POINTER(C.c_float)
_i64p, _i32p, _u8p, _i8p = C.POINTER(C.c_int64), C.POINTER(C.c_int32), C.POINTER(C.c_uint8), C.POINTER(C.c_int8)

# name -> (restype, argtypes); mirrors include/eahr.h
# eahr_rank_observer (include/eahr.h)
RANK_OBSERVER = C.CFUNCTYPE(None, C.c_void_p, C.c_int32, C.c_int32, C.c_int64,
                            C.POINTER(C.c_int64), C.POINTER(C.c_float), C.c_int64)

SIGNATURES = {
    "pvs_build": (C.c_int, [_P, _i64, _i32, _i32, _P, C.POINTER(_P)]),
    "pvs_build_quant": (C.c_int, [_P, _i64, _i32, _i32, _P, _i32, C.POINTER(_P)]),
    "pvs_insert": (C.c_int, [_P, _P, _i64, _i32, _i64p]),
    "pvs_delete": (C.c_int, [_P, _i64p, _i64]),
    "pvs_snapshot": (C.c_int, [_P, _i64p]),
    "pvs_info": (C.c_int, [_P, _i64, _i64p, _i32p, _i64p]),
    "pvs_open": (C.c_int, [_P, _i64, _P, _i32, _i32, C.POINTER(_P)]),
    "pvs_open_gen": (C.c_int, [_P, _i64, _P, _i32, _i32, _i32, C.POINTER(_P)]),
    "pvs_merge_open": (C.c_int, [C.POINTER(_P), _i64p, C.POINTER(_i64p), C.POINTER(_i64p), _i32, _P,
                                 _i32, _i32, C.POINTER(_P)]),
    "pvs_merge_shards": (C.c_int, [C.POINTER(_P), _i32, C.POINTER(_P)]),
    "pvs_merge_next": (C.c_int, [_P, _i32, _u8p, _i64p, _f32p, _i32p, _i32p]),
    "pvs_merge_close": (None, [_P]),
    "pvs_next": (C.c_int, [_P, _i32, _u8p, _i64p, _f32p, _i32p, _i32p]),
    "pvs_stats": (C.c_int, [_P, C.POINTER(pvs_counters)]),
    "pvs_profile_enable": (C.c_int, [_i32]),
    "pvs_profile_read": (C.c_int, [C.POINTER(pvs_profile)]),
    "pvs_read_index": (C.c_int, [_P, _i64, _i64, _i8p, _f32p]),
    "pvs_read_query": (C.c_int, [_P, _i8p, _f32p]),
    "pvs_intervals": (C.c_int, [_P, _i32, _i64p, _i64, _f32p, _f32p]),
    "pvs_scores": (C.c_int, [_P, _i32, _i64p, _i64, _f32p]),
    "eahr_set_rank_observer": (C.c_int, [RANK_OBSERVER, _P]),
    "pvs_scores_noalloc": (C.c_int, [_P, _i32, _i64p, _i64, _f32p]),
    "pvs_close": (None, [_P]),
    "pvs_free": (None, [_P]),
    "pbm_build": (C.c_int, [_i64p, _i32, _i32p, _f32p, _i64, _i32, C.POINTER(_P)]),
    "pbm_free": (None, [_P]),
    "pbm_open": (C.c_int, [_P, C.POINTER(eahr_sparse_query), C.POINTER(_P)]),
    "pbm_open_gen": (C.c_int, [_P, C.POINTER(eahr_sparse_query), _i32, C.POINTER(_P)]),
    "pbm_next": (C.c_int, [_P, _i32, _i64p, _f32p, _i32p, _i32p]),
    "pbm_close": (None, [_P]),
    "pbm_debug_set_blockmax": (C.c_int, [_P, _i32, _i64, C.c_float]),
    "pbm_upload": (C.c_int, [_P]),
    "pbm_gpu_open": (C.c_int, [_P, C.POINTER(eahr_sparse_query), _i32, C.POINTER(_P)]),
    "pbm_gpu_next": (C.c_int, [_P, _i32p, C.POINTER(_i64p), C.POINTER(_f32p), _i32p, _i32p]),
    "pbm_gpu_counters": (C.c_int, [_P, _i32, _i64p]),
    "pbm_gpu_close": (None, [_P]),
    "eahr_topk": (C.c_int, [_P, _i64, _P, _P, _i32, C.POINTER(eahr_sparse_query), _i32,
                            C.POINTER(eahr_params), _i64p, _i32p, _i32p,
                            C.POINTER(eahr_query_stats)]),
    "eahr_topk_merged": (C.c_int, [_P, _P, C.POINTER(eahr_sparse_query), _i32, C.POINTER(eahr_params),
                                   _i64p, _i32p, _i32p, C.POINTER(eahr_query_stats)]),
    "eahr_fuse_lists": (C.c_int, [_i64p, _i64, _i64p, _i64, C.POINTER(eahr_params), _i32, _i64p,
                                  _i32p, C.POINTER(eahr_query_stats)]),
    "eahr_last_error": (C.c_char_p, []),
}

_lib = None


def load() -> C.CDLL:
    """Load libeahr.so (raises ImportError when it is missing)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2608_07152_amd.build`")
    # torch ships its own HIP runtime under the same SONAME (libamdhip64.so.7).
    # Loading torch first makes the library bind to that copy, so the process
    # holds one HIP runtime and torch device pointers and streams are valid here.
    try:
        import torch  # noqa: F401
    except ImportError:  # pragma: no cover
        pass
    lib = C.CDLL(LIB_PATH)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(rc: int):
    if rc != EAHR_OK:
        raise EahrError(rc, load().eahr_last_error().decode())


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(C.POINTER(ctype))


def _array_arg(x, dtype=np.float32):
    """(pointer, ptr_kind, keepalive, shape) for a numpy array or torch tensor."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            if x.dtype != torch.float32:
                raise TypeError("expected a float32 tensor")
            x = x.contiguous()
            if x.is_cuda:
                return C.c_void_p(x.data_ptr()), PTR_DEVICE, x, tuple(x.shape)
            x = x.numpy()
    except ImportError:  # pragma: no cover
        pass
    a = np.ascontiguousarray(x, dtype=dtype)
    return C.c_void_p(a.ctypes.data), PTR_HOST, a, a.shape


def _stream_ptr(stream) -> C.c_void_p:
    if stream is None:
        return C.c_void_p(0)
    if isinstance(stream, int):
        return C.c_void_p(stream)
    return C.c_void_p(int(stream.cuda_stream))


# ------------------------------------------------------------------ handles
class PvsIndex:
    def __init__(self, handle: C.c_void_p, d: int):
        self.h = handle
        self.d = d

    def free(self):
        if self.h:
            load().pvs_free(self.h)
            self.h = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


class PvsState:
    def __init__(self, handle: C.c_void_p, index: PvsIndex, B: int):
        self.h = handle
        self.index = index   # keeps the index alive
        self.B = B

    def close(self):
        if self.h:
            load().pvs_close(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class PvsMerge:
    """A merged dense ranking (a Shard over Segments, or a request over
    Shards); keeps its indexes alive."""

    def __init__(self, handle, keep, B: int):
        self.h = handle
        self.keep = keep
        self.B = B

    def close(self):
        if self.h:
            load().pvs_merge_close(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class PbmIndex:
    def __init__(self, handle):
        self.h = handle

    def free(self):
        if self.h:
            load().pbm_free(self.h)
            self.h = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


class PbmState:
    def __init__(self, handle, index):
        self.h = handle
        self.index = index

    def close(self):
        if self.h:
            load().pbm_close(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class PbmGpuState:
    def __init__(self, handle, index, keep):
        self.h = handle
        self.index = index
        self._keep = keep

    def close(self):
        if self.h:
            load().pbm_gpu_close(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ------------------------------------------------------------------- dense
def pvs_build(corpus, stream=None) -> PvsIndex:
    """Quantise a float32 corpus [n, d] (numpy or torch CUDA tensor)."""
    p, kind, keep, shape = _array_arg(corpus)
    n, d = shape
    h = C.c_void_p()
    _check(load().pvs_build(p, n, d, kind, _stream_ptr(stream), C.byref(h)))
    return PvsIndex(h, d)


QUANT_MODES = {"per_vector": 0, "global": 1}


def pvs_build_quant(corpus, quant: str = "per_vector", stream=None) -> PvsIndex:
    """pvs_build with a choice of scale: "per_vector" (PVS) or "global" (one
    scale shared by every row, the scalar-quantisation generator)."""
    p, kind, keep, shape = _array_arg(corpus)
    n, d = shape
    h = C.c_void_p()
    _check(load().pvs_build_quant(p, n, d, kind, _stream_ptr(stream), QUANT_MODES[quant], C.byref(h)))
    return PvsIndex(h, d)


def pvs_insert(index: PvsIndex, rows) -> int:
    p, kind, keep, shape = _array_arg(rows)
    first = C.c_int64()
    _check(load().pvs_insert(index.h, p, shape[0], kind, C.byref(first)))
    return first.value


def pvs_delete(index: PvsIndex, ids) -> None:
    a = np.ascontiguousarray(ids, dtype=np.int64)
    _check(load().pvs_delete(index.h, _ptr(a, C.c_int64), len(a)))


def pvs_snapshot(index: PvsIndex) -> int:
    e = C.c_int64()
    _check(load().pvs_snapshot(index.h, C.byref(e)))
    return e.value


def pvs_info(index: PvsIndex, epoch: int = 0) -> Tuple[int, int, int]:
    rows, d, vis = C.c_int64(), C.c_int32(), C.c_int64()
    _check(load().pvs_info(index.h, epoch, C.byref(rows), C.byref(d), C.byref(vis)))
    return rows.value, d.value, vis.value


GENERATORS = {"intervals": 0, "full_scan": 1}


def pvs_open(index: PvsIndex, queries, epoch: int = 0, generator: str = "intervals") -> PvsState:
    """Encode a query batch and open resumable dense state; ``generator`` is
    "intervals" (interval scans) or "full_scan" (one exhaustive float32 scan)."""
    p, kind, keep, shape = _array_arg(queries)
    if len(shape) == 1:
        shape = (1, shape[0])
    h = C.c_void_p()
    if generator == "intervals":
        _check(load().pvs_open(index.h, epoch, p, shape[0], kind, C.byref(h)))
    else:
        _check(load().pvs_open_gen(index.h, epoch, p, shape[0], kind, GENERATORS[generator], C.byref(h)))
    return PvsState(h, index, shape[0])


def pvs_next(state: PvsState, m: int, active: Optional[Sequence[bool]] = None):
    """Next m exact ranks per query: (ids [B,m] int64, scores [B,m] f32,
    count [B] int32, status [B] int32)."""
    B = state.B
    ids = np.full((B, max(m, 1)), -1, dtype=np.int64)
    sc = np.zeros((B, max(m, 1)), dtype=np.float32)
    cnt = np.zeros(B, dtype=np.int32)
    stt = np.zeros(B, dtype=np.int32)
    act = None
    if active is not None:
        act = np.ascontiguousarray(np.asarray(active, dtype=np.uint8))
    _check(load().pvs_next(state.h, m, _ptr(act, C.c_uint8) if act is not None else None,
                           _ptr(ids, C.c_int64), _ptr(sc, C.c_float), _ptr(cnt, C.c_int32),
                           _ptr(stt, C.c_int32)))
    return ids[:, :m], sc[:, :m], cnt, stt


def pvs_merge_open(segments: Sequence[PvsIndex], gids, queries, versions=None, epochs=None) -> PvsMerge:
    """A Shard over Segments: segments[s] with its row -> global id map
    gids[s] (strictly ascending) and optional per-row versions."""
    n = len(segments)
    p, kind, keep, shape = _array_arg(queries)
    if len(shape) == 1:
        shape = (1, shape[0])
    segs = (_P * n)(*[sg.h for sg in segments])
    g = [np.ascontiguousarray(x, dtype=np.int64) for x in gids]
    gp = (_i64p * n)(*[_ptr(x, C.c_int64) for x in g])
    v = None
    vp = None
    if versions is not None:
        v = [None if x is None else np.ascontiguousarray(x, dtype=np.int64) for x in versions]
        vp = (_i64p * n)(*[(_ptr(x, C.c_int64) if x is not None else None) for x in v])
    e = None
    if epochs is not None:
        e = np.ascontiguousarray(epochs, dtype=np.int64)
    h = C.c_void_p()
    _check(load().pvs_merge_open(segs, _ptr(e, C.c_int64) if e is not None else None, gp, vp, n, p,
                                 shape[0], kind, C.byref(h)))
    return PvsMerge(h, list(segments), shape[0])


def pvs_merge_shards(shards: Sequence[PvsMerge]) -> PvsMerge:
    """The request-level merge over Shards; takes ownership of them."""
    n = len(shards)
    arr = (_P * n)(*[s.h for s in shards])
    h = C.c_void_p()
    _check(load().pvs_merge_shards(arr, n, C.byref(h)))
    keep = []
    for s in shards:
        keep.append(s.keep)
        s.h = None          # owned by the request-level merge now
    return PvsMerge(h, keep, shards[0].B)


def pvs_merge_next(mg: PvsMerge, m: int, active: Optional[Sequence[bool]] = None):
    """Next m merged ranks per query: (global ids [B,m], scores [B,m], count, status)."""
    B = mg.B
    ids = np.full((B, max(m, 1)), -1, dtype=np.int64)
    sc = np.zeros((B, max(m, 1)), dtype=np.float32)
    cnt = np.zeros(B, dtype=np.int32)
    stt = np.zeros(B, dtype=np.int32)
    act = None
    if active is not None:
        act = np.ascontiguousarray(np.asarray(active, dtype=np.uint8))
    _check(load().pvs_merge_next(mg.h, m, _ptr(act, C.c_uint8) if act is not None else None,
                                 _ptr(ids, C.c_int64), _ptr(sc, C.c_float), _ptr(cnt, C.c_int32),
                                 _ptr(stt, C.c_int32)))
    return ids[:, :m], sc[:, :m], cnt, stt


def pvs_stats(state: PvsState) -> dict:
    c = pvs_counters()
    _check(load().pvs_stats(state.h, C.byref(c)))
    return c.as_dict()


def pvs_profile_enable(on: bool = True) -> None:
    _check(load().pvs_profile_enable(1 if on else 0))


def pvs_profile_read() -> dict:
    p = pvs_profile()
    _check(load().pvs_profile_read(C.byref(p)))
    return p.as_dict()


def pvs_read_index(index: PvsIndex, row0: int, n: int):
    codes = np.zeros((n, index.d), dtype=np.int8)
    meta = np.zeros((n, 3), dtype=np.float32)
    _check(load().pvs_read_index(index.h, row0, n, _ptr(codes, C.c_int8), _ptr(meta, C.c_float)))
    return codes, meta


def pvs_read_query(state: PvsState):
    codes = np.zeros((state.B, state.index.d), dtype=np.int8)
    meta = np.zeros((state.B, 4), dtype=np.float32)
    _check(load().pvs_read_query(state.h, _ptr(codes, C.c_int8), _ptr(meta, C.c_float)))
    return codes, meta


def pvs_intervals(state: PvsState, b: int, rows):
    r = np.ascontiguousarray(rows, dtype=np.int64)
    lo = np.zeros(len(r), dtype=np.float32)
    hi = np.zeros(len(r), dtype=np.float32)
    _check(load().pvs_intervals(state.h, b, _ptr(r, C.c_int64), len(r), _ptr(lo, C.c_float),
                                _ptr(hi, C.c_float)))
    return lo, hi


def pvs_scores(state: PvsState, b: int, rows):
    r = np.ascontiguousarray(rows, dtype=np.int64)
    out = np.zeros(len(r), dtype=np.float32)
    _check(load().pvs_scores(state.h, b, _ptr(r, C.c_int64), len(r), _ptr(out, C.c_float)))
    return out


NOALLOC_MAX_ROWS = 65536


def pvs_scores_noalloc(state: PvsState, b: int, rows):
    """pvs_scores through the entry point that allocates nothing (at most
    NOALLOC_MAX_ROWS rows per call)."""
    r = np.ascontiguousarray(rows, dtype=np.int64)
    out = np.zeros(len(r), dtype=np.float32)
    _check(load().pvs_scores_noalloc(state.h, b, _ptr(r, C.c_int64), len(r), _ptr(out, C.c_float)))
    return out


def pvs_close(state: PvsState) -> None:
    state.close()


def pvs_free(index: PvsIndex) -> None:
    index.free()


# ------------------------------------------------------------------ sparse
def pbm_build(term_ptr, docs, impacts, n_docs: int, range_size: int = 4096) -> PbmIndex:
    tp = np.ascontiguousarray(term_ptr, dtype=np.int64)
    dc = np.ascontiguousarray(docs, dtype=np.int32)
    im = np.ascontiguousarray(impacts, dtype=np.float32)
    h = C.c_void_p()
    _check(load().pbm_build(_ptr(tp, C.c_int64), len(tp) - 1, _ptr(dc, C.c_int32),
                            _ptr(im, C.c_float), n_docs, range_size, C.byref(h)))
    return PbmIndex(h)


def _sparse_query(terms, weights):
    t = np.ascontiguousarray(terms, dtype=np.int32)
    w = np.ascontiguousarray(weights, dtype=np.float32)
    q = eahr_sparse_query(_ptr(t, C.c_int32), _ptr(w, C.c_float), len(t))
    return q, (t, w)


def pbm_open(index: PbmIndex, terms, weights, generator: str = "pbm") -> PbmState:
    """Resumable exact sparse ranking of one query; ``generator`` is "pbm"
    (Posting Block-Max) or "complete" (every document scored and sorted at the
    first call)."""
    q, keep = _sparse_query(terms, weights)
    h = C.c_void_p()
    if generator == "pbm":
        _check(load().pbm_open(index.h, C.byref(q), C.byref(h)))
    else:
        _check(load().pbm_open_gen(index.h, C.byref(q), SPARSE_GENERATORS[generator], C.byref(h)))
    return PbmState(h, index)


def pbm_next(state: PbmState, m: int):
    ids = np.full(max(m, 1), -1, dtype=np.int64)
    sc = np.zeros(max(m, 1), dtype=np.float32)
    cnt, stt = C.c_int32(), C.c_int32()
    _check(load().pbm_next(state.h, m, _ptr(ids, C.c_int64), _ptr(sc, C.c_float), C.byref(cnt),
                           C.byref(stt)))
    return ids[:cnt.value], sc[:cnt.value], stt.value


def pbm_close(state: PbmState) -> None:
    state.close()


def pbm_free(index: PbmIndex) -> None:
    index.free()


def pbm_debug_set_blockmax(index: PbmIndex, term: int, range_: int, value: float) -> None:
    _check(load().pbm_debug_set_blockmax(index.h, term, range_, value))


PBM_GPU_MAX_RANGE = 16384


def pbm_upload(index: PbmIndex) -> None:
    _check(load().pbm_upload(index.h))


def pbm_gpu_open(index: PbmIndex, queries: Sequence[Tuple[np.ndarray, np.ndarray]]) -> PbmGpuState:
    """A batch of sparse queries ranked by Posting Block-Max with the posting
    work on the GPU; ``queries`` is a list of (terms, weights)."""
    B = len(queries)
    qs = (eahr_sparse_query * max(B, 1))()
    keep = []
    for b, (t, w) in enumerate(queries):
        q, k = _sparse_query(t, w)
        qs[b] = q
        keep.append(k)
    h = C.c_void_p()
    _check(load().pbm_gpu_open(index.h, qs, B, C.byref(h)))
    return PbmGpuState(h, index, keep)


def pbm_gpu_next(state: PbmGpuState, m):
    """The next m[b] ranks of every query (m: an int for all, or one per
    query; 0 leaves a query untouched).  Returns a list of (ids, scores,
    status) per query."""
    B = len(state._keep)
    mm = np.ascontiguousarray(np.broadcast_to(np.asarray(m, dtype=np.int32), (B,)))
    ids = [np.full(max(int(v), 1), -1, dtype=np.int64) for v in mm]
    sc = [np.zeros(max(int(v), 1), dtype=np.float32) for v in mm]
    pid = (C.POINTER(C.c_int64) * max(B, 1))(*[_ptr(a, C.c_int64) for a in ids])
    psc = (C.POINTER(C.c_float) * max(B, 1))(*[_ptr(a, C.c_float) for a in sc])
    cnt = np.zeros(max(B, 1), dtype=np.int32)
    stt = np.zeros(max(B, 1), dtype=np.int32)
    _check(load().pbm_gpu_next(state.h, _ptr(mm, C.c_int32), pid, psc, _ptr(cnt, C.c_int32),
                               _ptr(stt, C.c_int32)))
    return [(ids[b][:cnt[b]], sc[b][:cnt[b]], int(stt[b])) for b in range(B)]


def pbm_gpu_counters(state: PbmGpuState, b: int):
    """(postings visited, documents scored, ranges expanded) of query b."""
    out = np.zeros(3, dtype=np.int64)
    _check(load().pbm_gpu_counters(state.h, b, _ptr(out, C.c_int64)))
    return int(out[0]), int(out[1]), int(out[2])


def pbm_gpu_close(state: PbmGpuState) -> None:
    state.close()


# ------------------------------------------------------------------ fusion
SCHEDULES = {"doubling": 0, "frozen": 1}
SPARSE_GENERATORS = {"pbm": 0, "complete": 1, "pbm_gpu": 2}


def _params(K, k_rrf, w_dense, w_sparse, depth0, growth, generator="intervals", schedule="doubling",
            sparse_generator="pbm"):
    for v in (k_rrf, w_dense, w_sparse):
        if int(v) != v:
            raise ValueError("k and the weights must be integers")
    return eahr_params(int(K), int(depth0), int(growth), int(k_rrf), int(w_dense), int(w_sparse),
                       GENERATORS[generator], SCHEDULES[schedule], SPARSE_GENERATORS[sparse_generator])


def eahr_topk(dense: Optional[PvsIndex], sparse: Optional[PbmIndex], q_dense,
              q_sparse: Sequence[Tuple[np.ndarray, np.ndarray]], K: int = 20, k_rrf: int = 60,
              w_dense: int = 1, w_sparse: int = 1, epoch: int = 0, depth0: int = 20,
              growth: int = 2, allow_failed: bool = False, dense_generator: str = "intervals",
              schedule: str = "doubling", sparse_generator: str = "pbm"):
    """Ordered Top-K of complete-list weighted RRF for a batch of queries
    (``dense_generator``: "intervals" or "full_scan", see pvs_open).

    Returns (ids [B,K] int64 with -1 padding, count [B], status [B], stats list)."""
    B = len(q_sparse) if q_sparse is not None else int(np.shape(q_dense)[0])
    if q_dense is not None:
        p, kind, keepd, shape = _array_arg(q_dense)
        B = shape[0]
    else:
        p, kind, keepd = None, PTR_HOST, None
    qs = (eahr_sparse_query * B)()
    keep = []
    if q_sparse is not None:
        for b, (t, w) in enumerate(q_sparse):
            q, k = _sparse_query(t, w)
            qs[b] = q
            keep.append(k)
    prm = _params(K, k_rrf, w_dense, w_sparse, depth0, growth, dense_generator, schedule, sparse_generator)
    ids = np.full((B, max(K, 1)), -1, dtype=np.int64)
    cnt = np.zeros(B, dtype=np.int32)
    stt = np.zeros(B, dtype=np.int32)
    stats = (eahr_query_stats * B)()
    rc = load().eahr_topk(dense.h if dense is not None else None, epoch,
                          sparse.h if sparse is not None else None, p, kind, qs, B, C.byref(prm),
                          _ptr(ids, C.c_int64), _ptr(cnt, C.c_int32), _ptr(stt, C.c_int32), stats)
    if not (rc == EAHR_E_FAILED and allow_failed):
        _check(rc)
    return ids[:, :K], cnt, stt, [s.as_dict() for s in stats]


def eahr_topk_merged(dense: Optional[PvsMerge], sparse: Optional[PbmIndex],
                     q_sparse: Sequence[Tuple[np.ndarray, np.ndarray]], B: int, K: int = 20,
                     k_rrf: int = 60, w_dense: int = 1, w_sparse: int = 1, depth0: int = 20,
                     growth: int = 2, allow_failed: bool = False):
    """eahr_topk over a merged dense ranking (pvs_merge_open / pvs_merge_shards)."""
    qs = (eahr_sparse_query * B)()
    keep = []
    if q_sparse is not None:
        for b, (t, w) in enumerate(q_sparse):
            q, k = _sparse_query(t, w)
            qs[b] = q
            keep.append(k)
    prm = _params(K, k_rrf, w_dense, w_sparse, depth0, growth)
    ids = np.full((B, max(K, 1)), -1, dtype=np.int64)
    cnt = np.zeros(B, dtype=np.int32)
    stt = np.zeros(B, dtype=np.int32)
    stats = (eahr_query_stats * B)()
    rc = load().eahr_topk_merged(dense.h if dense is not None else None,
                                 sparse.h if sparse is not None else None, qs, B, C.byref(prm),
                                 _ptr(ids, C.c_int64), _ptr(cnt, C.c_int32), _ptr(stt, C.c_int32), stats)
    if not (rc == EAHR_E_FAILED and allow_failed):
        _check(rc)
    return ids[:, :K], cnt, stt, [s.as_dict() for s in stats]


def eahr_fuse_lists(list_d, list_s, K: int = 20, k_rrf: int = 60, w_dense: int = 1,
                    w_sparse: int = 1, step: int = 0, depth0: int = 20, growth: int = 2,
                    schedule: str = "doubling"):
    """Fusion over two complete host rankings; returns (top ids, stats dict)."""
    a = np.ascontiguousarray(list_d, dtype=np.int64)
    b = np.ascontiguousarray(list_s, dtype=np.int64)
    prm = _params(K, k_rrf, w_dense, w_sparse, depth0, growth, schedule=schedule)
    out = np.full(max(K, 1), -1, dtype=np.int64)
    cnt = C.c_int32()
    st = eahr_query_stats()
    _check(load().eahr_fuse_lists(_ptr(a, C.c_int64), len(a), _ptr(b, C.c_int64), len(b),
                                  C.byref(prm), step, _ptr(out, C.c_int64), C.byref(cnt),
                                  C.byref(st)))
    return out[:cnt.value], st.as_dict()


class RankRecorder:
    """Context manager around eahr_set_rank_observer: records every rank the
    fusion reads, per (query, list), as (ids, scores) arrays.

        with RankRecorder() as rec:
            eahr_topk(...)
        ids, scores = rec.ranks(b, 0)      # dense ranks read for query b
    """

    def __init__(self):
        self._parts = {}
        self._cb = RANK_OBSERVER(self._record)

    def _record(self, user, query, lst, first, ids, scores, n):
        key = (int(query), int(lst))
        parts = self._parts.setdefault(key, [])
        have = sum(len(p[0]) for p in parts)
        assert first == have, (key, first, have)
        parts.append((np.ctypeslib.as_array(ids, shape=(n,)).copy(),
                      np.ctypeslib.as_array(scores, shape=(n,)).copy()))

    def __enter__(self):
        _check(load().eahr_set_rank_observer(self._cb, None))
        return self

    def __exit__(self, *exc):
        load().eahr_set_rank_observer(RANK_OBSERVER(), None)
        return False

    def ranks(self, query: int, lst: int):
        parts = self._parts.get((query, lst), [])
        if not parts:
            return np.zeros(0, np.int64), np.zeros(0, np.float32)
        return (np.concatenate([p[0] for p in parts]), np.concatenate([p[1] for p in parts]))


def eahr_set_rank_observer(fn, user=None) -> None:
    """Register a RANK_OBSERVER (or None to clear); keep fn referenced."""
    _check(load().eahr_set_rank_observer(fn if fn is not None else RANK_OBSERVER(), user))


def exported_symbols() -> List[str]:
    return list(SIGNATURES)
